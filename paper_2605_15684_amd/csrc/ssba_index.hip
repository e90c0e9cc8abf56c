// SSBA gate kernels for gfx950: block pooling, block affinity, top-k ranking
// (Section 2.2.1 "Block Compression" Eq. 1, "Affinity Matrix", "Top-k Gating";
// Algorithm 1 pool, affinity and top-k steps) and the data-independent window
// and dense gates.
//
// Bit-reproducibility: pooled sums start from the block's first slot and add
// the following slots in order in fp64; each affinity is the channel-ordered
// fp64 sum of individually rounded products.  This file is compiled with
// -ffp-contract=off and the arithmetic is written with explicit
// round-to-nearest intrinsics, so no multiply-add is ever fused.
#include <hip/hip_runtime.h>
#include <type_traits>
#include <hip/hip_bf16.h>

#include "ssba_common.h"

namespace ssba {
namespace {

// (block, head, batch) of a workgroup in a 1-D grid of n_tiles * heads *
// batch workgroups.  Consecutive hardware ids go round-robin over the 8 XCDs;
// when the (batch, head) count divides by 8, each XCD gets whole heads -- the
// same heads the attention kernel gives it -- so pooled sums, index rows and
// the head's Q/K stay in one XCD's L2 from kernel to kernel.
__device__ __forceinline__ void unit_of(const IndexArgs& a, int& t, int& h, int& b) {
  const int id = blockIdx.x, nbh = a.batch * a.heads;
  int bh, r;
  if ((nbh & 7) == 0) {
    const int xcd = id & 7, s = id >> 3;
    bh = xcd * (nbh >> 3) + s / a.n_tiles;
    r = s % a.n_tiles;
  } else {
    bh = id / a.n_tiles;
    r = id % a.n_tiles;
  }
  t = r;
  b = bh / a.heads;
  h = bh - b * a.heads;
}

// Block pooling.  One workgroup pools Q and K (NT = 2), or K alone (NT = 1),
// of one block.  The block's rows are staged in LDS, up to 64 slots at a
// time, by all 256 threads with wide loads; then NT * D threads (one per
// channel of each tensor) add the staged slots in slot order in fp64, the
// ordered sum that makes the lists exact.  Pooled q is stored block-major
// [B][H][T_b][D]; pooled k channel-major [B][H][D][T_b], so that the gate
// reads one channel of all key blocks with one coalesced load.
template <int DTYPE, int TILE_LOG2, int D, int NT>
__device__ __forceinline__ void pool_block(const IndexArgs& a) {
  constexpr int SLOTS = 1 << (2 * TILE_LOG2);
  constexpr int SB = SLOTS < 64 ? SLOTS : 64;          // slots per stage
  constexpr bool BF16 = DTYPE == SSBA_DT_BF16;
  constexpr int EPV = BF16 ? 8 : 1;                    // elements per load
  constexpr int VPR = D / EPV;                         // loads per token row
  constexpr int LOADS = NT * SB * VPR;                 // per stage, (Q then) K
  using Vec = typename std::conditional<BF16, uint4, float>::type;
  __shared__ Vec stage[LOADS];
  int t, h, b;
  unit_of(a, t, h, b);
  const int tid = threadIdx.x;
  const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const int which = tid / D, c = tid % D;              // summing threads: tid < NT D
  double sum = 0.0;
#pragma unroll 1
  for (int s0 = 0; s0 < SLOTS; s0 += SB) {
    static_assert(LOADS % 256 == 0, "whole rounds of loads");
    Vec v[LOADS / 256];
#pragma unroll
    for (int r = 0; r < LOADS / 256; ++r) {
      const int idx = tid + 256 * r;
      const int tensor = idx / (SB * VPR), rem = idx % (SB * VPR);
      const int slot = rem / VPR, part = rem % VPR;
      const int64_t off = base + (int64_t)frame_row(a.f, t, s0 + slot) * a.st + part * EPV;
      const void* src = (NT == 2 && tensor == 0) ? a.q : a.k;
      v[r] = *reinterpret_cast<const Vec*>(static_cast<const char*>(src) + off * (BF16 ? 2 : 4));
    }
#pragma unroll
    for (int r = 0; r < LOADS / 256; ++r) stage[tid + 256 * r] = v[r];
    __syncthreads();
    if (tid < NT * D) {
      const char* col = reinterpret_cast<const char*>(stage) +
                        ((size_t)which * SB * D + c) * (BF16 ? 2 : 4);
      // Every staged value of the chain is read before the first add, so
      // the dependent fp64 adds never wait on LDS.
      float xs[SB];
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        if (BF16)   // bf16 -> f32 is exact
          xs[u] = __uint_as_float((uint32_t)*reinterpret_cast<const uint16_t*>(col + (size_t)u * D * 2) << 16);
        else
          xs[u] = *reinterpret_cast<const float*>(col + (size_t)u * D * 4);
      }
#pragma unroll
      for (int u = 0; u < SB; ++u) {
        const double x = (double)xs[u];
        sum = (s0 + u == 0) ? x : __dadd_rn(sum, x);
      }
    }
    __syncthreads();
  }
  if (tid < NT * D) {
    const int64_t bh = (int64_t)b * a.heads + h;
    if (NT == 2 && which == 0)
      a.qb[(bh * a.n_tiles + t) * D + c] = sum;
    else
      a.kb[(bh * D + c) * a.n_tiles + t] = sum;
  }
}

template <int DTYPE, int TILE_LOG2, int D, int NT>
__global__ void __launch_bounds__(256) k_pool(IndexArgs a) {
  pool_block<DTYPE, TILE_LOG2, D, NT>(a);
}

// Pooled key sums of several layers (grid y = layer), bf16, 8x8 blocks.
template <int D>
__global__ void __launch_bounds__(256) k_pool_keys_layers(PoolLayers p) {
  const int l = blockIdx.y;
  IndexArgs a = p.a;
  a.k = p.k[l];
  a.kb = p.kb[l];
  a.f = p.f[p.parity[l] & 1];
  pool_block<SSBA_DT_BF16, 3, D, 1>(a);
}

// S[i][j] of one (batch, head): the channel-ordered sum of the rounded
// products of the pooled query row qr (channel c at qr[c]) and the pooled key
// column kc (channel c at kc[c * tb]).  Each batch of pooled-k loads is
// requested before its first product, so a batch costs one memory round trip.
template <int D>
__device__ __forceinline__ double affinity_entry(const double* qr, const double* kc, int tb) {
  constexpr int BATCH = D < 64 ? D : 64;
  double s = 0.0;
#pragma unroll
  for (int c0 = 0; c0 < D; c0 += BATCH) {
    double kv[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) kv[u] = kc[(int64_t)(c0 + u) * tb];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const double p = __dmul_rn(qr[c0 + u], kv[u]);
      s = (c0 + u == 0) ? p : __dadd_rn(s, p);
    }
  }
  return s;
}

// Kept flag of block j (thread j of the workgroup) among the tb keys of the
// row: the `keep` first in (key descending, block id ascending).  MAXT == 64
// ranks in one wave; larger rows count, per key, the keys ranked before it.
template <int MAXT>
__device__ __forceinline__ bool rank_kept(uint64_t key, int j, int tb, int keep, const uint64_t* keys) {
  if (MAXT == 64) return wave_topk(key, j < tb, keep, j & 63);
  if (j >= tb) return false;
  int rank = 0;
  for (int jj = 0; jj < tb; ++jj) {
    const uint64_t kj = keys[jj];
    rank += (kj > key || (kj == key && jj < j)) ? 1 : 0;
  }
  return rank < keep;
}

// One workgroup per query block (i, h, b); thread j computes S[i][j] (the
// channel-ordered sum of rounded products) and its rank.  The `keep` blocks of
// lowest rank are kept and written in ascending block order.
template <int D, int MAXT>
__global__ void __launch_bounds__(MAXT) k_gate_topk(IndexArgs a) {
  extern __shared__ uint64_t keys[];   // [T_b]
  __shared__ int wave_kept[16];
  __shared__ int bad;
  int i, h, b;
  unit_of(a, i, h, b);
  const int tb = a.n_tiles;
  const int j = threadIdx.x, lane = j & 63, wave = j >> 6;
  const int64_t bh = (int64_t)b * a.heads + h;
  if (j == 0) bad = 0;
  __syncthreads();
  uint64_t key = 0;
  if (j < tb) {
    // the same query row for every thread; channel c of block j at kc[c * tb]
    const double s = affinity_entry<D>(a.qb + (bh * tb + i) * D, a.kb + bh * D * tb + j, tb);
    if (!isfinite(s)) atomicOr(&bad, 1);
    key = rank_key(s);
    keys[j] = key;
  }
  __syncthreads();
  const bool kept = rank_kept<MAXT>(key, j, tb, a.keep, keys);
  // Position of a kept block in the ascending list: kept blocks of lower id.
  const uint64_t mask = __ballot(kept);
  if (lane == 0) wave_kept[wave] = __popcll(mask);
  __syncthreads();
  int pos = __popcll(mask & ((1ull << lane) - 1ull));
  for (int w = 0; w < wave; ++w) pos += wave_kept[w];
  int32_t* out = a.index + (bh * tb + i) * (tb + 1);
  if (j < tb) {
    if (kept) out[1 + pos] = j;
    if (j >= a.keep) out[1 + j] = -1;
  }
  if (j == 0) {
    out[0] = a.keep;
    a.flags[bh * tb + i] = bad;
  }
}

// Head-shared gate, step 1: one workgroup per query block (i, h, b) writes
// its row of the per-head affinity, S_h[i][j] for j < T_b, to srows.
template <int D, int MAXT>
__device__ __forceinline__ void affinity_rows_body(const IndexArgs& a) {
  int i, h, b;
  unit_of(a, i, h, b);
  const int tb = a.n_tiles, j = threadIdx.x;
  const int64_t bh = (int64_t)b * a.heads + h;
  if (j < tb)
    a.srows[(bh * tb + i) * tb + j] = affinity_entry<D>(a.qb + (bh * tb + i) * D, a.kb + bh * D * tb + j, tb);
}

template <int D, int MAXT>
__global__ void __launch_bounds__(MAXT) k_affinity_rows(IndexArgs a) {
  affinity_rows_body<D, MAXT>(a);
}

// Head-shared gate, step 2: one workgroup per query block (i, b); thread j
// adds S_h[i][j] over heads h = 0, 1, ..., H-1 in that order (fp64), ranks
// the sums and writes the same kept list and status flag for every head.
template <int MAXT>
__device__ __forceinline__ void gate_shared_body(const IndexArgs& a) {
  extern __shared__ uint64_t keys[];   // [T_b]
  __shared__ int wave_kept[16];
  __shared__ int bad;
  const int tb = a.n_tiles;
  const int b = blockIdx.x / tb, i = blockIdx.x - b * tb;
  const int j = threadIdx.x, lane = j & 63, wave = j >> 6;
  if (j == 0) bad = 0;
  __syncthreads();
  uint64_t key = 0;
  if (j < tb) {
    const double* col = a.srows + ((int64_t)b * a.heads * tb + i) * tb + j;   // head h at col[h * tb * tb]
    const int64_t hstride = (int64_t)tb * tb;
    double s = 0.0;
    for (int h0 = 0; h0 < a.heads; h0 += 16) {
      const int nh = min(16, a.heads - h0);
      double v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = u < nh ? col[(h0 + u) * hstride] : 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (u < nh) s = (h0 + u == 0) ? v[u] : __dadd_rn(s, v[u]);
    }
    if (!isfinite(s)) atomicOr(&bad, 1);
    key = rank_key(s);
    keys[j] = key;
  }
  __syncthreads();
  const bool kept = rank_kept<MAXT>(key, j, tb, a.keep, keys);
  const uint64_t mask = __ballot(kept);
  if (lane == 0) wave_kept[wave] = __popcll(mask);
  __syncthreads();
  int pos = __popcll(mask & ((1ull << lane) - 1ull));
  for (int w = 0; w < wave; ++w) pos += wave_kept[w];
  for (int h = 0; h < a.heads; ++h) {
    const int64_t bh = (int64_t)b * a.heads + h;
    int32_t* out = a.index + (bh * tb + i) * (tb + 1);
    if (j < tb) {
      if (kept) out[1 + pos] = j;
      if (j >= a.keep) out[1 + j] = -1;
    }
    if (j == 0) {
      out[0] = a.keep;
      a.flags[bh * tb + i] = bad;
    }
  }
}

template <int MAXT>
__global__ void __launch_bounds__(MAXT) k_gate_shared(IndexArgs a) {
  gate_shared_body<MAXT>(a);
}

// The head-shared gate of several layers of one shape, one launch per step
// (grid y = layer): each workgroup does what it does for its own layer.
__device__ __forceinline__ IndexArgs layer_index_args(const IndexLayers& p) {
  const int l = blockIdx.y;
  IndexArgs a = p.a;
  a.q = p.q[l];
  a.k = p.k[l];
  a.index = p.index[l];
  a.qb = p.qb[l];
  a.kb = p.kb[l];
  a.flags = p.flags[l];
  a.srows = p.srows[l];
  a.keep = p.keep[l];
  a.f = p.f[p.parity[l] & 1];
  return a;
}

template <int TILE_LOG2, int D>
__global__ void __launch_bounds__(256) k_pool_layers(IndexLayers p) {
  pool_block<SSBA_DT_BF16, TILE_LOG2, D, 2>(layer_index_args(p));
}

template <int D>
__global__ void __launch_bounds__(64) k_affinity_rows_layers(IndexLayers p) {
  affinity_rows_body<D, 64>(layer_index_args(p));
}

__global__ void __launch_bounds__(64) k_gate_shared_layers(IndexLayers p) {
  gate_shared_body<64>(layer_index_args(p));
}

// Window (win_h x win_w blocks of the shifted frame) and dense gates.
__global__ void __launch_bounds__(1024) k_gate_static(IndexArgs a, int gate) {
  int i, h, b;
  unit_of(a, i, h, b);
  const int tb = a.n_tiles, nx = a.f.nx;
  const int j = threadIdx.x;
  const int64_t bh = (int64_t)b * a.heads + h;
  int32_t* out = a.index + (bh * tb + i) * (tb + 1);
  int count;
  if (gate == SSBA_GATE_DENSE) {
    count = tb;
    if (j < tb) out[1 + j] = j;
  } else {
    const int iy = i / nx, ix = i - iy * nx;
    const int wy0 = iy - iy % a.win_h, wx0 = ix - ix % a.win_w;
    count = a.win_h * a.win_w;
    if (j < tb) {
      const int jy = j / nx, jx = j - jy * nx;
      if (jy >= wy0 && jy < wy0 + a.win_h && jx >= wx0 && jx < wx0 + a.win_w)
        out[1 + (jy - wy0) * a.win_w + (jx - wx0)] = j;   // row-major = ascending
      if (j >= count) out[1 + j] = -1;
    }
  }
  if (j == 0) {
    out[0] = count;
    a.flags[bh * tb + i] = 0;
  }
}

int round_threads(int n) { return ((n + 63) / 64) * 64; }

template <int DTYPE, int D>
void launch_pool_d(const IndexArgs& a, hipStream_t s) {
  dim3 grid(a.n_tiles * a.heads * a.batch), block(256);
  switch (a.f.tile_log2) {
    case 2: hipLaunchKernelGGL((k_pool<DTYPE, 2, D, 2>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_pool<DTYPE, 3, D, 2>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((k_pool<DTYPE, 4, D, 2>), grid, block, 0, s, a); break;
  }
}

template <int DTYPE>
void launch_pool_t(const IndexArgs& a, hipStream_t s) {
  if (a.head_dim == 64) launch_pool_d<DTYPE, 64>(a, s);
  else launch_pool_d<DTYPE, 128>(a, s);
}

}  // namespace

hipError_t launch_pool(const IndexArgs& a, int dtype, hipStream_t s) {
  if (dtype == SSBA_DT_F32)
    launch_pool_t<SSBA_DT_F32>(a, s);
  else
    launch_pool_t<SSBA_DT_BF16>(a, s);
  return hipGetLastError();
}

hipError_t launch_pool_keys(const IndexArgs& a, hipStream_t s) {
  if (a.f.tile_log2 != 3) return hipErrorInvalidValue;   // 8x8 blocks (the gated attention kernel)
  dim3 grid(a.n_tiles * a.heads * a.batch), block(256);
  if (a.head_dim == 64) hipLaunchKernelGGL((k_pool<SSBA_DT_BF16, 3, 64, 1>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((k_pool<SSBA_DT_BF16, 3, 128, 1>), grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pool_keys_layers(const PoolLayers& p, int n_layers, hipStream_t s) {
  if (p.a.f.tile_log2 != 3 || p.f[0].tile_log2 != 3 || p.f[1].tile_log2 != 3 || n_layers < 1 ||
      n_layers > kPoolLayersMax)
    return hipErrorInvalidValue;
  dim3 grid(p.a.n_tiles * p.a.heads * p.a.batch, n_layers), block(256);
  if (p.a.head_dim == 64) hipLaunchKernelGGL((k_pool_keys_layers<64>), grid, block, 0, s, p);
  else hipLaunchKernelGGL((k_pool_keys_layers<128>), grid, block, 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gate_topk(const IndexArgs& a, hipStream_t s) {
  dim3 grid(a.n_tiles * a.heads * a.batch), block(round_threads(a.n_tiles));
  size_t lds = sizeof(uint64_t) * (size_t)a.n_tiles;
  // Small block counts get a small thread bound, which leaves registers to
  // hold every pooled-k load of a thread in flight at once.
  if (a.head_dim == 64) {
    if (block.x <= 64) hipLaunchKernelGGL((k_gate_topk<64, 64>), grid, block, lds, s, a);
    else if (block.x <= 256) hipLaunchKernelGGL((k_gate_topk<64, 256>), grid, block, lds, s, a);
    else hipLaunchKernelGGL((k_gate_topk<64, 1024>), grid, block, lds, s, a);
  } else {
    if (block.x <= 64) hipLaunchKernelGGL((k_gate_topk<128, 64>), grid, block, lds, s, a);
    else if (block.x <= 256) hipLaunchKernelGGL((k_gate_topk<128, 256>), grid, block, lds, s, a);
    else hipLaunchKernelGGL((k_gate_topk<128, 1024>), grid, block, lds, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_gate_topk_shared(const IndexArgs& a, hipStream_t s) {
  dim3 grid_rows(a.n_tiles * a.heads * a.batch), grid_b(a.n_tiles * a.batch), block(round_threads(a.n_tiles));
  const size_t lds = sizeof(uint64_t) * (size_t)a.n_tiles;
  if (block.x <= 64) {
    if (a.head_dim == 64) hipLaunchKernelGGL((k_affinity_rows<64, 64>), grid_rows, block, 0, s, a);
    else hipLaunchKernelGGL((k_affinity_rows<128, 64>), grid_rows, block, 0, s, a);
    hipLaunchKernelGGL((k_gate_shared<64>), grid_b, block, lds, s, a);
  } else if (block.x <= 256) {
    if (a.head_dim == 64) hipLaunchKernelGGL((k_affinity_rows<64, 256>), grid_rows, block, 0, s, a);
    else hipLaunchKernelGGL((k_affinity_rows<128, 256>), grid_rows, block, 0, s, a);
    hipLaunchKernelGGL((k_gate_shared<256>), grid_b, block, lds, s, a);
  } else {
    if (a.head_dim == 64) hipLaunchKernelGGL((k_affinity_rows<64, 1024>), grid_rows, block, 0, s, a);
    else hipLaunchKernelGGL((k_affinity_rows<128, 1024>), grid_rows, block, 0, s, a);
    hipLaunchKernelGGL((k_gate_shared<1024>), grid_b, block, lds, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_topk_shared_layers(const IndexLayers& p, int n_layers, hipStream_t s) {
  const IndexArgs& a = p.a;
  const int tl = a.f.tile_log2;
  if (n_layers < 1 || n_layers > kIndexLayersMax || a.n_tiles < 1 || a.n_tiles > 64 || (tl != 3 && tl != 4) ||
      p.f[0].tile_log2 != tl || p.f[1].tile_log2 != tl || (a.head_dim != 64 && a.head_dim != 128))
    return hipErrorInvalidValue;
  const dim3 grid_rows(a.n_tiles * a.heads * a.batch, n_layers), grid_b(a.n_tiles * a.batch, n_layers);
  const dim3 block_pool(256), block(round_threads(a.n_tiles));
  const size_t lds = sizeof(uint64_t) * (size_t)a.n_tiles;
  if (a.head_dim == 64) {
    if (tl == 3) hipLaunchKernelGGL((k_pool_layers<3, 64>), grid_rows, block_pool, 0, s, p);
    else hipLaunchKernelGGL((k_pool_layers<4, 64>), grid_rows, block_pool, 0, s, p);
    hipLaunchKernelGGL((k_affinity_rows_layers<64>), grid_rows, block, 0, s, p);
  } else {
    if (tl == 3) hipLaunchKernelGGL((k_pool_layers<3, 128>), grid_rows, block_pool, 0, s, p);
    else hipLaunchKernelGGL((k_pool_layers<4, 128>), grid_rows, block_pool, 0, s, p);
    hipLaunchKernelGGL((k_affinity_rows_layers<128>), grid_rows, block, 0, s, p);
  }
  hipLaunchKernelGGL(k_gate_shared_layers, grid_b, block, lds, s, p);
  return hipGetLastError();
}

hipError_t launch_gate_static(const IndexArgs& a, int gate, hipStream_t s) {
  dim3 grid(a.n_tiles * a.heads * a.batch), block(round_threads(a.n_tiles));
  hipLaunchKernelGGL(k_gate_static, grid, block, 0, s, a, gate);
  return hipGetLastError();
}

}  // namespace ssba
