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

// fp64 -> bf16 bits, round to nearest even, in one rounding: the value is
// first rounded to 8 significant bits in fp64 (integer arithmetic on its
// bits), which fp32 then holds exactly.  Finite values of normal bf16 range.
__device__ __forceinline__ uint32_t bf16_bits_rne(double x) {
  uint64_t b = (uint64_t)__double_as_longlong(x);
  b += 0x00000FFFFFFFFFFFull + ((b >> 45) & 1ull);   // half of 2^45 minus one, plus the kept lsb
  b &= ~0x00001FFFFFFFFFFFull;                       // keep sign, exponent, 7 fraction bits
  return __float_as_uint((float)__longlong_as_double((long long)b)) >> 16;
}

// Rotary pre-pass of the fused call (Algorithm 1, first step; 2-D axial
// reading).  Per (batch, head) the workgroups are: one per image block for K
// (rotate the block's K rows, write them, pool the rotated keys like
// k_pool), one per image block for Q (rotate and write), and one per 64 text
// rows (copy Q and K unchanged).  Channels [0, D/2) turn with the token's
// row, [D/2, D) with its column; pair i of a half (channels 2i, 2i + 1) by
// pos * inv_freq[i]; (a, b) -> (a cos - b sin, a sin + b cos) in fp64 with
// every product rounded, then rounded to bf16.  The block's 8 rows and 8
// columns give 2 * 8 * D/4 (cos, sin) pairs, computed while the block's rows
// are being read.
template <int D>
__global__ void __launch_bounds__(256) k_rope_pool_keys(RopeArgs r) {
  constexpr int P = D / 4;            // pairs per half
  constexpr int VPR = D / 8;          // 16-byte pieces per row
  constexpr int PER = 64 * VPR / 256; // pieces per thread
  __shared__ double cs[2][8][P][2];   // [row / column][index][pair][cos, sin]
  __shared__ uint4 stage[64 * VPR];   // rotated K of the block, [slot][piece]
  const IndexArgs& a = r.a;
  const int groups = 2 * a.n_tiles + r.n_text_groups;
  const int id = blockIdx.x, nbh = a.batch * a.heads;
  int bh, g;
  if ((nbh & 7) == 0) {   // whole heads per XCD, as the attention kernel maps them
    const int xcd = id & 7, sx = id >> 3;
    bh = xcd * (nbh >> 3) + sx / groups;
    g = sx % groups;
  } else {
    bh = id / groups;
    g = id % groups;
  }
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const int tid = threadIdx.x;
  if (g >= 2 * a.n_tiles) {   // text rows: copied
    const uint16_t* qin = static_cast<const uint16_t*>(a.q) + base;
    const uint16_t* kin = static_cast<const uint16_t*>(a.k) + base;
    uint16_t* qout = static_cast<uint16_t*>(r.q_out) + base;
    uint16_t* kout = static_cast<uint16_t*>(r.k_out) + base;
    const int row0 = 64 * (g - 2 * a.n_tiles);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int idx = tid + 256 * u, slot = idx / VPR, part = idx % VPR, row = row0 + slot;
      if (row < a.f.n_text) {
        const int64_t off = (int64_t)row * a.st + part * 8;
        *reinterpret_cast<uint4*>(qout + off) = *reinterpret_cast<const uint4*>(qin + off);
        *reinterpret_cast<uint4*>(kout + off) = *reinterpret_cast<const uint4*>(kin + off);
      }
    }
    return;
  }
  const bool is_k = g < a.n_tiles;
  const int t = is_k ? g : g - a.n_tiles, W = a.f.grid_w;
  const uint16_t* in = static_cast<const uint16_t*>(is_k ? a.k : a.q) + base;
  uint16_t* out = static_cast<uint16_t*>(is_k ? r.k_out : r.q_out) + base;
  // The block's rows, requested first.
  uint4 v[PER];
  int64_t off[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int idx = tid + 256 * u, slot = idx / VPR, part = idx % VPR;
    off[u] = (int64_t)frame_row(a.f, t, slot) * a.st + part * 8;
    v[u] = *reinterpret_cast<const uint4*>(in + off[u]);
  }
  // (cos, sin) of the block's rows and columns.
  for (int k = tid; k < 2 * 8 * P; k += 256) {
    const int axis = k / (8 * P), j = (k / P) % 8, i = k % P;
    // image id of slot (j, 0) (row j) or (0, j) (column j) of block t
    const int tok = frame_row(a.f, t, axis == 0 ? 8 * j : j) - a.f.n_text;
    const int pos = axis == 0 ? tok / W : tok % W;
    double sn, c;
    sincos(__dmul_rn((double)pos, r.inv_freq[i]), &sn, &c);
    cs[axis][j][i][0] = c;
    cs[axis][j][i][1] = sn;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int idx = tid + 256 * u, slot = idx / VPR, part = idx % VPR;
    const int c0 = 8 * part, axis = c0 / (D / 2), i0 = (c0 % (D / 2)) / 2;
    const int j = axis == 0 ? slot / 8 : slot % 8;
    const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {   // word e holds channels c0 + 2e (low half) and c0 + 2e + 1
      const double x0 = (double)__uint_as_float(w[e] << 16);
      const double x1 = (double)__uint_as_float(w[e] & 0xFFFF0000u);
      const double c = cs[axis][j][i0 + e][0], sn = cs[axis][j][i0 + e][1];
      const double y0 = __dsub_rn(__dmul_rn(x0, c), __dmul_rn(x1, sn));
      const double y1 = __dadd_rn(__dmul_rn(x0, sn), __dmul_rn(x1, c));
      o[e] = bf16_bits_rne(y0) | (bf16_bits_rne(y1) << 16);
    }
    const uint4 ov = make_uint4(o[0], o[1], o[2], o[3]);
    *reinterpret_cast<uint4*>(out + off[u]) = ov;
    if (is_k) stage[idx] = ov;
  }
  if (!is_k) return;
  __syncthreads();
  // Pooled rotated keys: thread c adds channel c over the slots in order.
  if (tid < D) {
    const char* col = reinterpret_cast<const char*>(stage) + (size_t)tid * 2;
    float xs[64];
#pragma unroll
    for (int u = 0; u < 64; ++u)   // bf16 -> f32 is exact
      xs[u] = __uint_as_float((uint32_t)*reinterpret_cast<const uint16_t*>(col + (size_t)u * D * 2) << 16);
    double sum = 0.0;
#pragma unroll
    for (int u = 0; u < 64; ++u) {
      const double x = (double)xs[u];
      sum = (u == 0) ? x : __dadd_rn(sum, x);
    }
    a.kb[((int64_t)bh * D + tid) * a.n_tiles + t] = sum;
  }
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

hipError_t launch_rope_pool_keys(const RopeArgs& r, hipStream_t s) {
  const IndexArgs& a = r.a;
  if (a.f.tile_log2 != 3 || (a.head_dim != 64 && a.head_dim != 128) || r.n_text_groups < 0)
    return hipErrorInvalidValue;   // 8x8 blocks (the gated attention kernel)
  dim3 grid((2 * a.n_tiles + r.n_text_groups) * a.heads * a.batch), block(256);
  if (a.head_dim == 64) hipLaunchKernelGGL((k_rope_pool_keys<64>), grid, block, 0, s, r);
  else hipLaunchKernelGGL((k_rope_pool_keys<128>), grid, block, 0, s, r);
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
