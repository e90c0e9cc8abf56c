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
#include <hip/hip_bf16.h>

#include "ssba_common.h"

namespace ssba {
namespace {

__device__ __forceinline__ double load_as_f64(const void* base, int64_t off, int dtype) {
  if (dtype == SSBA_DT_F32) return (double)static_cast<const float*>(base)[off];
  const uint16_t bits = static_cast<const uint16_t*>(base)[off];
  return (double)__uint_as_float((uint32_t)bits << 16);  // bf16 -> f32 is exact
}

// One workgroup per (block t, head h, batch b); threads [0, D) pool Q channel
// c, threads [D, 2D) pool K channel c.  Reads every image row of Q and K once.
template <int DTYPE>
__global__ void __launch_bounds__(256) k_pool(IndexArgs a) {
  const int t = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int D = a.head_dim;
  const int which = threadIdx.x / D;  // 0 = Q, 1 = K
  const int c = threadIdx.x - which * D;
  if (which > 1) return;
  const void* src = which == 0 ? a.q : a.k;
  double* dst = which == 0 ? a.qb : a.kb;
  const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh + c;
  const int slots = 1 << (2 * a.f.tile_log2);
  double sum = load_as_f64(src, base + (int64_t)frame_row(a.f, t, 0) * a.st, DTYPE);
  for (int s = 1; s < slots; ++s)
    sum = __dadd_rn(sum, load_as_f64(src, base + (int64_t)frame_row(a.f, t, s) * a.st, DTYPE));
  dst[(((int64_t)b * a.heads + h) * a.n_tiles + t) * D + c] = sum;
}

// Strict total order used for ranking: a larger affinity first, NaN after every
// number, equal values (including +0 / -0) by ascending block index.
__device__ __forceinline__ bool ranks_before(double sa, int ja, double sb, int jb) {
  const bool na = sa != sa, nb = sb != sb;
  if (na || nb) return (!na) || (na && nb && ja < jb);
  return sa > sb || (sa == sb && ja < jb);
}

// One workgroup per query block (i, h, b); thread j computes S[i][j] and its
// rank.  Blocks ranked below `keep` are kept; the kept ids are written in
// ascending order.
__global__ void __launch_bounds__(1024) k_gate_topk(IndexArgs a) {
  extern __shared__ double smem[];
  double* qrow = smem;                 // [D]
  double* srow = smem + a.head_dim;    // [T_b]
  __shared__ int keptf[1024];
  __shared__ int bad;
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int D = a.head_dim, tb = a.n_tiles;
  const int j = threadIdx.x;
  const int64_t bh = (int64_t)b * a.heads + h;
  if (j == 0) bad = 0;
  for (int c = j; c < D; c += blockDim.x) qrow[c] = a.qb[(bh * tb + i) * D + c];
  __syncthreads();
  double s = 0.0;
  if (j < tb) {
    const double* kr = a.kb + (bh * tb + j) * D;
    s = __dmul_rn(qrow[0], kr[0]);
    for (int c = 1; c < D; ++c) s = __dadd_rn(s, __dmul_rn(qrow[c], kr[c]));
    srow[j] = s;
    if (!isfinite(s)) atomicOr(&bad, 1);
  }
  __syncthreads();
  int kept = 0;
  if (j < tb) {
    int rank = 0;
    for (int jj = 0; jj < tb; ++jj) rank += ranks_before(srow[jj], jj, s, j) ? 1 : 0;
    kept = rank < a.keep;
    keptf[j] = kept;
  }
  __syncthreads();
  int32_t* out = a.index + (bh * tb + i) * (tb + 1);
  if (j < tb) {
    if (kept) {
      int pos = 0;
      for (int jj = 0; jj < j; ++jj) pos += keptf[jj];
      out[1 + pos] = j;
    }
    if (j >= a.keep) out[1 + j] = -1;
  }
  if (j == 0) {
    out[0] = a.keep;
    a.flags[bh * tb + i] = bad;
  }
}

// Window (win_h x win_w blocks of the shifted frame) and dense gates.
__global__ void __launch_bounds__(1024) k_gate_static(IndexArgs a, int gate) {
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
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

}  // namespace

hipError_t launch_pool(const IndexArgs& a, int dtype, hipStream_t s) {
  dim3 grid(a.n_tiles, a.heads, a.batch), block(2 * a.head_dim);
  if (dtype == SSBA_DT_F32)
    hipLaunchKernelGGL(k_pool<SSBA_DT_F32>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_pool<SSBA_DT_BF16>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gate_topk(const IndexArgs& a, hipStream_t s) {
  dim3 grid(a.n_tiles, a.heads, a.batch), block(round_threads(a.n_tiles));
  size_t lds = sizeof(double) * (size_t)(a.head_dim + a.n_tiles);
  hipLaunchKernelGGL(k_gate_topk, grid, block, lds, s, a);
  return hipGetLastError();
}

hipError_t launch_gate_static(const IndexArgs& a, int gate, hipStream_t s) {
  dim3 grid(a.n_tiles, a.heads, a.batch), block(round_threads(a.n_tiles));
  hipLaunchKernelGGL(k_gate_static, grid, block, 0, s, a, gate);
  return hipGetLastError();
}

}  // namespace ssba
