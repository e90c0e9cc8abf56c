// SSBA block-sparse attention forward in fp32 (fp32 inputs, products,
// accumulation and output) for gfx950 -- the full-precision path.
//
// Same decomposition and key order as the bf16 kernel (Algorithm 1, attend
// step; masked blocks are never read): a workgroup of 64 threads owns up to
// 64 query rows of one query block (or of the natural-order rows), one row per
// thread, and streams 64-key chunks through LDS.  Each chunk is scored into
// LDS, then folded into the running max / sum / output of every row.
#include <hip/hip_runtime.h>

#include "ssba_common.h"

namespace ssba {
namespace {

constexpr int KC = 64;
constexpr int NT = 64;

struct Plan {
  const int32_t* list;
  int count, img_chunks, n_chunks, natural_end;
};

__device__ __forceinline__ int key_row(const Plan& p, const AttnArgs& a, int slots, int c, int kk) {
  if (p.natural_end) {
    const int r = c * KC + kk;
    return r < p.natural_end ? r : -1;
  }
  if (c < p.img_chunks) {
    int e, s;
    if (slots >= KC) {
      const int cpt = slots / KC;
      e = c / cpt;
      s = (c - e * cpt) * KC + kk;
    } else {
      e = c * (KC / slots) + kk / slots;
      s = kk % slots;
      if (e >= p.count) return -1;
    }
    const int j = p.list[1 + e];
    if ((unsigned)j >= (unsigned)a.n_tiles) return -1;
    return frame_row(a.f, j, s);
  }
  const int r = (c - p.img_chunks) * KC + kk;
  return r < a.f.n_text ? r : -1;
}

template <int D>
__global__ void __launch_bounds__(NT) k_attn_f32(AttnArgs a, int qr_img) {
  __shared__ float ks[KC][D + 1];
  __shared__ float vs[KC][D + 1];
  __shared__ float sc[NT][KC + 1];
  __shared__ int rows[KC];

  const int L = blockIdx.x;
  const int bh = L / a.groups_per_bh;
  const int r = L - bh * a.groups_per_bh;
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t off = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const float* qbase = static_cast<const float*>(a.q) + off;
  const float* kbase = static_cast<const float*>(a.k) + off;
  const float* vbase = static_cast<const float*>(a.v) + off;
  float* obase = static_cast<float*>(a.o) + off;
  const int tid = threadIdx.x;
  const int slots = 1 << (2 * a.f.tile_log2);

  Plan p;
  int qrow = -1;
  if (a.dense || r < a.n_text_groups) {
    const int end = a.dense ? a.seq : a.f.n_text;
    const int q = r * NT + tid;
    qrow = q < end ? q : -1;
    p.list = nullptr;
    p.count = 0;
    p.img_chunks = 0;
    p.natural_end = a.seq;
    p.n_chunks = (a.seq + KC - 1) / KC;
  } else {
    const int ir = r - a.n_text_groups;
    const int i = ir / a.groups_per_tile, part = ir - i * a.groups_per_tile;
    qrow = tid < qr_img ? frame_row(a.f, i, part * qr_img + tid) : -1;
    p.list = a.index + (bh * (int64_t)a.n_tiles + i) * (a.n_tiles + 1);
    p.count = min(max(p.list[0], 0), a.n_tiles);
    p.img_chunks = slots >= KC ? p.count * (slots / KC) : (p.count + (KC / slots) - 1) / (KC / slots);
    p.natural_end = 0;
    p.n_chunks = p.img_chunks + (a.f.n_text + KC - 1) / KC;
  }

  float qv[D], acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qv[d] = qrow >= 0 ? qbase[(int64_t)qrow * a.st + d] : 0.f;
    acc[d] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;

  for (int c = 0; c < p.n_chunks; ++c) {
    rows[tid] = key_row(p, a, slots, c, tid);
    __syncthreads();
    for (int e = tid; e < KC * D; e += NT) {
      const int kk = e / D, d = e - kk * D;
      const int row = rows[kk];
      ks[kk][d] = row >= 0 ? kbase[(int64_t)row * a.st + d] : 0.f;
      vs[kk][d] = row >= 0 ? vbase[(int64_t)row * a.st + d] : 0.f;
    }
    __syncthreads();
    float cmax = -INFINITY;
    for (int kk = 0; kk < KC; ++kk) {
      float s = -INFINITY;
      if (rows[kk] >= 0) {
        float dot = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) dot = __builtin_fmaf(qv[d], ks[kk][d], dot);
        s = dot * a.scale;
      }
      sc[tid][kk] = s;
      cmax = fmaxf(cmax, s);
    }
    const float m_new = fmaxf(m_run, cmax);
    if (m_new > -INFINITY) {
      const float alpha = expf(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] *= alpha;
      m_run = m_new;
      for (int kk = 0; kk < KC; ++kk) {
        const float pk = expf(sc[tid][kk] - m_run);
        l_run += pk;
#pragma unroll
        for (int d = 0; d < D; ++d) acc[d] = __builtin_fmaf(pk, vs[kk][d], acc[d]);
      }
    }
    __syncthreads();
  }
  if (qrow >= 0) {
    const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) obase[(int64_t)qrow * a.st + d] = acc[d] * inv;
  }
}

template <int D>
hipError_t launch_t(const AttnArgs& a0, int tile, hipStream_t s) {
  AttnArgs a = a0;
  const int slots = tile * tile;
  const int qr = slots < NT ? slots : NT;
  const int nat_qr = NT;
  if (a.dense) {
    a.n_text_groups = 0;
    a.groups_per_tile = 1;
    a.groups_per_bh = (a.seq + nat_qr - 1) / nat_qr;
  } else {
    a.n_text_groups = (a.f.n_text + nat_qr - 1) / nat_qr;
    a.groups_per_tile = slots / qr;
    a.groups_per_bh = a.n_text_groups + a.n_tiles * a.groups_per_tile;
  }
  const int64_t total = (int64_t)a.batch * a.heads * a.groups_per_bh;
  if (total <= 0) return hipSuccess;
  // Natural-order groups (text rows, dense path) hold 64 rows; image groups
  // hold min(64, tile^2) rows of one block.
  hipLaunchKernelGGL(k_attn_f32<D>, dim3((unsigned)total), dim3(NT), 0, s, a, qr);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, int tile, hipStream_t s) {
  if (head_dim == 64) return launch_t<64>(a, tile, s);
  return launch_t<128>(a, tile, s);
}

}  // namespace ssba
