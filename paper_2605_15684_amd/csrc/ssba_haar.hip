// Multi-level 2-D Haar transform pair of the Tiny DWT-Distilled VAE
// (Section 2.3.1: the DWT equation, a single Haar kernel bank applied level
// after level; the IWT equation, the decoder's inverse pyramid with a
// residual per level).  Both directions are streaming: one thread owns a
// strip of 2^L rows x 8 columns of one (n, c) plane, reads it once, runs every
// level in registers and writes every level's bands (or reads every level's
// bands and writes the strip), so each byte crosses HBM once.  Adjacent
// threads own adjacent strips of a row, so every row access of a wave is one
// contiguous run.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssba_haar.h"

namespace ssba_haar {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

struct Args {
  const void* x;        // DWT input / IWT output plane data
  void* y;              // IWT output
  void* lv[3];          // level l + 1: [N][4C][H >> (l+1)][W >> (l+1)]
  const void* res[3];   // IWT residual of LL^(l) (l = 0: the output), or null
  int64_t planes;       // N * C
  int h, w;             // input plane size
  int64_t strips;       // planes * (h >> L) * (w / 8)
};

// N consecutive elements of one row, as floats.
template <typename T, int N>
__device__ __forceinline__ void load_row(const T* p, float (&v)[N]) {
  if constexpr (sizeof(T) == 4) {
    if constexpr (N == 8) {
      const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else if constexpr (N == 4) {
      const float4 a = *reinterpret_cast<const float4*>(p);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    } else if constexpr (N == 2) {
      const float2 a = *reinterpret_cast<const float2*>(p);
      v[0] = a.x; v[1] = a.y;
    } else {
      v[0] = *reinterpret_cast<const float*>(p);
    }
  } else {   // bf16: widen exactly by moving the bits to the top half
    uint32_t u[(N + 1) / 2];
    if constexpr (N == 8) {
      const uint4 a = *reinterpret_cast<const uint4*>(p);
      u[0] = a.x; u[1] = a.y; u[2] = a.z; u[3] = a.w;
    } else if constexpr (N == 4) {
      const uint2 a = *reinterpret_cast<const uint2*>(p);
      u[0] = a.x; u[1] = a.y;
    } else if constexpr (N == 2) {
      u[0] = *reinterpret_cast<const uint32_t*>(p);
    } else {
      u[0] = *reinterpret_cast<const uint16_t*>(p);
    }
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = __uint_as_float(((u[i / 2] >> (16 * (i & 1))) & 0xFFFFu) << 16);
  }
}

// Two floats -> two bf16 (round to nearest even) in one word.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

template <typename T, int N>
__device__ __forceinline__ void store_row(T* p, const float (&v)[N]) {
  if constexpr (sizeof(T) == 4) {
    if constexpr (N == 8) {
      reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
      reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
    } else if constexpr (N == 4) {
      *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    } else if constexpr (N == 2) {
      *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
    } else {
      *reinterpret_cast<float*>(p) = v[0];
    }
  } else {
    if constexpr (N == 8) {
      *reinterpret_cast<uint4*>(p) = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
    } else if constexpr (N == 4) {
      *reinterpret_cast<uint2*>(p) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
    } else if constexpr (N == 2) {
      *reinterpret_cast<uint32_t*>(p) = pack2(v[0], v[1]);
    } else {
      *reinterpret_cast<uint16_t*>(p) = (uint16_t)(pack2(v[0], 0.f) & 0xFFFFu);
    }
  }
}

// Strip of thread `t`: plane, first row and first column (in input pixels).
template <int L>
__device__ __forceinline__ bool strip_of(const Args& a, int64_t t, int64_t& plane, int& r0, int& c0) {
  if (t >= a.strips) return false;
  const int sx = a.w / 8, sy = a.h >> L;
  const int64_t per_plane = (int64_t)sx * sy;
  plane = t / per_plane;
  const int rem = (int)(t - plane * per_plane);
  r0 = (rem / sx) << L;
  c0 = (rem % sx) * 8;
  return true;
}

// Forward: the strip's 2^L x 8 pixels -> level 1 .. L bands.  Level l works
// on the LL tile of level l - 1 (2^(L-l+1) x 8/2^(l-1), unrounded) and writes
// its four bands, 2^(L-l) rows of 8/2^l values each.
template <typename T, int L>
__global__ void __launch_bounds__(256) k_haar_dwt(Args a) {
  int64_t plane;
  int r0, c0;
  if (!strip_of<L>(a, (int64_t)blockIdx.x * blockDim.x + threadIdx.x, plane, r0, c0)) return;
  constexpr int R = 1 << L;
  float t[R][8];
  const T* xp = static_cast<const T*>(a.x) + (plane * a.h + r0) * a.w + c0;
#pragma unroll
  for (int r = 0; r < R; ++r) load_row<T, 8>(xp + (int64_t)r * a.w, t[r]);
#pragma unroll
  for (int l = 1; l <= L; ++l) {
    const int rows = R >> l, cols = 8 >> l;               // output tile of this level
    const int hl = a.h >> l, wl = a.w >> l;
    T* base = static_cast<T*>(a.lv[l - 1]);
    float band[4][R / 2][4];
#pragma unroll
    for (int i = 0; i < R / 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (i < rows && j < cols) {
          const float p = t[2 * i][2 * j], q = t[2 * i][2 * j + 1];
          const float u = t[2 * i + 1][2 * j], v = t[2 * i + 1][2 * j + 1];
          band[0][i][j] = ((p + q) + (u + v)) * 0.5f;
          band[1][i][j] = ((p - q) + (u - v)) * 0.5f;
          band[2][i][j] = ((p + q) - (u + v)) * 0.5f;
          band[3][i][j] = ((p - q) - (u - v)) * 0.5f;
        }
    const int orow = (r0 >> l), ocol = (c0 >> l);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      T* bp = base + ((plane * 4 + b) * hl + orow) * (int64_t)wl + ocol;
#pragma unroll
      for (int i = 0; i < R / 2; ++i)
        if (i < rows) {
          if (cols == 4) {
            float v4[4] = {band[b][i][0], band[b][i][1], band[b][i][2], band[b][i][3]};
            store_row<T, 4>(bp + (int64_t)i * wl, v4);
          } else if (cols == 2) {
            float v2[2] = {band[b][i][0], band[b][i][1]};
            store_row<T, 2>(bp + (int64_t)i * wl, v2);
          } else {
            float v1[1] = {band[b][i][0]};
            store_row<T, 1>(bp + (int64_t)i * wl, v1);
          }
        }
    }
    // The next level works on this level's LL tile.
#pragma unroll
    for (int i = 0; i < R / 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (i < rows && j < cols) t[i][j] = band[0][i][j];
  }
}

// Inverse: from the coarsest level's LL and every level's detail bands back
// to the strip, adding the residual of each reconstructed LL when given.
template <typename T, int L>
__global__ void __launch_bounds__(256) k_haar_iwt(Args a) {
  int64_t plane;
  int r0, c0;
  if (!strip_of<L>(a, (int64_t)blockIdx.x * blockDim.x + threadIdx.x, plane, r0, c0)) return;
  constexpr int R = 1 << L;
  float t[R][8];   // the current LL tile: (R >> l) x (8 >> l) at level l
  {
    const int hl = a.h >> L, wl = a.w >> L, cols = 8 >> L;
    const T* p = static_cast<const T*>(a.lv[L - 1]) + ((plane * 4 + 0) * hl + (r0 >> L)) * (int64_t)wl + (c0 >> L);
    float v[8];
    if (cols == 1) { float x1[1]; load_row<T, 1>(p, x1); v[0] = x1[0]; }
    else if (cols == 2) { float x2[2]; load_row<T, 2>(p, x2); v[0] = x2[0]; v[1] = x2[1]; }
    else { float x4[4]; load_row<T, 4>(p, x4); v[0] = x4[0]; v[1] = x4[1]; v[2] = x4[2]; v[3] = x4[3]; }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < cols) t[0][j] = v[j];
  }
#pragma unroll
  for (int l = L; l >= 1; --l) {
    const int rows = R >> l, cols = 8 >> l;               // band tile of this level
    const int hl = a.h >> l, wl = a.w >> l;
    const T* base = static_cast<const T*>(a.lv[l - 1]);
    float d[3][R / 2][4];
#pragma unroll
    for (int b = 1; b < 4; ++b) {
      const T* bp = base + ((plane * 4 + b) * hl + (r0 >> l)) * (int64_t)wl + (c0 >> l);
#pragma unroll
      for (int i = 0; i < R / 2; ++i)
        if (i < rows) {
          if (cols == 4) {
            float v4[4];
            load_row<T, 4>(bp + (int64_t)i * wl, v4);
#pragma unroll
            for (int j = 0; j < 4; ++j) d[b - 1][i][j] = v4[j];
          } else if (cols == 2) {
            float v2[2];
            load_row<T, 2>(bp + (int64_t)i * wl, v2);
            d[b - 1][i][0] = v2[0];
            d[b - 1][i][1] = v2[1];
          } else {
            float v1[1];
            load_row<T, 1>(bp + (int64_t)i * wl, v1);
            d[b - 1][i][0] = v1[0];
          }
        }
    }
    float n[R][8];
#pragma unroll
    for (int i = 0; i < R / 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (i < rows && j < cols) {
          const float ll = t[i][j], hlv = d[0][i][j], lh = d[1][i][j], hh = d[2][i][j];
          n[2 * i][2 * j] = ((ll + hlv) + (lh + hh)) * 0.5f;
          n[2 * i][2 * j + 1] = ((ll - hlv) + (lh - hh)) * 0.5f;
          n[2 * i + 1][2 * j] = ((ll + hlv) - (lh + hh)) * 0.5f;
          n[2 * i + 1][2 * j + 1] = ((ll - hlv) - (lh - hh)) * 0.5f;
        }
    // Residual of LL^(l-1) (the output when l == 1).
    const int h0 = a.h >> (l - 1), w0 = a.w >> (l - 1);
    if (a.res[l - 1]) {
      const T* rp = static_cast<const T*>(a.res[l - 1]) + (plane * h0 + (r0 >> (l - 1))) * (int64_t)w0 + (c0 >> (l - 1));
#pragma unroll
      for (int i = 0; i < R; ++i)
        if (i < 2 * rows) {
          float rv[8];
          if (2 * cols == 8) load_row<T, 8>(rp + (int64_t)i * w0, rv);
          else if (2 * cols == 4) { float x4[4]; load_row<T, 4>(rp + (int64_t)i * w0, x4); for (int j = 0; j < 4; ++j) rv[j] = x4[j]; }
          else { float x2[2]; load_row<T, 2>(rp + (int64_t)i * w0, x2); rv[0] = x2[0]; rv[1] = x2[1]; }
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (j < 2 * cols) n[i][j] += rv[j];
        }
    }
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (i < 2 * rows && j < 2 * cols) t[i][j] = n[i][j];
  }
  T* yp = static_cast<T*>(a.y) + (plane * a.h + r0) * a.w + c0;
#pragma unroll
  for (int r = 0; r < R; ++r) store_row<T, 8>(yp + (int64_t)r * a.w, t[r]);
}

template <typename T>
hipError_t launch(const Args& a, int levels, bool inverse, hipStream_t s) {
  const dim3 block(256), grid((unsigned)((a.strips + 255) / 256));
  if (!inverse) {
    switch (levels) {
      case 1: hipLaunchKernelGGL((k_haar_dwt<T, 1>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((k_haar_dwt<T, 2>), grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL((k_haar_dwt<T, 3>), grid, block, 0, s, a); break;
    }
  } else {
    switch (levels) {
      case 1: hipLaunchKernelGGL((k_haar_iwt<T, 1>), grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL((k_haar_iwt<T, 2>), grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL((k_haar_iwt<T, 3>), grid, block, 0, s, a); break;
    }
  }
  return hipGetLastError();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

ssba_status check(const ssba_haar_desc* d, Args& a) {
  if (!d) return SSBA_ERR_ARG;
  if (d->n < 1 || d->c < 1 || d->h < 1 || d->w < 1) return SSBA_ERR_SHAPE;
  if (d->levels < 1 || d->levels > 3) return SSBA_ERR_UNSUPPORTED;
  if (d->dtype != SSBA_DT_BF16 && d->dtype != SSBA_DT_F32) return SSBA_ERR_ARG;
  if (d->h % (1 << d->levels) || d->w % 8) return SSBA_ERR_SHAPE;
  const int64_t planes = (int64_t)d->n * d->c;
  const int64_t elems = planes * d->h * d->w;
  if (elems > ((int64_t)1 << 40)) return SSBA_ERR_UNSUPPORTED;
  a = Args{};
  a.planes = planes;
  a.h = d->h;
  a.w = d->w;
  a.strips = planes * (d->h >> d->levels) * (d->w / 8);
  if ((a.strips + 255) / 256 > 0x7FFFFFFF) return SSBA_ERR_UNSUPPORTED;
  return SSBA_OK;
}

}  // namespace
}  // namespace ssba_haar

extern "C" {

ssba_status ssba_haar_dwt(const ssba_haar_desc* d, const void* x, void* const* levels, void* stream) {
  ssba_haar::Args a;
  const ssba_status st = ssba_haar::check(d, a);
  if (st != SSBA_OK) return st;
  if (!x || !levels || !ssba_haar::aligned16(x)) return SSBA_ERR_ARG;
  for (int l = 0; l < d->levels; ++l) {
    if (!levels[l] || !ssba_haar::aligned16(levels[l])) return SSBA_ERR_ARG;
    a.lv[l] = levels[l];
  }
  a.x = x;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  const hipError_t e = d->dtype == SSBA_DT_F32 ? ssba_haar::launch<float>(a, d->levels, false, hs)
                                               : ssba_haar::launch<uint16_t>(a, d->levels, false, hs);
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_haar_iwt(const ssba_haar_desc* d, const void* const* levels, const void* const* residuals,
                          void* x, void* stream) {
  ssba_haar::Args a;
  const ssba_status st = ssba_haar::check(d, a);
  if (st != SSBA_OK) return st;
  if (!x || !levels || !ssba_haar::aligned16(x)) return SSBA_ERR_ARG;
  for (int l = 0; l < d->levels; ++l) {
    if (!levels[l] || !ssba_haar::aligned16(levels[l])) return SSBA_ERR_ARG;
    a.lv[l] = const_cast<void*>(levels[l]);
    const void* r = residuals ? residuals[l] : nullptr;
    if (r && !ssba_haar::aligned16(r)) return SSBA_ERR_ARG;
    a.res[l] = r;
  }
  a.y = x;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  const hipError_t e = d->dtype == SSBA_DT_F32 ? ssba_haar::launch<float>(a, d->levels, true, hs)
                                               : ssba_haar::launch<uint16_t>(a, d->levels, true, hs);
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

const char* ssba_haar_kernel_name(const ssba_haar_desc* d, int inverse) {
  static const char* const names[2][2][3] = {
      {{"k_haar_dwt<unsigned short, 1>", "k_haar_dwt<unsigned short, 2>", "k_haar_dwt<unsigned short, 3>"},
       {"k_haar_dwt<float, 1>", "k_haar_dwt<float, 2>", "k_haar_dwt<float, 3>"}},
      {{"k_haar_iwt<unsigned short, 1>", "k_haar_iwt<unsigned short, 2>", "k_haar_iwt<unsigned short, 3>"},
       {"k_haar_iwt<float, 1>", "k_haar_iwt<float, 2>", "k_haar_iwt<float, 3>"}}};
  ssba_haar::Args a;
  if (ssba_haar::check(d, a) != SSBA_OK) return nullptr;
  return names[inverse ? 1 : 0][d->dtype == SSBA_DT_F32 ? 1 : 0][d->levels - 1];
}

}  // extern "C"
