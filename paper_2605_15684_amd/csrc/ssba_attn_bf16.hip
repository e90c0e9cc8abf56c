// SSBA block-sparse attention forward, bf16 in / bf16 out, for gfx950.
//
// Computes the attend step of Algorithm 1 (Section 2.2.1, "Efficient Sparse
// Execution"): each image query block attends only the key blocks its gate
// kept (masked blocks are never read from memory) plus every text key; text
// query rows attend every key.  The dense control runs the same code with
// every row in natural order over every key.
//
// Work decomposition.  One workgroup owns up to 64 query rows of one
// (batch, head): a query block of the shifted frame (or a quarter of a 16x16
// block), or 64 consecutive rows in natural order.  Wave w owns 16 of them.
// Keys stream through LDS in chunks of 64 (one 8x8 block, a quarter of a
// 16x16 block, four 4x4 blocks, or 64 consecutive rows), double-buffered
// through registers.  Rows are gathered through the shifted-frame address map,
// so the shift never moves data.
//
// Per chunk and wave, with lane = 16 * g + n (query n of the wave, key group g):
//   S^T[64 keys][16 queries] = K_chunk . Q^T     v_mfma_f32_16x16x32_bf16, fp32 acc
//   online softmax in the log2 domain; a query's row maximum is reduced over
//   its four lanes, so every lane holds its query's running max and a partial
//   row sum; the output is rescaled only when the max grows by more than 2^8.
//   O^T[D][16 queries] += V_chunk^T . P^T        P rounded to bf16 (RNE)
// Computing the transposed products keeps each query's scores, probabilities
// and output in its own lanes, so P feeds the second product straight from
// registers.  The second product contracts keys in the order its operands
// hold them: key group g of 32-key step k holds keys 32k + 4g + {0..3} and
// 32k + 16 + 4g + {0..3}; V is stored transposed in LDS so both runs are
// 8-byte reads.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>

#include "ssba_common.h"

namespace ssba {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

constexpr int KC = 64;                 // keys per chunk
constexpr float kRescaleSlack = 8.0f;  // log2 units: rescale when the max grows by > 2^8

template <int TILE_LOG2>
constexpr int threads_of() { return TILE_LOG2 == 2 ? 64 : 256; }  // 4x4 blocks: one wave per block

template <int D, int TILE_LOG2>
struct Cfg {
  static constexpr int WAVES = threads_of<TILE_LOG2>() / 64;
  static constexpr int NT = 64 * WAVES;
  static constexpr int QR = 16 * WAVES;                   // query rows per workgroup
  static constexpr int SLOTS = 1 << (2 * TILE_LOG2);
  static constexpr int KROW = D + 8;                      // K row stride in LDS (elements)
  static constexpr int VROW = KC + 4;                     // V^T row stride in LDS (elements)
  static constexpr int K_ELEMS = KC * KROW;
  static constexpr int V_ELEMS = D * VROW;
  static constexpr int BUF = K_ELEMS + V_ELEMS;
  static constexpr int KP = KC * D / 8 / NT;              // 16-byte K pieces per thread
  static constexpr int VG = KC * D / 16 / NT;             // 4-key x 4-channel V groups per thread
  static_assert(KP >= 1 && VG >= 1, "tiling");
};

// Where the keys of one workgroup come from.
struct Plan {
  const int32_t* list;  // kept block ids (image mode)
  int count;            // kept blocks
  int img_chunks;       // chunks drawn from the kept blocks
  int n_chunks;         // total chunks
  int natural_end;      // natural mode: keys are rows [0, natural_end); 0 = image mode
};

template <int TILE_LOG2>
__device__ __forceinline__ int key_row(const Plan& p, const AttnArgs& a, int c, int kk) {
  constexpr int SLOTS = 1 << (2 * TILE_LOG2);
  if (p.natural_end) {
    const int r = c * KC + kk;
    return r < p.natural_end ? r : -1;
  }
  if (c < p.img_chunks) {
    int e, s;
    if constexpr (SLOTS >= KC) {
      constexpr int CPT = SLOTS / KC;
      e = c / CPT;
      s = (c - e * CPT) * KC + kk;
    } else {
      e = c * (KC / SLOTS) + kk / SLOTS;
      s = kk % SLOTS;
      if (e >= p.count) return -1;
    }
    const int j = p.list[1 + e];
    if ((unsigned)j >= (unsigned)a.n_tiles) return -1;
    return frame_row(a.f, j, s);
  }
  const int r = (c - p.img_chunks) * KC + kk;
  return r < a.f.n_text ? r : -1;
}

// Validity of the 64 keys of chunk c as a bit mask (uniform across the group).
template <int TILE_LOG2>
__device__ __forceinline__ uint64_t chunk_mask(const Plan& p, const AttnArgs& a, int c) {
  constexpr int SLOTS = 1 << (2 * TILE_LOG2);
  int end;
  if (p.natural_end) {
    end = p.natural_end - c * KC;
  } else if (c < p.img_chunks) {
    if constexpr (SLOTS >= KC) {
      const int j = p.list[1 + c / (SLOTS / KC)];
      return ((unsigned)j < (unsigned)a.n_tiles) ? ~0ull : 0ull;
    } else {
      uint64_t m = 0;
      for (int q = 0; q < KC / SLOTS; ++q) {
        const int e = c * (KC / SLOTS) + q;
        if (e < p.count && (unsigned)p.list[1 + e] < (unsigned)a.n_tiles)
          m |= ((1ull << SLOTS) - 1) << (q * SLOTS);
      }
      return m;
    }
  } else {
    end = a.f.n_text - (c - p.img_chunks) * KC;
  }
  return end >= KC ? ~0ull : ((1ull << end) - 1);
}

template <int D, int TILE_LOG2>
struct Stage {
  uint4 kr[Cfg<D, TILE_LOG2>::KP];
  uint2 vr[Cfg<D, TILE_LOG2>::VG][4];
};

template <int D, int TILE_LOG2>
__device__ __forceinline__ void fetch(Stage<D, TILE_LOG2>& st, const Plan& p, const AttnArgs& a,
                                      const u16* kbase, const u16* vbase, int c) {
  using C = Cfg<D, TILE_LOG2>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < C::KP; ++i) {
    const int pc = tid + C::NT * i;
    const int kk = pc / (D / 8), c8 = pc % (D / 8);
    const int row = key_row<TILE_LOG2>(p, a, c, kk);
    st.kr[i] = row >= 0 ? *reinterpret_cast<const uint4*>(kbase + (int64_t)row * a.st + c8 * 8)
                        : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < C::VG; ++i) {
    const int g = tid + C::NT * i;
    const int kq = g / (D / 4), dq = g % (D / 4);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = key_row<TILE_LOG2>(p, a, c, 4 * kq + r);
      st.vr[i][r] = row >= 0 ? *reinterpret_cast<const uint2*>(vbase + (int64_t)row * a.st + dq * 4)
                             : make_uint2(0, 0);
    }
  }
}

template <int D, int TILE_LOG2>
__device__ __forceinline__ void commit(const Stage<D, TILE_LOG2>& st, u16* buf) {
  using C = Cfg<D, TILE_LOG2>;
  const int tid = threadIdx.x;
  u16* ks = buf;
  u16* vt = buf + C::K_ELEMS;
#pragma unroll
  for (int i = 0; i < C::KP; ++i) {
    const int pc = tid + C::NT * i;
    const int kk = pc / (D / 8), c8 = pc % (D / 8);
    *reinterpret_cast<uint4*>(ks + kk * C::KROW + c8 * 8) = st.kr[i];
  }
#pragma unroll
  for (int i = 0; i < C::VG; ++i) {
    const int g = tid + C::NT * i;
    const int kq = g / (D / 4), dq = g % (D / 4);
    const uint2* r = st.vr[i];
    // 4 keys x 4 channels -> for each channel, its 4 keys side by side.
    const uint32_t c0a = (r[0].x & 0xffffu) | (r[1].x << 16), c0b = (r[2].x & 0xffffu) | (r[3].x << 16);
    const uint32_t c1a = (r[0].x >> 16) | (r[1].x & 0xffff0000u), c1b = (r[2].x >> 16) | (r[3].x & 0xffff0000u);
    const uint32_t c2a = (r[0].y & 0xffffu) | (r[1].y << 16), c2b = (r[2].y & 0xffffu) | (r[3].y << 16);
    const uint32_t c3a = (r[0].y >> 16) | (r[1].y & 0xffff0000u), c3b = (r[2].y >> 16) | (r[3].y & 0xffff0000u);
    u16* dst = vt + (4 * dq) * C::VROW + 4 * kq;
    *reinterpret_cast<uint2*>(dst) = make_uint2(c0a, c0b);
    *reinterpret_cast<uint2*>(dst + C::VROW) = make_uint2(c1a, c1b);
    *reinterpret_cast<uint2*>(dst + 2 * C::VROW) = make_uint2(c2a, c2b);
    *reinterpret_cast<uint2*>(dst + 3 * C::VROW) = make_uint2(c3a, c3b);
  }
}

__device__ __forceinline__ float xmax4(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}
__device__ __forceinline__ float xsum4(float v) {
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(u16, a) | ((uint32_t)__builtin_bit_cast(u16, b) << 16);
}

template <int D, int TILE_LOG2>
__global__ void __launch_bounds__(threads_of<TILE_LOG2>())
k_attn_bf16(AttnArgs a) {
  using C = Cfg<D, TILE_LOG2>;
  __shared__ __attribute__((aligned(16))) u16 lds[2 * C::BUF];

  // XCD-aware placement: consecutive hardware workgroup ids go to the 8 XCDs
  // in turn; give each XCD a contiguous range of logical groups so the groups
  // of one (batch, head) share that XCD's L2.
  const int nwg = gridDim.x, bid = blockIdx.x;
  const int xcd = bid & 7, slot = bid >> 3;
  const int per = nwg >> 3, rem = nwg & 7;
  const int L = xcd * per + min(xcd, rem) + slot;

  const int bh = L / a.groups_per_bh;
  const int r = L - bh * a.groups_per_bh;
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t off = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const u16* qbase = static_cast<const u16*>(a.q) + off;
  const u16* kbase = static_cast<const u16*>(a.k) + off;
  const u16* vbase = static_cast<const u16*>(a.v) + off;
  u16* obase = static_cast<u16*>(a.o) + off;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 15, lg = lane >> 4;

  Plan p;
  int qrow;  // this lane's query row (-1: none)
  if (a.dense || r < a.n_text_groups) {
    const int end = a.dense ? a.seq : a.f.n_text;
    const int q = r * C::QR + wave * 16 + lq;
    qrow = q < end ? q : -1;
    p.list = nullptr;
    p.count = 0;
    p.img_chunks = 0;
    p.natural_end = a.seq;
    p.n_chunks = (a.seq + KC - 1) / KC;
  } else {
    const int ir = r - a.n_text_groups;
    const int i = ir / a.groups_per_tile, part = ir - i * a.groups_per_tile;
    qrow = frame_row(a.f, i, part * C::QR + wave * 16 + lq);
    p.list = a.index + (bh * (int64_t)a.n_tiles + i) * (a.n_tiles + 1);
    p.count = min(max(p.list[0], 0), a.n_tiles);
    if constexpr (C::SLOTS >= KC)
      p.img_chunks = p.count * (C::SLOTS / KC);
    else
      p.img_chunks = (p.count + (KC / C::SLOTS) - 1) / (KC / C::SLOTS);
    p.natural_end = 0;
    p.n_chunks = p.img_chunks + (a.f.n_text + KC - 1) / KC;
  }

  // Q^T operand: query lq, channels 8 * lg + 32 * ks + [0, 8).
  bf16x8 qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    if (qrow >= 0)
      qf[ks] = *reinterpret_cast<const bf16x8*>(qbase + (int64_t)qrow * a.st + 32 * ks + 8 * lg);
    else
      qf[ks] = bf16x8{};
  }

  floatx4 oacc[D / 16];
#pragma unroll
  for (int db = 0; db < D / 16; ++db) oacc[db] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -1e30f, l_run = 0.f;
  const float c2 = a.scale_log2;

  Stage<D, TILE_LOG2> stg;
  if (p.n_chunks > 0) {
    fetch<D, TILE_LOG2>(stg, p, a, kbase, vbase, 0);
    commit<D, TILE_LOG2>(stg, lds);
  }
  __syncthreads();

  for (int c = 0; c < p.n_chunks; ++c) {
    const bool more = c + 1 < p.n_chunks;
    if (more) fetch<D, TILE_LOG2>(stg, p, a, kbase, vbase, c + 1);
    const u16* ks_l = lds + (c & 1) * C::BUF;
    const u16* vt_l = ks_l + C::K_ELEMS;

    // S^T = K . Q^T : 4 key blocks of 16.
    floatx4 st[KC / 16];
#pragma unroll
    for (int kb = 0; kb < KC / 16; ++kb) {
      st[kb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks_l + (16 * kb + lq) * C::KROW + 32 * ks + 8 * lg);
        st[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], st[kb], 0, 0, 0);
      }
    }
    const uint64_t vmask = chunk_mask<TILE_LOG2>(p, a, c);
    if (vmask != ~0ull) {
#pragma unroll
      for (int kb = 0; kb < KC / 16; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!((vmask >> (16 * kb + 4 * lg + e)) & 1ull)) st[kb][e] = -INFINITY;
    }

    // Online softmax (log2 domain).
    float mx = st[0][0];
#pragma unroll
    for (int kb = 0; kb < KC / 16; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = fmaxf(mx, st[kb][e]);
    mx = xmax4(mx) * c2;
    const bool grow = mx > m_run + kRescaleSlack;
    if (__any(grow)) {
      const float m_new = grow ? mx : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < D / 16; ++db) oacc[db] *= alpha;
    }
    float ps = 0.f;
    uint32_t pk[KC / 16][2];
#pragma unroll
    for (int kb = 0; kb < KC / 16; ++kb) {
      float pv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pv[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[kb][e], c2, -m_run));
        ps += pv[e];
      }
      pk[kb][0] = pack_bf16x2(pv[0], pv[1]);
      pk[kb][1] = pack_bf16x2(pv[2], pv[3]);
    }
    l_run += ps;

    // O^T += V^T . P^T : D / 16 channel blocks x 2 key steps of 32.
#pragma unroll
    for (int kstep = 0; kstep < KC / 32; ++kstep) {
      bf16x8 pf;
      {
        uint4 u = make_uint4(pk[2 * kstep][0], pk[2 * kstep][1], pk[2 * kstep + 1][0], pk[2 * kstep + 1][1]);
        pf = __builtin_bit_cast(bf16x8, u);
      }
#pragma unroll
      for (int db = 0; db < D / 16; ++db) {
        const u16* vrow = vt_l + (16 * db + lq) * C::VROW + 32 * kstep + 4 * lg;
        const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
        const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
        const bf16x8 vf = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
        oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, oacc[db], 0, 0, 0);
      }
    }

    if (more) commit<D, TILE_LOG2>(stg, lds + ((c + 1) & 1) * C::BUF);
    __syncthreads();
  }

  const float l = xsum4(l_run);
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  if (qrow >= 0) {
    u16* orow = obase + (int64_t)qrow * a.st;
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
      const uint2 w = make_uint2(pack_bf16x2(oacc[db][0] * inv, oacc[db][1] * inv),
                                 pack_bf16x2(oacc[db][2] * inv, oacc[db][3] * inv));
      *reinterpret_cast<uint2*>(orow + 16 * db + 4 * lg) = w;
    }
  }
}

template <int D, int TILE_LOG2>
hipError_t launch_t(const AttnArgs& a0, hipStream_t s) {
  using C = Cfg<D, TILE_LOG2>;
  AttnArgs a = a0;
  const int bh = a.batch * a.heads;
  if (a.dense) {
    a.n_text_groups = 0;
    a.groups_per_tile = 1;
    a.groups_per_bh = (a.seq + C::QR - 1) / C::QR;
  } else {
    a.n_text_groups = (a.f.n_text + C::QR - 1) / C::QR;
    a.groups_per_tile = C::SLOTS / C::QR;
    a.groups_per_bh = a.n_text_groups + a.n_tiles * a.groups_per_tile;
  }
  const int64_t total = (int64_t)bh * a.groups_per_bh;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_attn_bf16<D, TILE_LOG2>), dim3((unsigned)total), dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, int tile, hipStream_t s) {
  if (mfma_supported(head_dim, tile, a.dense != 0, a.n_tiles, a.seq, (int64_t)a.seq * a.st))
    return launch_attn_mfma(a, head_dim, tile, s);
  if (head_dim == 64) {
    if (tile == 4) return launch_t<64, 2>(a, s);
    if (tile == 8) return launch_t<64, 3>(a, s);
    return launch_t<64, 4>(a, s);
  }
  if (tile == 4) return launch_t<128, 2>(a, s);
  if (tile == 8) return launch_t<128, 3>(a, s);
  return launch_t<128, 4>(a, s);
}

}  // namespace ssba
