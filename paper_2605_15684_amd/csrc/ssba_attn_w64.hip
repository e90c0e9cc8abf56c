// SSBA attention forward, bf16, head_dim 64, 64 query rows per workgroup.
//
// Specialised path for the 1024-px class shapes (8x8-token blocks, so one
// query block is exactly 64 rows) and for natural-order rows (text queries,
// dense control).  Computes the attend step of Algorithm 1 like the generic
// kernel; it differs only in how data reaches the matrix cores.
//
// At head_dim 64 the softmax of a block pair costs as many VALU cycles as its
// two products cost MFMA cycles, so the kernel is built for overlap between
// waves:
//   * a workgroup owns the 64 query rows of one block with four waves: wave w
//     takes queries 32 (w % 2) .. + 31 and the keys 32 (w / 2) .. + 31 of every
//     64-key chunk (one 8x4 half of a kept block), so each SIMD holds four
//     waves; the two key streams are merged once at the end;
//   * every 32-key half chunk of K and V is copied once per workgroup, by DMA
//     (buffer_load_dwordx4 ... lds; the two waves of a stream split it), into
//     double-buffered LDS.  Row offsets are scalar operands and the per-lane
//     part is one VGPR per chunk, so a copy costs almost no vector ALU work.
//     Out-of-range rows read as zeros (the buffer bound is the (batch, head)
//     slice);
//   * the softmax is optimistic: probabilities are taken against the running
//     max; only when a lane's chunk sum exceeds 2^20 (the max grew, or the
//     first chunk) is the chunk max taken, O and l rescaled and the chunk
//     redone, so the common chunk needs no max reduction;
//   * products use v_mfma_f32_32x32x16_bf16 in the transposed orientation
//     (S^T = K Q^T, O^T = V^T P^T), so each lane holds 16 keys of one query
//     and a row max or sum needs one exchange with lane ^ 32
//     (v_permlane32_swap);
//   * V^T operands come straight from the row-major V tile through
//     ds_read_b64_tr_b16, which hands each lane 4 keys of one channel.
//
// Register layouts of v_mfma_f32_32x32x16_bf16 (lane l, hw = l / 32):
//   A[i][k]: lane holds row i = l % 32, k = 8 hw + e  (e = 0..7)
//   B[k][j]: lane holds col j = l % 32, k = 8 hw + e
//   D[i][j]: lane holds col j = l % 32, rows i = 8 (r / 4) + 4 hw + r % 4 (r = 0..15)
// In S^T the lane holds, for its query, the keys 32 kb + 8 (r / 4) + 4 hw + r % 4.
// The 16-key step ks of P V contracts keys 16 ks + 8 (e / 4) + 4 hw + e % 4
// for element e: exactly the lane's own probabilities, so P^T never leaves
// its registers.
//
// LDS tiles are 32 rows (keys) of 128 bytes.  A 16-byte column chunk c of key
// k sits at chunk c ^ ((k >> 1) & 7) in the K tile and c ^ (4 ((k >> 1) & 1))
// in the V tile; with these swizzles the K operand reads (ds_read_b128), the
// V transposing reads and the DMA writes all spread evenly over the banks.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>

#include "ssba_common.h"

namespace ssba {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int D = 64;
constexpr int KC = 64;                 // keys per chunk (one 8x8 block)
constexpr int KH = 32;                 // keys per stream and chunk
constexpr int HALF_BYTES = KH * D * 2; // one K or V half chunk in LDS (4 KB)
constexpr float kSumLimit = 1048576.0f;   // 2^20: redo a chunk above this lane sum
// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8): every vector memory operation done.
constexpr int kWaitVm0 = 0x0F70;
// Buffer resource word 3 for raw (unformatted, unswizzled) dword access.
constexpr int kRawBufferFlags = 0x00020000;

// Where one workgroup's keys come from.
struct Plan {
  int img_chunks;    // leading chunks drawn from kept blocks (8x8 = 64 keys each)
  int n_chunks;      // total chunks
  int natural_end;   // > 0: keys are rows [0, natural_end) in order
};

// Copy addresses of this stream's half of one chunk: copy instruction m
// (0..3; the wave issues two of them) lane l moves key 8 m + l / 8 of the
// half from element row row0 + m * step (+ wrap when y0 + m < 0: a block row
// above the grid wraps to its bottom) and byte lane_off within that row's
// 8-key group, relative to the (batch, head) slice.  Keys outside [lo, hi)
// of the half are masked.
struct Chunk {
  int row0, step, y0;
  unsigned lane_off;
  int lo, hi;
};

__device__ __forceinline__ float swap_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float swap_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Two fp32 -> two bf16 (round to nearest even) in one 32-bit word.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// DENSE: every group runs natural-order rows over all keys (no index).
template <bool DENSE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
k_attn_w64(AttnArgs a) {
  // K and V buffers A and B (alternate chunks); stream s uses bytes
  // [4096 s, 4096 s + 4096) of each.  Declared separately so every access
  // names one buffer statically: the compiler can then tell that a read of
  // one chunk does not overlap the copy of the next still in flight.
  __shared__ __attribute__((aligned(16))) char kA[2 * HALF_BYTES];
  __shared__ __attribute__((aligned(16))) char kB[2 * HALF_BYTES];
  __shared__ __attribute__((aligned(16))) char vA[2 * HALF_BYTES];
  __shared__ __attribute__((aligned(16))) char vB[2 * HALF_BYTES];

  // Logical group id.  Consecutive hardware ids go round-robin over the 8
  // XCDs; when the (batch, head) count divides by 8 each XCD gets whole
  // heads (their K/V stay in its L2), long natural-order groups first.
  const int bid = blockIdx.x;
  int bh, r;
  const int nbh = a.batch * a.heads;
  if ((nbh & 7) == 0) {
    const int xcd = bid & 7, s = bid >> 3;
    const int hpx = nbh >> 3;
    const int n_nat = a.n_text_groups, n_img = a.groups_per_bh - a.n_text_groups;
    if (s < hpx * n_nat) {
      const int d = n_nat > 0 ? n_nat : 1;
      bh = xcd * hpx + s / d;
      r = s % d;
    } else {
      const int s2 = s - hpx * n_nat;
      const int d = n_img > 0 ? n_img : 1;
      bh = xcd * hpx + s2 / d;
      r = n_nat + s2 % d;
    }
  } else {
    bh = bid / a.groups_per_bh;
    r = bid - bh * a.groups_per_bh;
  }
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t off = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const u16* qbase = static_cast<const u16*>(a.q) + off;
  const u16* kbase = static_cast<const u16*>(a.k) + off;
  const u16* vbase = static_cast<const u16*>(a.v) + off;
  u16* obase = static_cast<u16*>(a.o) + off;
  const int st = (int)a.st;

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int qh = w & 1;    // query half
  const int sk = w >> 1;   // key stream: keys 32 sk .. 32 sk + 31 of each chunk
  const int hw = lane >> 5, l32 = lane & 31;

  Plan p;
  int qrow;
  int listv = -1;   // lane e holds kept block id number e (image groups)
  if (DENSE || r < a.n_text_groups) {   // natural order: text rows, or every row
    const int end = DENSE ? a.seq : a.f.n_text;
    const int q = r * 64 + 32 * qh + l32;
    qrow = q < end ? q : -1;
    p.img_chunks = 0;
    p.natural_end = a.seq;
    p.n_chunks = (a.seq + KC - 1) / KC;
  } else {
    const int i = r - a.n_text_groups;
    qrow = frame_row(a.f, i, 32 * qh + l32);
    const int32_t* list = a.index + (bh * (int64_t)a.n_tiles + i) * (a.n_tiles + 1);
    const int count = min(max(list[0], 0), min(a.n_tiles, 64));
    const int e = lane < count ? list[1 + lane] : 0;
    listv = (unsigned)e < (unsigned)a.n_tiles ? e : -1;
    p.img_chunks = count;
    p.natural_end = 0;
    p.n_chunks = p.img_chunks + (a.f.n_text + KC - 1) / KC;
  }

  // Q^T operand [ks]: query 32 qh + l32, channels 16 ks + 8 hw + [0, 8).
  bf16x8 qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qbase + max(qrow, 0) * st + 16 * ks + 8 * hw);

  // Buffer resources over this (batch, head) slice: rows [0, seq).
  const unsigned slice_bytes = 2u * (unsigned)((a.seq - 1) * st + D);
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(kbase), (short)0, (int)slice_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(vbase), (short)0, (int)slice_bytes, kRawBufferFlags);

  // DMA lane mapping: lane l of instruction m fills key 8 m + l / 8 of the
  // half, physical chunk l % 8 -- logical K chunk (l % 8) ^ ((key >> 1) & 7)
  // and logical V chunk (l % 8) ^ (4 ((key >> 1) & 1)), where
  // (key >> 1) & 7 = 4 (m & 1) + l / 16.
  const int vk = lane >> 3;
  const unsigned kc0 = 16u * ((lane & 7) ^ (lane >> 4));          // bytes, m even
  const unsigned kc1 = 16u * ((lane & 7) ^ (4 + (lane >> 4)));    // bytes, m odd
  const unsigned vcb = 16u * ((lane & 7) ^ (4 * ((lane >> 4) & 1)));
  // K operand reads: key l32, logical chunk 2 ks + hw.
  const int g = (l32 >> 1) & 7;
  int koff[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) koff[ks] = HALF_BYTES * sk + l32 * 128 + 16 * ((2 * ks + hw) ^ g);
  // V transposing reads: 16-lane group G = lane / 16, i = lane % 16 points at
  // key 16 ks + 8 r' + 4 hw + i / 4, channels 32 db + 16 (G % 2) + 4 (i % 4).
  const int G = lane >> 4, li = lane & 15;
  int voff[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
    voff[db] = HALF_BYTES * sk + (4 * hw + (li >> 2)) * 128 + 64 * (db ^ ((li >> 3) & 1)) +
               32 * (G & 1) + 8 * (li & 3);

  // Frame origin (y0, x0) of each kept block, one block per lane.
  const int W = a.f.grid_w, H = a.f.grid_h;
  int orig_y = 0, orig_x = 0;
  if (listv >= 0) {
    const int ty = listv / a.f.nx;
    orig_y = ty * 8 - a.f.sy;
    orig_x = (listv - ty * a.f.nx) * 8 - a.f.sx;
  }

  // This stream's half of chunk c.  Image chunks: block rows 4 sk .. 4 sk + 3;
  // each lane's column wraps to the right edge when it starts left of it.
  // Natural-order chunks always cover 64 existing rows: a ragged last chunk
  // is moved back to end at the last row and masks the keys the previous
  // chunk already covered (rows of a ragged text chunk that run into the
  // image rows exist too).
  auto chunk_of = [&](int c) {
    Chunk ch;
    if (!DENSE && c < p.img_chunks) {
      const int j = __builtin_amdgcn_readlane(listv, c);
      const int x0 = __builtin_amdgcn_readlane(orig_x, c);
      ch.y0 = __builtin_amdgcn_readlane(orig_y, c) + 4 * sk;
      ch.row0 = a.f.n_text + ch.y0 * W;
      ch.step = W;
      const unsigned x = (unsigned)(x0 + vk);
      ch.lane_off = 2u * min(x, x + (unsigned)W) * (unsigned)st;   // x < 0 wraps by W
      ch.lo = 0;
      ch.hi = j >= 0 ? KH : 0;
      return ch;
    }
    const int end = p.natural_end ? p.natural_end : a.f.n_text;
    int base = p.natural_end ? c * KC : (c - p.img_chunks) * KC;
    int lo = 0, hi = min(end - base, KC);
    if (hi < KC && end >= KC) {   // ragged last chunk: end it at the last row
      lo = KC - hi;
      hi = KC;
      base = end - KC;
    }
    ch.lo = min(max(lo - KH * sk, 0), KH);
    ch.hi = min(max(hi - KH * sk, 0), KH);
    ch.row0 = base + KH * sk;
    ch.step = 8;
    ch.y0 = 0;
    ch.lane_off = 2u * (unsigned)(vk * st);
    return ch;
  };
  const int wrap = H * W;

  // This wave's two of the four copy instructions of a half chunk, into
  // the stream's 4 KB of buffer `dst`.  The LDS base is kept opaque so each
  // instruction's LDS address is one scalar add rather than a held register.
  auto copy = [&](const __amdgpu_buffer_rsrc_t& rs, const Chunk& ch, char* dst, bool is_k) {
    int lb = HALF_BYTES * sk + 2048 * qh;
    asm volatile("" : "+s"(lb));
#pragma unroll
    for (int mm = 0; mm < 2; ++mm) {
      const int m = 2 * qh + mm;
      const int row = ch.row0 + m * ch.step + (ch.y0 + m < 0 ? wrap : 0);
      const unsigned col = is_k ? ((mm & 1) ? kc1 : kc0) : vcb;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + lb + 1024 * mm), 16,
                                               ch.lane_off + col, 2u * (unsigned)row * (unsigned)st, 0, 0);
    }
  };

  floatx16 oacc[2];   // [db]
  oacc[0] = floatx16{};
  oacc[1] = floatx16{};
  float m_run = -1e30f, l_run = 0.f;
  const float c2 = a.scale_log2;
  const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};

  // One half chunk: K in kt, V in vt (this stream's halves), keys outside
  // [lo, hi) masked.
  auto step = [&](const char* kt, const char* vt, int lo, int hi) {
    // S^T = K . Q^T: the lane's 16 keys 8 (r / 4) + 4 hw + r % 4 of its query.
    floatx16 sc = floatx16{};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kt + koff[ks]);
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc, 0, 0, 0);
    }
    if (lo > 0 || hi < KH) {   // rare: ragged chunk or invalid block id
      int l4 = lo - 4 * hw, h4 = hi - 4 * hw;
      asm volatile("" : "+v"(l4), "+v"(h4));
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int key = 8 * (rr >> 2) + (rr & 3);   // minus 4 * hw
        if (key < l4 || key >= h4) sc[rr] = -INFINITY;
      }
    }
    // P = exp2(c2 S - m) as bf16 pairs and the lane's sum of the rounded P.
    uint32_t pk[8];
    float ls;
    auto probs = [&]() {
      const float mneg = -m_run;
      float ls0 = 0.f, ls1 = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; rr += 2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[rr], c2, mneg));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[rr + 1], c2, mneg));
        pk[rr >> 1] = pack2(p0, p1);
        if (rr & 2) ls1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[rr >> 1]), one2, ls1, false);
        else        ls0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[rr >> 1]), one2, ls0, false);
      }
      ls = ls0 + ls1;
    };
    probs();
    if (__any(!(ls <= kSumLimit))) {   // the max grew (or first chunk): rescale, redo
      float mx = sc[0];
#pragma unroll
      for (int rr = 1; rr < 16; ++rr) mx = fmaxf(mx, sc[rr]);
      mx = swap_max(mx) * c2;
      if (mx > m_run) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - mx);
        m_run = mx;
        l_run *= alpha;
        oacc[0] *= alpha;
        oacc[1] *= alpha;
      }
      probs();
    }
    l_run += ls;
    // O^T[db] += V^T . P^T over 2 key steps of 16 (V^T operands: keys
    // 16 ks + 8 (e / 4) + 4 hw + e % 4, channel 32 db + lane % 32).
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
#pragma unroll
      for (int db = 0; db < 2; ++db) {
        const s16x4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + voff[db] + 2048 * ks));
        const s16x4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + voff[db] + 2048 * ks + 1024));
        const s16x8 v8 = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, v8), pb, oacc[db], 0, 0, 0);
      }
    }
  };

  const int n = p.n_chunks;
  int lo_c = 0, hi_c = 0;
  if (n > 0) {
    const Chunk ch0 = chunk_of(0);
    copy(rk, ch0, kA, true);
    copy(rv, ch0, vA, false);
    lo_c = ch0.lo;
    hi_c = ch0.hi;
  }
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();

  // Chunk c from buffers (kt, vt) while chunk c + 1 is copied into (kn, vn).
  auto body = [&](int c, const char* kt, const char* vt, char* kn, char* vn) {
    const int lo = lo_c, hi = hi_c;
    if (c + 1 < n) {
      const Chunk cn = chunk_of(c + 1);
      copy(rk, cn, kn, true);
      copy(rv, cn, vn, false);
      lo_c = cn.lo;
      hi_c = cn.hi;
    }
    step(kt, vt, lo, hi);
    // Chunk c + 1 has landed (this wave's part) and every wave is past its
    // reads of chunk c before any starts chunk c + 2 into the same buffers.
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
  };
  for (int c = 0; c < n; c += 2) {
    body(c, kA, vA, kB, vB);
    if (c + 1 < n) body(c + 1, kB, vB, kA, vA);
  }

  // Merge the two key streams: stream 1 leaves (m, l, O) in LDS, stream 0
  // combines and stores.  The K/V buffers are free after the last barrier.
  float* xo = reinterpret_cast<float*>(qh ? kB : kA);   // [32 values][64 lanes]
  float* xml = reinterpret_cast<float*>(vA) + 128 * qh; // [2][64 lanes]
  if (sk == 1) {
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) xo[(16 * db + j) * 64 + lane] = oacc[db][j];
    xml[lane] = m_run;
    xml[64 + lane] = l_run;
  }
  __syncthreads();
  if (sk == 1) return;
  {
    const float m1 = xml[lane], l1 = xml[64 + lane];
    const float mm = fmaxf(m_run, m1);
    const float a0 = __builtin_amdgcn_exp2f(m_run - mm), a1 = __builtin_amdgcn_exp2f(m1 - mm);
    l_run = l_run * a0 + l1 * a1;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) oacc[db][j] = oacc[db][j] * a0 + xo[(16 * db + j) * 64 + lane] * a1;
  }

  // Epilogue: O = O^T / l, 4 consecutive channels per store.
  const float l = swap_sum(l_run);
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  if (qrow >= 0) {
    u16* orow = obase + qrow * st;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint2 wv = make_uint2(pack2(oacc[db][4 * j] * inv, oacc[db][4 * j + 1] * inv),
                                    pack2(oacc[db][4 * j + 2] * inv, oacc[db][4 * j + 3] * inv));
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j + 4 * hw) = wv;
      }
  }
}

}  // namespace

const char* w64_kernel_name(bool dense) { return dense ? "k_attn_w64<true>" : "k_attn_w64<false>"; }

bool w64_supported(int head_dim, int tile, bool dense, int n_tiles, int seq, int64_t span) {
  // 32-bit byte offsets inside one (batch, head); at most 64 kept blocks;
  // natural-order chunks need at least one full chunk of rows.
  return head_dim == 64 && (dense || (tile == 8 && n_tiles <= 64)) && seq >= KC &&
         span < ((int64_t)1 << 31);
}

hipError_t launch_attn_w64(const AttnArgs& a0, hipStream_t s) {
  AttnArgs a = a0;
  if (a.dense) {
    a.n_text_groups = (a.seq + 63) / 64;    // every group runs natural-order rows
    a.groups_per_tile = 1;
    a.groups_per_bh = a.n_text_groups;
  } else {
    a.n_text_groups = (a.f.n_text + 63) / 64;
    a.groups_per_tile = 1;
    a.groups_per_bh = a.n_text_groups + a.n_tiles;
  }
  const int64_t total = (int64_t)a.batch * a.heads * a.groups_per_bh;
  if (total <= 0) return hipSuccess;
  if (a.dense)
    hipLaunchKernelGGL(k_attn_w64<true>, dim3((unsigned)total), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_attn_w64<false>, dim3((unsigned)total), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ssba
