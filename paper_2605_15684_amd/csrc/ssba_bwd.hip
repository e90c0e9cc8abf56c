// SSBA attention backward (gradients of Algorithm 1's attend step with the
// gate held fixed, i.e. through the same kept lists): for the masked softmax
// P = softmax(scale Q K^T + mask) and the upstream gradient dO,
//   D = rowsum(dO * O),  dV = P^T dO,  dP = dO V^T,  dS = P * (dP - D),
//   dQ = scale dS K,  dK = scale dS^T Q,
// with P recomputed from the forward's per-row log-sum-exp.
//
// Kernels (bf16 tensors, 8x8 or 16x16 blocks, head_dim 64 / 128, at most 64
// blocks).  Work goes in chunks of 64 rows: an 8x8 block, or a quarter (four
// block rows) of a 16x16 block; an image chunk is named by block * GPB +
// quarter (GPB = chunks per block), a text chunk t by -1 - t.
//   k_bwd_dq        query side, like the forward: a 64-query group forms D and
//                   the log-sum-exp in log2 units of its rows and the 64-bit
//                   mask of its kept blocks (all stored for the key side),
//                   then walks the chunks of its kept key blocks and the text
//                   keys;
//   k_bwd_dkdv      key side: a 64-key group reads the head's masks, ballots
//                   the query blocks that kept its block (ascending) and walks
//                   their chunks plus the text queries (text key groups:
//                   every query).
// Both main kernels use v_mfma_f32_32x32x16_bf16 with four waves per group:
// two row halves of the group x two streams over each 64-row chunk of the
// other side, merged once at the end.  Chunks are copied into LDS with
// buffer_load ... lds in a row layout whose swizzle is conflict-free both for
// 16-byte row reads and for ds_read_b64_tr_b16 transposed reads, so one copy
// serves both operand orientations.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssba_common.h"

namespace ssba {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kWaitVm0 = 0x0F70;          // s_waitcnt: every vector memory operation done
constexpr int kRawBufferFlags = 0x00020000;
constexpr float kLog2e = 1.4426950408889634f;

template <int D>
struct BShape {
  static constexpr int CPR = D / 8;            // 16-byte chunks per row
  static constexpr int ROWB = 2 * D;           // bytes per row
  static constexpr int KPI = 1024 / ROWB;      // rows per copy instruction
  static constexpr int NI = 32 / KPI;          // copy instructions per 32-row half
  static constexpr int NIW = NI / 2;           // ... per wave (two waves share a half)
  static constexpr int HALF = 32 * ROWB;       // bytes of a half tile
  static constexpr int NKS = D / 16;           // 16-channel steps of a row product
  static constexpr int NDB = D / 32;           // 32-channel output tiles
};

// Physical 16-byte chunk of logical chunk c in row k (0..31) of a half tile.
// Chosen (by exhaustive search over XOR maps of the row bits) so that both the
// 16-byte row reads of 32 rows at one chunk and the transposed 8-byte reads of
// four rows x four channel quads hit distinct banks.
template <int D>
__device__ __forceinline__ int swz(int k, int c) {
  if constexpr (D == 64)
    return c ^ ((4 * ((k >> 1) & 1)) ^ ((k >> 2) & 1) ^ (2 * ((k >> 3) & 1)));
  else
    return c ^ ((4 * (k & 1)) ^ (8 * ((k >> 1) & 1)) ^ ((k >> 2) & 1) ^ (2 * ((k >> 3) & 1)));
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

// Row operand of a 32x32x16 product from a half tile: row l % 32, logical
// chunk 2 ks + l / 32 (eight consecutive channels).
template <int D>
__device__ __forceinline__ bf16x8 row_frag(const char* half, int lane, int ks) {
  const int k = lane & 31, c = 2 * ks + (lane >> 5);
  return *reinterpret_cast<const bf16x8*>(half + k * BShape<D>::ROWB + 16 * swz<D>(k, c));
}

// Transposed operand (channels x rows) of a 32x32x16 product from a half
// tile: 32 channels 32 db + (lane % 32) ... as the hardware transposing read
// lays them out, over rows 16 ks + 8 (e / 4) + 4 (lane / 32) + e % 4.
template <int D>
__device__ __forceinline__ s16x8 tr_frag(const char* half, int lane, int ks, int db) {
  const int G = lane >> 4, li = lane & 15, hw = lane >> 5;
  const int ch = 32 * db + 16 * (G & 1) + 4 * (li & 3);
  const int c = ch >> 3, off = 2 * (ch & 7);
  s16x4 x[2];
#pragma unroll
  for (int rr = 0; rr < 2; ++rr) {
    const int k = 16 * ks + 8 * rr + 4 * hw + (li >> 2);
    x[rr] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4*)(half + k * BShape<D>::ROWB + 16 * swz<D>(k, c) + off));
  }
  return s16x8{x[0][0], x[0][1], x[0][2], x[0][3], x[1][0], x[1][1], x[1][2], x[1][3]};
}

// B operand from registers: P^T / dS^T rows 16 ks + 8 (e / 4) + 4 (lane / 32) + e % 4.
__device__ __forceinline__ bf16x8 packed_frag(const uint32_t (&pk)[8], int ks) {
  return __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
}

// Sum of v over lanes l and l ^ 32 (the swap returns both halves' values).
__device__ __forceinline__ float swap_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sequence row of row s (0..63) of chunk `src`: image chunk src = block * GPB
// + quarter of the shifted frame (GPB = 1 << QL chunks per block), or text
// chunk -1 - src (rows 64 c ..), clamped into the text rows; `valid` is false
// for clamped rows.
template <int QL>
__device__ __forceinline__ int chunk_row(const Frame& f, int src, int s, bool& valid) {
  if (src >= 0) {
    valid = true;
    return frame_row(f, src >> QL, 64 * (src & ((1 << QL) - 1)) + s);
  }
  const int r = 64 * (-1 - src) + s;
  valid = r < f.n_text;
  return valid ? r : f.n_text - 1;
}

// Copies of a half tile: two waves share a half, sub = 0 / 1 selecting NIW
// of its NI copy instructions.  Lane l of instruction m fills row
// k = KPI m + l / CPR of the half, physical chunk l % CPR, i.e. the logical
// chunk that the swizzle puts there; zoff[mm] is that chunk's byte offset
// (a per-lane constant).
template <int D>
__device__ __forceinline__ void swizzle_offsets(int sub, int lane, unsigned (&zoff)[BShape<D>::NIW]) {
  using S = BShape<D>;
  const int kin = lane / S::CPR, pch = lane % S::CPR;
#pragma unroll
  for (int mm = 0; mm < S::NIW; ++mm) {
    const int k = S::KPI * (S::NIW * sub + mm) + kin;
    zoff[mm] = 16u * (unsigned)swz<D>(k, pch);   // swz is an involution on the chunk bits
  }
}

// Byte offsets, inside the (batch, head) slice, of this wave's copy
// instructions for half `hf` of chunk `src` (image chunk block * GPB +
// quarter of a 2^TL x 2^TL block, or text chunk -1 - src with rows past the
// text clamped to its last row).  The block origin is found once per chunk;
// an instruction's rows lie in one block row (KPI <= 2^TL), so only the
// column depends on the lane.
template <int D, int TL>
__device__ __forceinline__ void copy_offsets(const Frame& f, int src, int hf, int sub, unsigned st2,
                                             const unsigned (&zoff)[BShape<D>::NIW],
                                             unsigned (&off)[BShape<D>::NIW]) {
  using S = BShape<D>;
  constexpr int TILE = 1 << TL, QL = 2 * TL - 6;
  static_assert(S::KPI <= TILE && TILE % S::KPI == 0, "an instruction stays inside one block row");
  // The lane's row in an instruction, recomputed here from the lane id (two
  // VALU instructions) rather than kept live across the chunk loop.
  int ln = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  asm volatile("" : "+v"(ln));
  const int kin = ln / S::CPR;
  if (src >= 0) {
    const int blk = src >> QL, quarter = src & ((1 << QL) - 1);
    const int ty = blk / f.nx, tx = blk - ty * f.nx;
    const int y0 = (ty << TL) - f.sy, x0 = (tx << TL) - f.sx;
#pragma unroll
    for (int mm = 0; mm < S::NIW; ++mm) {
      // first slot of the instruction in the block
      const int slot = 64 * quarter + 32 * hf + S::KPI * (S::NIW * sub + mm);
      int y = y0 + (slot >> TL);
      y += y < 0 ? f.grid_h : 0;
      int x = x0 + (slot & (TILE - 1)) + kin;
      x += x < 0 ? f.grid_w : 0;
      off[mm] = st2 * (unsigned)(f.n_text + y * f.grid_w) + st2 * (unsigned)x + zoff[mm];
    }
  } else {
    const int base = 64 * (-1 - src) + 32 * hf;
#pragma unroll
    for (int mm = 0; mm < S::NIW; ++mm) {
      const int row = min(base + S::KPI * (S::NIW * sub + mm) + kin, f.n_text - 1);
      off[mm] = st2 * (unsigned)row + zoff[mm];
    }
  }
}

// This wave's share of the copy of a half tile from the tensor behind `rs`
// into `dst` (the half tile's LDS base), at offsets from copy_offsets.
template <int D>
__device__ __forceinline__ void copy_half(const __amdgpu_buffer_rsrc_t& rs, const unsigned* off, int sub, char* dst) {
  using S = BShape<D>;
#pragma unroll
  for (int mm = 0; mm < S::NIW; ++mm)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + 1024 * (S::NIW * sub + mm)), 16, off[mm], 0, 0, 0);
}

// One float per chunk row (the log-sum-exp or D of the 64 rows) into LDS.
template <int QL>
__device__ __forceinline__ void copy_rowvals(const __amdgpu_buffer_rsrc_t& rs, const Frame& f, int src,
                                             float* dst, int lane) {
  bool valid;
  const int row = chunk_row<QL>(f, src, lane, valid);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 4, 4u * (unsigned)row, 0, 0, 0);
}

// The key-side kernel's order of work for head bh: its key blocks sorted by
// the number of query blocks that keep them (descending, ties by block id),
// written to korder[bh][rank].  A key block's workgroup loops over exactly
// those query blocks, so with the groups dispatched in this order the longest
// start first and the short ones fill the slots that free up (longest-first
// list scheduling); the results do not depend on the order.  All four waves
// of one workgroup take part (the call is workgroup-uniform); `cnt` is 64
// ints of LDS that no wave reads or writes meanwhile.  The lists come from
// the index, complete before the backward starts.
__device__ __forceinline__ void write_key_order(const BwdArgs& a, int bh, int w, int lane, int* cnt) {
  const int tb = a.n_tiles;   // <= 64
  const int32_t* head = a.index + (int64_t)bh * tb * (tb + 1);
  constexpr int LPW = 16;     // lists per wave: wave w takes lists w, w + 4, ...
  // Every load is issued before any is used: lane i holds list i's length,
  // lane e entry e of each of the wave's lists.
  const int len = lane < tb ? head[(int64_t)lane * (tb + 1)] : 0;
  int e[LPW];
#pragma unroll
  for (int u = 0; u < LPW; ++u) {
    const int i = w + 4 * u;
    e[u] = i < tb && lane < tb ? head[(int64_t)i * (tb + 1) + 1 + lane] : -1;
  }
  if (w == 0) cnt[lane] = 0;
  __syncthreads();
#pragma unroll
  for (int u = 0; u < LPW; ++u) {
    const int i = w + 4 * u;
    const int n = i < tb ? min(max(__builtin_amdgcn_readlane(len, i), 0), tb) : 0;
    if (lane < n && (unsigned)e[u] < (unsigned)tb) atomicAdd(&cnt[e[u]], 1);
  }
  __syncthreads();
  if (w == 0 && lane < tb) {
    const int mine = cnt[lane];
    int rank = 0;
    for (int j = 0; j < tb; ++j) {
      const int c = cnt[j];
      rank += (c > mine || (c == mine && j < lane)) ? 1 : 0;
    }
    a.korder[(int64_t)bh * tb + rank] = lane;
  }
}

// Workgroup -> (b, h, group): every (b, h) owns n_text_groups text groups and
// n_tiles << QL image groups (one per chunk of every block); with a head count
// divisible by 8 each XCD (hardware ids go round-robin over the 8) gets whole
// heads, text groups first.
// With RANK_MAJOR the image groups are numbered group-major across heads
// (group 0 of every head, then group 1, ...; within each XCD's heads when
// the head count divides by 8, across all heads otherwise), so that the
// launch dispatches group g of those heads before group g + 1 of any.
template <int QL, bool RANK_MAJOR = false>
__device__ __forceinline__ void group_of(const BwdArgs& a, int& bh, int& r) {
  const int n_img = a.n_tiles << QL;
  const int bid = blockIdx.x, nbh = a.batch * a.heads, gpb = a.n_text_groups + n_img;
  if ((nbh & 7) == 0) {
    const int xcd = bid & 7, s = bid >> 3, hpx = nbh >> 3;
    const int nt = a.n_text_groups;
    if (s < hpx * nt) {
      bh = xcd * hpx + s / nt;
      r = s % nt;
    } else {
      const int s2 = s - hpx * nt;
      bh = xcd * hpx + (RANK_MAJOR ? s2 % hpx : s2 / n_img);
      r = nt + (RANK_MAJOR ? s2 / hpx : s2 % n_img);
    }
  } else if (RANK_MAJOR && bid >= nbh * a.n_text_groups) {
    const int s2 = bid - nbh * a.n_text_groups;
    bh = s2 % nbh;
    r = a.n_text_groups + s2 / nbh;
  } else if (RANK_MAJOR) {
    bh = bid / a.n_text_groups;
    r = bid - bh * a.n_text_groups;
  } else {
    bh = bid / gpb;
    r = bid - bh * gpb;
  }
}

// --------------------------------------------------------------------------
// dQ: one workgroup per 64-query group.  Wave w: query half qh = w % 2, key
// stream sk = w / 2 (keys 32 sk .. 32 sk + 31 of every 64-key chunk).
// Per chunk: S^T = K Q'^T - lse2 (Q' = Q scale log2 e rounded to bf16, as in
// the forward), P^T = exp2(S^T), dP^T = V dO^T, dS^T = P^T (dP^T - D),
// dQ^T += K^T dS^T.
// --------------------------------------------------------------------------
template <int D, int TL>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 2))) k_bwd_dq(BwdArgs a) {
  using S = BShape<D>;
  constexpr int HALF = S::HALF, NKS = S::NKS, NDB = S::NDB;
  constexpr int QL = 2 * TL - 6, GPB = 1 << QL;   // chunks (64-row groups) per block
  // K and V buffers A and B (alternate chunks; stream s at byte HALF s).
  // Separate variables, each named statically by every access, so that the
  // compiler can tell a read of one chunk from the copy of the next in flight.
  __shared__ __attribute__((aligned(16))) char kA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char kB[2 * HALF];
  __shared__ __attribute__((aligned(16))) char vA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char vB[2 * HALF];
  int bh, r;
  group_of<QL>(a, bh, r);
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t off = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const u16* qbase = static_cast<const u16*>(a.q) + off;
  const u16* kbase = static_cast<const u16*>(a.k) + off;
  const u16* vbase = static_cast<const u16*>(a.v) + off;
  const u16* gbase = static_cast<const u16*>(a.dout) + off;
  const int st = (int)a.st;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int qh = w & 1, sk = w >> 1, hw = lane >> 5, l32 = lane & 31;

  // This lane's query row and the chunk plan.  An image group is chunk gq of
  // query block qi.
  const bool text_group = r < a.n_text_groups;
  const int g = r - a.n_text_groups, qi = g >> QL, gq = g & (GPB - 1);
  int qrow;
  if (text_group) {
    const int q = 64 * r + 32 * qh + l32;
    qrow = q < a.f.n_text ? q : -1;
  } else {
    qrow = frame_row(a.f, qi, 64 * gq + 32 * qh + l32);
  }
  const int qr = max(qrow, 0);
  // Chunks: text groups see every key (the text chunks, then every image
  // chunk in block order); image groups the chunks of their kept blocks,
  // then the text.
  const int n_txt = (a.f.n_text + 63) / 64;
  int n_img, listv = -1;
  if (text_group) {
    n_img = a.n_tiles << QL;
  } else {
    const int32_t* list = a.index + ((int64_t)bh * a.n_tiles + qi) * (a.n_tiles + 1);
    const int raw = list[0];
    const int ent = lane < a.n_tiles ? list[1 + lane] : 0;
    const int n_blk = min(max(raw, 0), a.n_tiles);
    listv = lane < n_blk ? ent : -1;
    if ((unsigned)listv >= (unsigned)a.n_tiles) listv = -1;
    n_img = n_blk << QL;
  }
  const int n = n_img + n_txt;
  // Chunk c -> source: image chunks first (block id * GPB + quarter;
  // -1000000 marks an invalid id), then text chunk -1 - t.
  auto src_of = [&](int c) {
    if (c < n_img) {
      if (text_group) return c;
      const int j = __builtin_amdgcn_readlane(listv, c >> QL);
      return j >= 0 ? (j << QL) + (c & (GPB - 1)) : -1000000;   // invalid id: masked (rows of chunk 0)
    }
    return -1 - (c - n_img);
  };

  // Q' (scaled, rounded) and dO as B operands, lse2 and D of the lane's query.
  bf16x8 qf[NKS], gf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const bf16x8 raw = *reinterpret_cast<const bf16x8*>(qbase + (int64_t)qr * st + 16 * ks + 8 * hw);
    qf[ks] = __builtin_convertvector(__builtin_convertvector(raw, floatx8) * a.scale_log2, bf16x8);
    gf[ks] = *reinterpret_cast<const bf16x8*>(gbase + (int64_t)qr * st + 16 * ks + 8 * hw);
  }
  // D = rowsum(dO * O) of the lane's query (its 8 NKS channels here, the
  // other half in lane ^ 32) and the log-sum-exp in log2 units; both are
  // written for the key-side kernel, which runs after this one.
  const int64_t rowid = (int64_t)bh * a.seq + qr;
  const float lse2 = a.lse[rowid] * kLog2e;
  float dlt;
  {
    const u16* obase = static_cast<const u16*>(a.o) + off;
    float part = 0.f;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint4 x = *reinterpret_cast<const uint4*>(obase + (int64_t)qr * st + 16 * ks + 8 * hw);
      const uint4 y = __builtin_bit_cast(uint4, gf[ks]);
      const uint32_t xs[4] = {x.x, x.y, x.z, x.w}, ys[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        part += __uint_as_float(xs[e] << 16) * __uint_as_float(ys[e] << 16);
        part += __uint_as_float(xs[e] & 0xFFFF0000u) * __uint_as_float(ys[e] & 0xFFFF0000u);
      }
    }
    dlt = swap_sum(part);
  }
  if (sk == 0 && hw == 0 && qrow >= 0) {
    a.delta[rowid] = dlt;
    a.lse2[rowid] = lse2;
  }
  // dO fragments are read from LDS per chunk rather than held in registers
  // (four waves per SIMD at D 64 need <= 128 VGPRs): fragment ks of query
  // half qh at gstage + 1024 (NKS qh + ks), lane l's 16 bytes at 16 l, so the
  // reads are linear.  Written by the stream-0 waves, read after the first
  // barrier.
  __shared__ __attribute__((aligned(16))) char gstage[2 * NKS * 1024];
  if (sk == 0) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      *reinterpret_cast<bf16x8*>(gstage + 1024 * (NKS * qh + ks) + 16 * lane) = gf[ks];
  }
  const char* gfr = gstage + 1024 * NKS * qh + 16 * lane;
  const float nlse = -lse2, ndlt = -dlt;

  const unsigned slice_bytes = 2u * (unsigned)((a.seq - 1) * st + D);
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(kbase), (short)0, (int)slice_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(vbase), (short)0, (int)slice_bytes, kRawBufferFlags);

  unsigned zoff[S::NIW];
  swizzle_offsets<D>(qh, lane, zoff);
  auto issue = [&](int c, char* kd, char* vd) {
    const int src = src_of(c);
    unsigned offs[S::NIW];
    copy_offsets<D, TL>(a.f, src == -1000000 ? 0 : src, sk, qh, 2u * (unsigned)st, zoff, offs);
    copy_half<D>(rk, offs, qh, kd + HALF * sk);
    copy_half<D>(rv, offs, qh, vd + HALF * sk);
  };

  floatx16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = floatx16{};

  if (n > 0) issue(0, kA, vA);
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  // The kept blocks of an image block as a 64-bit mask, for the key side
  // (stored by the block's first group; the ids are wave-uniform reads).
  if (!text_group && gq == 0 && w == 0) {
    uint64_t kept = 0ull;
    for (int e = 0; e < (n_img >> QL); ++e) {
      const int j = __builtin_amdgcn_readlane(listv, e);
      if (j >= 0) kept |= 1ull << j;
    }
    if (lane == 0) a.kmask[(int64_t)bh * a.n_tiles + qi] = kept;
  }
  // Chunk c from (kc, vc) while chunk c + 1 is copied into (kn, vn).
  auto body = [&](int c, const char* kc, const char* vc, char* kn, char* vn) {
    if (c + 1 < n) issue(c + 1, kn, vn);
    const char* kt = kc + HALF * sk;
    const char* vt = vc + HALF * sk;
    // Valid keys of this stream's half: text chunks end at n_text.
    const int src = src_of(c);
    int lo = 0, hi = 32;
    if (src == -1000000) {
      hi = 0;
    } else if (src < 0) {
      const int base = 64 * (-1 - src) + 32 * sk;
      hi = min(max(a.f.n_text - base, 0), 32);
    }
    // The score accumulator starts from -lse2 and dP's from -D (so the
    // products leave exp2's argument and dP - D); the splats are rebuilt per
    // chunk from one register each instead of being held across the loop.
    float nl = nlse, nd = ndlt;
    asm volatile("" : "+v"(nl), "+v"(nd));
    floatx16 sc, dp;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      sc[e] = nl;
      dp[e] = nd;
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<D>(kt, lane, ks), qf[ks], sc, 0, 0, 0);
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<D>(vt, lane, ks),
                                                  *reinterpret_cast<const bf16x8*>(gfr + 1024 * ks), dp, 0, 0, 0);
    }
    if (lo > 0 || hi < 32) {   // rare: text tail or an invalid block id
      int l4 = lo - 4 * hw, h4 = hi - 4 * hw;
      asm volatile("" : "+v"(l4), "+v"(h4));
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int key = 8 * (rr >> 2) + (rr & 3);   // minus 4 * hw
        if (key < l4 || key >= h4) sc[rr] = -INFINITY;   // P = 0, so dS = 0 (dP is finite)
      }
    }
    uint32_t pk[8];
#pragma unroll
    for (int rr = 0; rr < 16; rr += 2) {
      float ds[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) ds[u] = __builtin_amdgcn_exp2f(sc[rr + u]) * dp[rr + u];
      pk[rr >> 1] = pack2(ds[0], ds[1]);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 pb = packed_frag(pk, ks);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, tr_frag<D>(kt, lane, ks, db)),
                                                         pb, acc[db], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
  };
  for (int c = 0; c < n; c += 2) {
    body(c, kA, vA, kB, vB);
    if (c + 1 < n) body(c + 1, kB, vB, kA, vA);
  }

  // Merge the two key streams through LDS (the K buffers are free now):
  // query half qh uses buffer A or B.
  float* xo = reinterpret_cast<float*>(qh ? kB : kA);
  static_assert(16 * NDB * 64 * 4 <= 2 * HALF, "merge area fits one K buffer");
  if (sk == 1) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) xo[(16 * db + j) * 64 + lane] = acc[db][j];
  }
  __syncthreads();
  if (sk == 0 && qrow >= 0) {
    u16* orow = static_cast<u16*>(a.dq) + off + (int64_t)qrow * st;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (acc[db][4 * j + e] + xo[(16 * db + 4 * j + e) * 64 + lane]) * a.scale;
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j + 4 * hw) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
      }
  }
  // The first image group of each head also orders the key-side work (the dO
  // stage is free after the chunk loop).
  if (!text_group && g == 0) write_key_order(a, bh, w, lane, reinterpret_cast<int*>(gstage));
}

// --------------------------------------------------------------------------
// dK, dV: one workgroup per 64-key group.  Wave w: key half kh = w % 2, query
// stream qs = w / 2 (queries 32 qs .. 32 qs + 31 of every 64-query chunk).
// Per chunk: S' = Q K'^T - lse2 (rows = queries; K' = K scale log2 e rounded
// to bf16), P = exp2(S'), dV^T += dO^T P, dP - D = dO V^T - D, dS = P (dP - D),
// dK^T += Q^T dS.  The two accumulators start from -lse2 and -D (row values
// read from LDS into them), so no per-element row values stay in registers.
// K' and V of the group are B operands read from LDS per chunk (fragment
// order, linear reads) rather than held in registers; at D 128 the chunk
// buffers are single (the next chunk is copied after every wave is done with
// the current one) so that two workgroups fit a CU, each one's copies then
// overlapping the other's products.
// --------------------------------------------------------------------------
template <int D, int TL>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2))) k_bwd_dkdv(BwdArgs a) {
  using S = BShape<D>;
  constexpr int HALF = S::HALF, NKS = S::NKS, NDB = S::NDB;
  constexpr int QL = 2 * TL - 6, GPB = 1 << QL;   // chunks (64-row groups) per block
  constexpr bool kSingle = D == 128;
  // Q, dO, lse2 and D buffers A and B (alternate chunks; query stream s of
  // Q / dO at byte HALF s), separate variables as in k_bwd_dq; B unused
  // (minimal) when single-buffered.
  __shared__ __attribute__((aligned(16))) char qA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char qB[kSingle ? 16 : 2 * HALF];
  __shared__ __attribute__((aligned(16))) char gA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char gB[kSingle ? 16 : 2 * HALF];
  __shared__ __attribute__((aligned(16))) float lA[64];   // lse2 of the chunk's rows
  __shared__ __attribute__((aligned(16))) float lB[kSingle ? 4 : 64];
  __shared__ __attribute__((aligned(16))) float dA[64];   // D of the chunk's rows
  __shared__ __attribute__((aligned(16))) float dB[kSingle ? 4 : 64];
  // K' and V fragments: fragment ks of key half kh at 1024 (NKS kh + ks),
  // lane l's 16 bytes at 16 l.
  __shared__ __attribute__((aligned(16))) char kst[2 * NKS * 1024];
  __shared__ __attribute__((aligned(16))) char vst[2 * NKS * 1024];
  int bh, r;
  group_of<QL, true>(a, bh, r);
  const int b = bh / a.heads, h = bh - b * a.heads;
  const int64_t off = (int64_t)b * a.sb + (int64_t)h * a.sh;
  const u16* qbase = static_cast<const u16*>(a.q) + off;
  const u16* kbase = static_cast<const u16*>(a.k) + off;
  const u16* vbase = static_cast<const u16*>(a.v) + off;
  const u16* gbase = static_cast<const u16*>(a.dout) + off;
  const int st = (int)a.st;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kh = w & 1, qs = w >> 1, hw = lane >> 5, l32 = lane & 31;
  const int tb = a.n_tiles;

  const bool text_group = r < a.n_text_groups;
  const int g = r - a.n_text_groups, kq = g & (GPB - 1);
  const uint64_t mask_i = lane < tb ? a.kmask[(int64_t)bh * tb + lane] : 0ull;   // query block i's kept set
  // Image group g serves the key block of rank g >> QL in the head's
  // longest-first order (written by the query-side kernel).
  const int kj = text_group ? 0 : a.korder[(int64_t)bh * tb + (g >> QL)];

  // This lane's key row.  An image group is chunk kq of key block kj.
  int krow;
  if (text_group) {
    const int kk = 64 * r + 32 * kh + l32;
    krow = kk < a.f.n_text ? kk : -1;
  } else {
    krow = frame_row(a.f, kj, 64 * kq + 32 * kh + l32);
  }
  const int kr = max(krow, 0);
  // Query chunks: the chunks of the query blocks that kept this key block
  // (text key groups: every block), then the text query chunks.
  const int n_txt = (a.f.n_text + 63) / 64;
  int n_img;
  uint64_t members = 0;   // bit i: query block i kept this key block
  if (text_group) {
    n_img = a.n_tiles << QL;
  } else {
    members = __ballot(((mask_i >> kj) & 1ull) != 0ull);
    n_img = __popcll(members) << QL;
  }
  const int n = n_img + n_txt;
  // Sources in chunk order: the chunks of the member query blocks ascending
  // (text key groups: every chunk), then text chunk -1 - t.  Taken once
  // each, when the chunk's copy is issued.
  uint64_t rest = members;
  int next_img = 0, next_txt = 0, cur = 0;
  auto pop_src = [&]() {
    if (next_img < n_img) {
      const int qc = next_img++ & (GPB - 1);
      if (text_group) return (next_img - 1);
      if (qc == 0) {   // next member block
        cur = (int)__builtin_ctzll(rest);
        rest &= rest - 1ull;
      }
      return (cur << QL) + qc;
    }
    return -1 - next_txt++;
  };

  // K' (scaled, rounded) and V rows of the lane's key into LDS (stream-0
  // waves; read after the first barrier).
  if (qs == 0) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x8 kraw = *reinterpret_cast<const bf16x8*>(kbase + (int64_t)kr * st + 16 * ks + 8 * hw);
      const bf16x8 vraw = *reinterpret_cast<const bf16x8*>(vbase + (int64_t)kr * st + 16 * ks + 8 * hw);
      *reinterpret_cast<bf16x8*>(kst + 1024 * (NKS * kh + ks) + 16 * lane) =
          __builtin_convertvector(__builtin_convertvector(kraw, floatx8) * a.scale_log2, bf16x8);
      *reinterpret_cast<bf16x8*>(vst + 1024 * (NKS * kh + ks) + 16 * lane) = vraw;
    }
  }
  const char* kfr = kst + 1024 * NKS * kh + 16 * lane;
  const char* vfr = vst + 1024 * NKS * kh + 16 * lane;

  const unsigned slice_bytes = 2u * (unsigned)((a.seq - 1) * st + D);
  const __amdgpu_buffer_rsrc_t rq =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(qbase), (short)0, (int)slice_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rg =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(gbase), (short)0, (int)slice_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.lse2 + (int64_t)bh * a.seq), (short)0, 4 * a.seq, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rdl = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.delta + (int64_t)bh * a.seq), (short)0, 4 * a.seq, kRawBufferFlags);

  unsigned zoff[S::NIW];
  swizzle_offsets<D>(kh, lane, zoff);
  auto issue = [&](int src, char* qd, char* gd, float* ld, float* dd) {
    unsigned offs[S::NIW];
    copy_offsets<D, TL>(a.f, src, qs, kh, 2u * (unsigned)st, zoff, offs);
    copy_half<D>(rq, offs, kh, qd + HALF * qs);
    copy_half<D>(rg, offs, kh, gd + HALF * qs);
    if (w == 0) copy_rowvals<QL>(rl, a.f, src, ld, lane);
    if (w == 1) copy_rowvals<QL>(rdl, a.f, src, dd, lane);
  };

  floatx16 dk[NDB], dv[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    dk[db] = floatx16{};
    dv[db] = floatx16{};
  }

  int src = n > 0 ? pop_src() : 0;
  if (n > 0) issue(src, qA, gA, lA, dA);
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  // The products of one chunk from the buffers (qc, gc, lc, dc).
  auto compute = [&](const char* qc, const char* gc, const float* lc, const float* dc) {
    const char* qt = qc + HALF * qs;
    const char* gt = gc + HALF * qs;
    // Valid queries of this stream's half (text chunks end at n_text).
    int hi = 32;
    if (src < 0) hi = min(max(a.f.n_text - (64 * (-1 - src) + 32 * qs), 0), 32);
    // Accumulators seeded with the row values: element e of the lane's tile
    // is query 8 (e / 4) + 4 hw + e % 4.
    floatx16 sc, dp;
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      const float4 x = *reinterpret_cast<const float4*>(&lc[32 * qs + 8 * gg + 4 * hw]);
      const float4 y = *reinterpret_cast<const float4*>(&dc[32 * qs + 8 * gg + 4 * hw]);
      sc[4 * gg] = -x.x; sc[4 * gg + 1] = -x.y; sc[4 * gg + 2] = -x.z; sc[4 * gg + 3] = -x.w;
      dp[4 * gg] = -y.x; dp[4 * gg + 1] = -y.y; dp[4 * gg + 2] = -y.z; dp[4 * gg + 3] = -y.w;
    }
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<D>(qt, lane, ks),
                                                   *reinterpret_cast<const bf16x8*>(kfr + 1024 * ks), sc, 0, 0, 0);
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag<D>(gt, lane, ks),
                                                   *reinterpret_cast<const bf16x8*>(vfr + 1024 * ks), dp, 0, 0, 0);
    }
    if (hi < 32) {   // rare: text tail
      int h4 = hi - 4 * hw;
      asm volatile("" : "+v"(h4));
#pragma unroll
      for (int rr = 0; rr < 16; ++rr)
        if (8 * (rr >> 2) + (rr & 3) >= h4) sc[rr] = -INFINITY;   // P = 0, so dS = 0
    }
    uint32_t pp[8], pd[8];
#pragma unroll
    for (int rr = 0; rr < 16; rr += 2) {
      float pr[2], ds[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        pr[u] = __builtin_amdgcn_exp2f(sc[rr + u]);
        ds[u] = pr[u] * dp[rr + u];
      }
      pp[rr >> 1] = pack2(pr[0], pr[1]);
      pd[rr >> 1] = pack2(ds[0], ds[1]);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 pb = packed_frag(pp, ks), db8 = packed_frag(pd, ks);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        dv[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, tr_frag<D>(gt, lane, ks, db)),
                                                        pb, dv[db], 0, 0, 0);
        dk[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, tr_frag<D>(qt, lane, ks, db)),
                                                        db8, dk[db], 0, 0, 0);
      }
    }
  };
  if constexpr (kSingle) {
    // Chunk c, then (every wave past it) the copy of chunk c + 1 into the
    // same buffers.
    for (int c = 0; c < n; ++c) {
      compute(qA, gA, lA, dA);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      if (c + 1 < n) {
        src = pop_src();
        issue(src, qA, gA, lA, dA);
      }
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      __syncthreads();
    }
  } else {
    // Chunk c from one buffer set while chunk c + 1 is copied into the other.
    auto body = [&](int c, const char* qc, const char* gc, const float* lc, const float* dc,
                    char* qn, char* gn, float* ln, float* dn) {
      const int nsrc = c + 1 < n ? pop_src() : 0;
      if (c + 1 < n) issue(nsrc, qn, gn, ln, dn);
      compute(qc, gc, lc, dc);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(kWaitVm0);
      __syncthreads();
      src = nsrc;
    };
    for (int c = 0; c < n; c += 2) {
      body(c, qA, gA, lA, dA, qB, gB, lB, dB);
      if (c + 1 < n) body(c + 1, qB, gB, lB, dB, qA, gA, lA, dA);
    }
  }

  // Merge the two query streams through LDS (every buffer is free now): key
  // half 0 uses the Q and dO chunk buffers, key half 1 the K' and V ones.
  static_assert(16 * NDB * 64 * 4 <= 2 * HALF && 16 * NDB * 64 * 4 <= 2 * NKS * 1024,
                "merge area fits the buffers");
  float* xk = reinterpret_cast<float*>(kh ? kst : qA);
  float* xv = reinterpret_cast<float*>(kh ? vst : gA);
  if (qs == 1) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        xk[(16 * db + j) * 64 + lane] = dk[db][j];
        xv[(16 * db + j) * 64 + lane] = dv[db][j];
      }
  }
  __syncthreads();
  if (qs == 1 || krow < 0) return;
  u16* krow_k = static_cast<u16*>(a.dk) + off + (int64_t)krow * st;
  u16* krow_v = static_cast<u16*>(a.dv) + off + (int64_t)krow * st;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float vk[4], vv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int x = (16 * db + 4 * j + e) * 64 + lane;
        vk[e] = (dk[db][4 * j + e] + xk[x]) * a.scale;
        vv[e] = dv[db][4 * j + e] + xv[x];
      }
      *reinterpret_cast<uint2*>(krow_k + 32 * db + 8 * j + 4 * hw) = make_uint2(pack2(vk[0], vk[1]), pack2(vk[2], vk[3]));
      *reinterpret_cast<uint2*>(krow_v + 32 * db + 8 * j + 4 * hw) = make_uint2(pack2(vv[0], vv[1]), pack2(vv[2], vv[3]));
    }
}

}  // namespace

hipError_t launch_backward(const BwdArgs& a0, int head_dim, hipStream_t s) {
  BwdArgs a = a0;
  a.n_text_groups = (a.f.n_text + 63) / 64;
  const int tl = a.f.tile_log2;
  if ((head_dim != 64 && head_dim != 128) || (tl != 3 && tl != 4)) return hipErrorInvalidValue;
  const dim3 blk(256);
  const int gpb = 1 << (2 * tl - 6);
  const dim3 grid((unsigned)(a.batch * a.heads * (a.n_text_groups + a.n_tiles * gpb)));
  if (head_dim == 64 && tl == 3) {
    hipLaunchKernelGGL((k_bwd_dq<64, 3>), grid, blk, 0, s, a);
    hipLaunchKernelGGL((k_bwd_dkdv<64, 3>), grid, blk, 0, s, a);
  } else if (head_dim == 64) {
    hipLaunchKernelGGL((k_bwd_dq<64, 4>), grid, blk, 0, s, a);
    hipLaunchKernelGGL((k_bwd_dkdv<64, 4>), grid, blk, 0, s, a);
  } else if (tl == 3) {
    hipLaunchKernelGGL((k_bwd_dq<128, 3>), grid, blk, 0, s, a);
    hipLaunchKernelGGL((k_bwd_dkdv<128, 3>), grid, blk, 0, s, a);
  } else {
    hipLaunchKernelGGL((k_bwd_dq<128, 4>), grid, blk, 0, s, a);
    hipLaunchKernelGGL((k_bwd_dkdv<128, 4>), grid, blk, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ssba
