// SSBA attention forward, bf16, head_dim 64 or 128, 8x8- or 16x16-token
// blocks: 64 query rows per workgroup.
//
// Computes the attend step of Algorithm 1 (image queries of a block attend to
// the image keys of its kept blocks and to every text key; text queries, and
// every query in the dense control, attend to every key in natural order)
// like the generic kernel; it differs only in how data reaches the matrix
// cores.
//
// At head_dim 64 the softmax of a block pair costs as many VALU cycles as its
// two products cost MFMA cycles; at 128 the products dominate.  The kernel:
//   * four waves own 64 query rows (one 8x8 block, or a quarter of a 16x16
//     block): wave w takes queries 32 (w % 2) .. + 31 and the keys
//     32 (w / 2) .. + 31 of every 64-key chunk; the two key streams are merged
//     once at the end;
//   * every 32-key half chunk of K and V is copied once per workgroup, by DMA
//     (buffer_load_dwordx4 ... lds; the two waves of a stream split it), into
//     double-buffered LDS.  Row offsets are scalar operands and the per-lane
//     part is one VGPR per copy instruction and chunk, so a copy costs almost
//     no vector ALU work (every row is a grid row by construction: kept block
//     ids are range-checked before use);
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
// In S^T the lane holds, for its query, the keys 8 (r / 4) + 4 hw + r % 4 of
// the half chunk.  The 16-key step ks of P V contracts keys
// 16 ks + 8 (e / 4) + 4 hw + e % 4 for element e: exactly the lane's own
// probabilities, so P^T never leaves its registers.
//
// LDS tiles hold 32 keys of 2 D bytes; 16-byte column chunks are permuted
// per key so that the DMA writes, the K operand reads (ds_read_b128, 16
// consecutive keys at one logical chunk) and the V transposing reads (4 keys
// x 64 bytes per half wave) spread evenly over the 64 banks:
//   K, D 64:  chunk c of key k at c ^ ((k >> 1) & 7)   (two keys per 256 B)
//   K, D 128: chunk c of key k at c ^ (k & 15)
//   V, D 64:  chunk c of key k at c ^ (4 ((k >> 1) & 1))
//   V, D 128: chunk c of key k at c ^ (4 (k & 3))
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
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint16_t u16;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int KC = 64;                 // keys per chunk
constexpr int KH = 32;                 // keys per stream and chunk
constexpr float kSumLimit = 1048576.0f;   // 2^20: redo a chunk above this lane sum
// s_waitcnt immediate (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8): every vector memory operation done.
constexpr int kWaitVm0 = 0x0F70;
// Buffer resource word 3 for raw (unformatted, unswizzled) dword access.
constexpr int kRawBufferFlags = 0x00020000;

template <int D, int TILE_LOG2>
struct Shape {
  static constexpr int BT = 1 << TILE_LOG2;        // block side (tokens)
  static constexpr int CPR = D / 8;                // 16-byte chunks per key row
  static constexpr int ROWB = 2 * D;               // bytes per key row
  static constexpr int KPI = 1024 / ROWB;          // keys per copy instruction
  static constexpr int NI = KH / KPI;              // copy instructions per half chunk
  static constexpr int NIW = NI / 2;               // ... per wave
  static constexpr int HALF = KH * ROWB;           // bytes of a half chunk tile
  static constexpr int CPB = BT * BT / KC;         // chunks per kept block
  static constexpr int GPB = BT * BT / 64;         // 64-query groups per block
  static constexpr int NKS = D / 16;               // 16-channel steps of Q K^T
  static constexpr int NDB = D / 32;               // 32-channel tiles of O
  static_assert(KPI <= BT, "a copy instruction stays inside one block row");
  static_assert(NIW <= 4, "copy instructions per wave fit a Chunk");
};

// Where one workgroup's keys come from.
struct Plan {
  int img_chunks;    // leading chunks drawn from kept blocks
  int n_chunks;      // total chunks
  int natural_end;   // > 0: keys are rows [0, natural_end) in order
};

// Copy addresses of this stream's half of one chunk, for copy instruction
// m = NIW * (wave % 2) + mm (NIW <= 4): element row row0 + rstep * ((KPI m) / BT)
// (+ wrap when the block row lies above the grid) and per-lane byte offset
// lane_off[mm] within that row, relative to the (batch, head) slice.  Keys
// outside [lo, hi) of the half are masked.  (A plain struct: with a
// per-shape template the host compiler drops the kernels' launch stubs.)
struct Chunk {
  int row0, rstep, y0;
  unsigned lane_off[4];
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

// Q^T operand of one query row: fragment ks holds channels 16 ks + 8 hw + [0, 8).
template <int NKS>
__device__ __forceinline__ void load_q(bf16x8 (&qf)[NKS], const u16* qbase, int qrow, int st, int hw) {
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qbase + max(qrow, 0) * st + 16 * ks + 8 * hw);
}

// Q^T operands scaled by softmax scale * log2(e) and rounded to bf16 (round
// to nearest even), so a product Q K^T is already the exponent of exp2.
template <int NKS>
__device__ __forceinline__ void scale_q(bf16x8 (&qf)[NKS], float c2) {
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = __builtin_convertvector(__builtin_convertvector(qf[ks], floatx8) * c2, bf16x8);
}

// Kept block ids of the current workgroup's gate, ascending (gated launches).
__shared__ int gate_list[64];

// Affinity of one query block with key block `lane` (Eq. 2 on pooled sums):
// the channel-ordered fp64 sum of the rounded products qsum[c] * kb[c][lane],
// from the head's pooled key sums copied contiguously into the four buffers
// (channel row c of T_b values in buffer c / (D/4)).  STRIDE = 64 gives every
// read a constant offset; 0 reads with the runtime row length tb.  Lanes past
// tb read a neighbouring row and are discarded by the caller.  At D 64 the
// pooled query sum of channel c is taken from lane c's `qreg` (the wave that
// formed it) as a scalar operand, which leaves one LDS read per channel.
template <int D, int STRIDE>
__device__ __forceinline__ double affinity(const double* qsum, const char* b0, const char* b1,
                                           const char* b2, const char* b3, int lane, int tb, double qreg) {
  constexpr int CPQ = D / 4;
  const int row = STRIDE ? STRIDE : tb;
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < D; ++c) {
    const int qi = c / CPQ, cc = c % CPQ;
    const char* src = qi == 0 ? b0 : qi == 1 ? b1 : qi == 2 ? b2 : b3;
    const double kv = reinterpret_cast<const double*>(src)[cc * row + lane];
    double qc;
    if constexpr (D == 64) {
      const uint64_t qbits = (uint64_t)__double_as_longlong(qreg);
      const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)qbits, c);
      const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(qbits >> 32), c);
      qc = __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
    } else {
      qc = qsum[c];
    }
    const double p = __dmul_rn(qc, kv);
    s = (c == 0) ? p : __dadd_rn(s, p);
  }
  return s;
}

// Top-k gate of query block i inside a gated launch (Section 2.2.1, Block
// Compression / Affinity Matrix / Top-k Gating; Algorithm 1 pool, affinity and
// top-k steps), with the arithmetic of the separate gate kernels so the index
// rows are bit-identical to theirs:
//   1. the head's pooled key sums [D][T_b] (written by the pooling pre-pass of
//      the same call) are copied into the four K/V buffers (a quarter of the
//      channels each; they are free until the first chunk is copied);
//   2. the block's pooled query sum (Eq. 1) is formed here from the Q
//      fragments the workgroup already holds: the two waves that hold the
//      block's 64 query rows (slots 0-31 and 32-63) stage them through LDS,
//      32 rows at a time, and thread c < D adds channel c of the slots in
//      slot order in fp64 -- the pooling kernel's order and arithmetic
//      (bf16 -> fp32 is exact), so the sum is the same to the bit;
//   3. wave 0, lane j < T_b: S[i][j] = sum over channels, in order, of the
//      rounded products; then the wave's radix select picks the keep largest.
// Writes the index row and status flag of block i; returns the kept count
// with the ids in gate_list.  Every wave of the workgroup calls it.
template <int D, int NKS>
__device__ __forceinline__ int gate_block(const AttnArgs& a, int bh, int i, int w, int lane, const bf16x8 (&qf)[NKS],
                                          char* b0, char* b1, char* b2, char* b3) {
  __shared__ double qsum[D];
  // 32 query rows, each padded by 16 bytes so that the 16-byte writes of
  // consecutive rows start on different banks.
  constexpr int QROW = 2 * D + 16;
  __shared__ __attribute__((aligned(16))) char qstage[32 * QROW];
  const int tb = a.n_tiles;
  const int quarter_bytes = 2 * D * tb;   // D * tb * 8 / 4
  // 1. pooled key sums of this (batch, head): wave w copies quarter w.
  {
    // The whole offset goes in the range-checked lane operand: bytes past the
    // head's slice (a partial last copy) read as zeros.
    const double* kbh = a.kb + (int64_t)bh * D * tb;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<double*>(kbh), (short)0, 4 * quarter_bytes, 0x00020000);
    char* dst = w == 0 ? b0 : w == 1 ? b1 : w == 2 ? b2 : b3;
    for (int o = 0; o < quarter_bytes; o += 1024)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(dst + o), 16,
                                               (unsigned)(w * quarter_bytes + o + 16 * lane), 0u, 0, 0);
  }
  // 2. pooled query sum of block i: channel c = thread id, slots in order.
  const int tid = 64 * w + lane;
  __builtin_amdgcn_s_waitcnt(0x0F70);   // the Q fragments and the copies have landed
  double qacc = 0.0;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (w == half) {   // wave half (key stream 0) holds slots 32 half .. 32 half + 31
      const int row = lane & 31, hw = lane >> 5;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        *reinterpret_cast<bf16x8*>(qstage + row * QROW + 32 * ks + 16 * hw) = qf[ks];
    }
    __syncthreads();
    if (tid < D) {
      float xs[32];
#pragma unroll
      for (int r = 0; r < 32; ++r)
        xs[r] = __uint_as_float((uint32_t)*reinterpret_cast<const uint16_t*>(qstage + r * QROW + 2 * tid) << 16);
#pragma unroll
      for (int r = 0; r < 32; ++r) qacc = (half == 0 && r == 0) ? (double)xs[r] : __dadd_rn(qacc, (double)xs[r]);
    }
    __syncthreads();
  }
  if (tid < D) qsum[tid] = qacc;
  __syncthreads();
  // 3. affinity row and ranking (wave 0).
  if (w == 0) {
    const bool valid = lane < tb;
    const double s = tb == 64 ? affinity<D, 64>(qsum, b0, b1, b2, b3, lane, tb, qacc)
                              : affinity<D, 0>(qsum, b0, b1, b2, b3, lane, tb, qacc);
    const uint64_t key = valid ? rank_key(s) : 0;
    const bool kept = wave_topk(key, valid, a.keep, lane);
    const uint64_t km = __builtin_amdgcn_ballot_w64(kept);
    const int pos = __popcll(km & ((1ull << lane) - 1ull));
    const bool bad = __builtin_amdgcn_ballot_w64(valid && !isfinite(s)) != 0;
    int32_t* out = a.index_out + ((int64_t)bh * tb + i) * (tb + 1);
    if (valid) {
      if (kept) {
        gate_list[pos] = lane;
        out[1 + pos] = lane;
      }
      if (lane >= a.keep) out[1 + lane] = -1;
    }
    if (lane == 0) {
      out[0] = a.keep;
      a.flags[(int64_t)bh * tb + i] = bad ? 1 : 0;
    }
  }
  // The list is published, and every wave is past the pooled sums before
  // the first chunk is copied over them.
  __syncthreads();
  return a.keep;
}

// DENSE: every group runs natural-order rows over all keys (no index).
// GATED: each image group computes its block's top-k gate first (from the
// pooled key sums) and writes the block's index row and status flag.
template <int D, int TILE_LOG2, bool DENSE, bool GATED>
__device__ __forceinline__ void attn_mfma_body(const AttnArgs& a) {
  using S = Shape<D, TILE_LOG2>;
  constexpr int BT = S::BT, CPR = S::CPR, KPI = S::KPI, NIW = S::NIW, HALF = S::HALF;
  constexpr int CPB = S::CPB, GPB = S::GPB, NKS = S::NKS, NDB = S::NDB;

  // K and V buffers A and B (alternate chunks); stream s uses bytes
  // [HALF s, HALF (s + 1)) of each.  Declared separately so every access
  // names one buffer statically: the compiler can then tell that a read of
  // one chunk does not overlap the copy of the next still in flight.
  __shared__ __attribute__((aligned(16))) char kA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char kB[2 * HALF];
  // D 128 without the gate keeps one V buffer (48 KiB in all, three
  // workgroups per CU): chunk c + 1's V is copied once every wave is past
  // chunk c's products, under chunk c + 1's scores and softmax.  The gated
  // kernel needs all four buffers for the pooled key sums.
  constexpr bool kSingleV = D == 128 && !GATED;
  __shared__ __attribute__((aligned(16))) char vA[2 * HALF];
  __shared__ __attribute__((aligned(16))) char vB[kSingleV ? 16 : 2 * HALF];

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
  bf16x8 qf[NKS];   // Q^T operand [ks]: query 32 qh + l32, channels 16 ks + 8 hw + [0, 8)
  int listv = -1;   // lane e holds kept block id number e (image groups)
  if (DENSE || r < a.n_text_groups) {   // natural order: text rows, or every row
    const int end = DENSE ? a.seq : a.f.n_text;
    const int q = r * 64 + 32 * qh + l32;
    qrow = q < end ? q : -1;
    load_q<NKS>(qf, qbase, qrow, st, hw);
    p.img_chunks = 0;
    p.natural_end = a.seq;
    p.n_chunks = (a.seq + KC - 1) / KC;
  } else {
    const int g = r - a.n_text_groups;     // image group: block i, quarter gq
    const int i = g / GPB, gq = g - i * GPB;
    qrow = frame_row(a.f, i, 64 * gq + 32 * qh + l32);
    load_q<NKS>(qf, qbase, qrow, st, hw);   // in flight during the gate or the list read
    int count, e;
    if constexpr (GATED) {
      count = gate_block<D, NKS>(a, bh, i, w, lane, qf, kA, kB, vA, vB);
      e = lane < count ? gate_list[lane] : 0;
    } else {
      // The count and the entries are requested together (one round trip).
      const int32_t* list = a.index + (bh * (int64_t)a.n_tiles + i) * (a.n_tiles + 1);
      const int raw = list[0];
      const int ent = lane < a.n_tiles ? list[1 + lane] : 0;
      count = min(max(raw, 0), min(a.n_tiles, 64));
      e = lane < count ? ent : 0;
    }
    listv = (unsigned)e < (unsigned)a.n_tiles ? e : -1;
    p.img_chunks = CPB * count;
    p.natural_end = 0;
    p.n_chunks = p.img_chunks + (a.f.n_text + KC - 1) / KC;
  }

  // Buffer resources over this (batch, head) slice: rows [0, seq).
  const unsigned slice_bytes = 2u * (unsigned)((a.seq - 1) * st + D);
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(kbase), (short)0, (int)slice_bytes, kRawBufferFlags);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<u16*>(vbase), (short)0, (int)slice_bytes, kRawBufferFlags);

  // DMA lane mapping: lane l of copy instruction m fills key KPI m + l / CPR
  // of the half, physical chunk l % CPR; it fetches the logical chunk that
  // the swizzle puts there.  kcol[mm] / vcol: that chunk's byte offset.
  const int kin = lane / CPR, pch = lane % CPR;   // key within the instruction, physical chunk
  unsigned kcol[NIW], vcol;
#pragma unroll
  for (int mm = 0; mm < NIW; ++mm) {
    const int key = KPI * (NIW * qh + mm) + kin;
    const int lc = D == 64 ? (pch ^ ((key >> 1) & 7)) : (pch ^ (key & 15));
    kcol[mm] = 16u * lc;
  }
  {
    const int key = kin;   // the V swizzle depends on key bits that KPI m leaves unchanged
    const int lc = D == 64 ? (pch ^ (4 * ((key >> 1) & 1))) : (pch ^ (4 * (key & 3)));
    vcol = 16u * lc;
  }
  // K operand reads: key l32, logical chunk 2 ks + hw.
  int koff[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const int lc = 2 * ks + hw;
    const int pc = D == 64 ? (lc ^ ((l32 >> 1) & 7)) : (lc ^ (l32 & 15));
    koff[ks] = HALF * sk + l32 * S::ROWB + 16 * pc;
  }
  // V transposing reads: 16-lane group G = lane / 16, i = lane % 16 reads
  // key 16 ks + 8 r' + 4 hw + i / 4 (r' = 0, 1: the two reads of a step),
  // channels 32 db + 16 (G % 2) + 4 (i % 4) .. + 3.
  const int G = lane >> 4, li = lane & 15;
  int voff[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    const int key = 4 * hw + (li >> 2);                 // + 8 r' + 16 ks (swizzle-neutral)
    const int lc = 4 * db + 2 * (G & 1) + ((li & 3) >> 1);
    const int pc = D == 64 ? (lc ^ (4 * ((key >> 1) & 1))) : (lc ^ (4 * (key & 3)));
    voff[db] = HALF * sk + key * S::ROWB + 16 * pc + 8 * (li & 1);
  }

  // Frame origin (y0, x0) of each kept block, one block per lane.
  const int W = a.f.grid_w, H = a.f.grid_h;
  int orig_y = 0, orig_x = 0;
  if (listv >= 0) {
    const int ty = listv / a.f.nx;
    orig_y = ty * BT - a.f.sy;
    orig_x = (listv - ty * a.f.nx) * BT - a.f.sx;
  }

  // This stream's half of chunk c.  Image chunks: block list[c / CPB], block
  // rows (c % CPB) * 64 / BT + sk * 32 / BT onwards; each lane's column wraps
  // to the right edge when it starts left of it.  Natural-order chunks always
  // cover 64 existing rows: a ragged last chunk is moved back to end at the
  // last row and masks the keys the previous chunk already covered (rows of a
  // ragged text chunk that run into the image rows exist too).
  auto chunk_of = [&](int c) {
    Chunk ch;
    if (!DENSE && c < p.img_chunks) {
      const int e = c / CPB, sub = c - e * CPB;
      const int j = __builtin_amdgcn_readlane(listv, e);
      const int x0 = __builtin_amdgcn_readlane(orig_x, e);
      ch.y0 = __builtin_amdgcn_readlane(orig_y, e) + sub * (KC / BT) + sk * (KH / BT);
      ch.row0 = a.f.n_text + ch.y0 * W;
      ch.rstep = W;
#pragma unroll
      for (int mm = 0; mm < NIW; ++mm) {
        const int col = (KPI * (NIW * qh + mm)) % BT + kin;
        const unsigned x = (unsigned)(x0 + col);
        ch.lane_off[mm] = 2u * min(x, x + (unsigned)W) * (unsigned)st;   // x < 0 wraps by W
      }
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
    // Natural rows: instruction m covers rows base + 32 sk + KPI m + [0, KPI).
    ch.row0 = base + KH * sk;
    ch.rstep = BT;   // (KPI m) / BT rows of BT keys: row0 + KPI m after the column term below
    ch.y0 = 0;
#pragma unroll
    for (int mm = 0; mm < NIW; ++mm) {
      const int col = (KPI * (NIW * qh + mm)) % BT + kin;
      ch.lane_off[mm] = 2u * (unsigned)(col * st);
    }
    return ch;
  };
  const int wrap = H * W;

  // This wave's NIW of the NI copy instructions of a half chunk, into its
  // stream's HALF bytes of buffer `dst`.  The LDS base is kept opaque so
  // each instruction's LDS address is one scalar add rather than a held
  // register.
  auto copy = [&](const __amdgpu_buffer_rsrc_t& rs, const Chunk& ch, char* dst, bool is_k) {
    int lb = HALF * sk + 1024 * NIW * qh;
    asm volatile("" : "+s"(lb));
#pragma unroll
    for (int mm = 0; mm < NIW; ++mm) {
      const int m = NIW * qh + mm;
      const int rr = (KPI * m) / BT;   // block row of the instruction within the half
      const int row = ch.row0 + rr * ch.rstep + (ch.y0 + rr < 0 ? wrap : 0);
      const unsigned col = is_k ? kcol[mm] : vcol;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + lb + 1024 * mm), 16,
                                               ch.lane_off[mm] + col, 2u * (unsigned)row * (unsigned)st, 0, 0);
    }
  };

  floatx16 oacc[NDB];   // [db]
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = floatx16{};
  // Softmax state per query (the lane's): running max m_run of the scaled
  // scores (-1e30 until a finite one is seen) and running sum l_run.  The
  // score products start from negm = -m_run (0 while unset), so the common
  // chunk feeds the accumulator straight into exp2.
  float m_run = -1e30f, l_run = 0.f;
  floatx16 negm = floatx16{};   // D 64: the seed of the score products
  float nm = 0.f;               // D 128: -m_run, added after the products (16 fewer VGPRs)
  scale_q<NKS>(qf, a.scale_log2);
  const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};

  // One half chunk: K in kt, V in vt (this stream's halves), keys outside
  // [lo, hi) masked.
  uint32_t pk[8];   // P of the current chunk, bf16 pairs
  auto scores = [&](const char* kt, int lo, int hi) {
    // S^T = K . Q^T: the lane's 16 keys 8 (r / 4) + 4 hw + r % 4 of its query.
    floatx16 sc = D == 64 ? negm : floatx16{};   // sc = s - m_run: the exponent of exp2
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kt + koff[ks]);
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc, 0, 0, 0);
    }
    if constexpr (D != 64) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) sc[rr] += nm;
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
    // P = exp2(sc - shift) as bf16 pairs and the lane's sum of the rounded P
    // (shift is 0 except when a chunk is redone).
    float ls;
    auto probs = [&](float shift, bool shifted) {
      float ls0 = 0.f, ls1 = 0.f;
#pragma unroll
      for (int rr = 0; rr < 16; rr += 2) {
        const float x0 = shifted ? sc[rr] - shift : sc[rr];
        const float x1 = shifted ? sc[rr + 1] - shift : sc[rr + 1];
        pk[rr >> 1] = pack2(__builtin_amdgcn_exp2f(x0), __builtin_amdgcn_exp2f(x1));
        if (rr & 2) ls1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[rr >> 1]), one2, ls1, false);
        else        ls0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[rr >> 1]), one2, ls0, false);
      }
      ls = ls0 + ls1;
    };
    probs(0.f, false);
    // Redo when a lane sum overflows the bound (the max grew) or the lane has
    // no max yet: take the chunk's max, rescale O and l, recompute P.
    if (__any(!(ls <= kSumLimit) || m_run < -1e29f)) {
      float mx = sc[0];
#pragma unroll
      for (int rr = 1; rr < 16; ++rr) mx = fmaxf(mx, sc[rr]);
      const float mb = m_run > -1e29f ? m_run : 0.f;   // the offset in sc
      const float mabs = mb + swap_max(mx);
      if (mabs > m_run) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - mabs);   // 0 while unset
        m_run = mabs;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
      }
      const float mnew = m_run > -1e29f ? m_run : 0.f;
      probs(mnew - mb, true);
      if constexpr (D == 64) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) negm[rr] = -mnew;
      } else {
        nm = -mnew;
      }
    }
    l_run += ls;
  };
  auto values = [&](const char* vt) {
    // O^T[db] += V^T . P^T over 2 key steps of 16 (V^T operands: keys
    // 16 ks + 8 (e / 4) + 4 hw + e % 4, channel 32 db + lane % 32).
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]));
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const s16x4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + voff[db] + 16 * S::ROWB * ks));
        const s16x4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + voff[db] + 16 * S::ROWB * ks + 8 * S::ROWB));
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

  // With the whole grid resident (a.equalize), the workgroups sharing a CU
  // would otherwise run oldest first: the youngest waits and finishes last
  // with the SIMDs to itself.  Waves with more chunks left get the higher
  // issue priority instead, so they finish together.  With more groups than
  // slots the oldest-first order frees slots sooner and stays.
  auto prioritise = [&](int c) {
    if (a.equalize) {
      const int rem = n - c;
      if (rem >= 24) __builtin_amdgcn_s_setprio(3);
      else if (rem >= 8) __builtin_amdgcn_s_setprio(2);
      else if (rem >= 4) __builtin_amdgcn_s_setprio(1);
      else __builtin_amdgcn_s_setprio(0);
    }
  };
  // Chunk c from buffers (kt, vt) while chunk c + 1 is copied into (kn, vn).
  auto body = [&](int c, const char* kt, const char* vt, char* kn, char* vn) {
    prioritise(c);
    const int lo = lo_c, hi = hi_c;
    if (c + 1 < n) {
      const Chunk cn = chunk_of(c + 1);
      copy(rk, cn, kn, true);
      copy(rv, cn, vn, false);
      lo_c = cn.lo;
      hi_c = cn.hi;
    }
    scores(kt, lo, hi);
    values(vt);
    // The products are issued before the wait, so they run during it.
    __builtin_amdgcn_sched_barrier(0);
    // Chunk c + 1 has landed (this wave's part) and every wave is past its
    // reads of chunk c before any starts chunk c + 2 into the same buffers.
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
  };
  // One V buffer: chunk c from (kt, vA) while chunk c + 1's K is copied into
  // kn; chunk c + 1's V follows once every wave is past chunk c's products.
  auto body_single_v = [&](int c, const char* kt, char* kn) {
    prioritise(c);
    const int lo = lo_c, hi = hi_c;
    const bool more = c + 1 < n;
    Chunk cn;
    if (more) {
      cn = chunk_of(c + 1);
      lo_c = cn.lo;
      hi_c = cn.hi;
    } else {
      // No next chunk: the same number of copies through a buffer resource
      // with no records, so every one is out of range (no memory traffic;
      // zeros land in kn, unread) and the wait below counts the same on
      // every path.
      cn.row0 = 0;
      cn.rstep = 0;
      cn.y0 = 0;
#pragma unroll
      for (int mm = 0; mm < NIW; ++mm) cn.lane_off[mm] = 0;
    }
    // (The resource is built here, record count chosen by `more`: a choice
    // between two resource variables would put them in memory.)
    const __amdgpu_buffer_rsrc_t rkn = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u16*>(kbase), (short)0, more ? (int)slice_bytes : 0, kRawBufferFlags);
    copy(rkn, cn, kn, true);
    scores(kt, lo, hi);
    // Chunk c's V (copied before chunk c + 1's K) has landed in every wave.
    __builtin_amdgcn_s_waitcnt(kWaitVm0 | NIW);
    __syncthreads();
    values(vA);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
    if (more) copy(rv, cn, vA, false);
  };
  if constexpr (kSingleV) {
    for (int c = 0; c < n; c += 2) {
      body_single_v(c, kA, kB);
      if (c + 1 < n) body_single_v(c + 1, kB, kA);
    }
  } else {
    for (int c = 0; c < n; c += 2) {
      body(c, kA, vA, kB, vB);
      if (c + 1 < n) body(c + 1, kB, vB, kA, vA);
    }
  }

  // Merge the two key streams: stream 1 leaves (m, l, O) in LDS, stream 0
  // combines and stores.  The K/V buffers are free after the last barrier.
  static_assert(16 * NDB * 64 * 4 <= 2 * HALF, "merge area fits one buffer");
  float* xo = reinterpret_cast<float*>(qh ? kB : kA);   // [16 NDB values][64 lanes]
  float* xml = reinterpret_cast<float*>(vA) + 128 * qh; // [2][64 lanes]
  if (sk == 1) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
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
    m_run = mm;   // l_run is now relative to the merged max
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) oacc[db][j] = oacc[db][j] * a0 + xo[(16 * db + j) * 64 + lane] * a1;
  }

  // Epilogue: O = O^T / l, 4 consecutive channels per store.
  const float l = swap_sum(l_run);
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  if (a.lse && qrow >= 0 && hw == 0)   // m and l are in units of log2: convert to natural log
    a.lse[(int64_t)bh * a.seq + qrow] = (m_run + __builtin_amdgcn_logf(l)) * 0.69314718055994531f;
  if (qrow >= 0) {
    u16* orow = obase + qrow * st;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint2 wv = make_uint2(pack2(oacc[db][4 * j] * inv, oacc[db][4 * j + 1] * inv),
                                    pack2(oacc[db][4 * j + 2] * inv, oacc[db][4 * j + 3] * inv));
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j + 4 * hw) = wv;
      }
  }
}

template <int D, int TILE_LOG2, bool DENSE, bool GATED>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : GATED ? 2 : 3)))
k_attn_mfma(AttnArgs a) {
  attn_mfma_body<D, TILE_LOG2, DENSE, GATED>(a);
}

// Attention of several layers in one launch (grid y = layer): the
// workgroups of layer l + 1 start as those of layer l finish, so one layer's
// tail and the next one's start overlap.  Each workgroup runs exactly what
// it runs in a one-layer launch.
template <int D, int TILE_LOG2, bool GATED>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : GATED ? 2 : 3)))
k_attn_mfma_layers(AttnLayers p) {
  const int l = blockIdx.y;
  AttnArgs a = p.a;
  a.q = p.q[l];
  a.k = p.k[l];
  a.v = p.v[l];
  a.o = p.o[l];
  if constexpr (GATED) {
    a.kb = p.kb[l];
    a.index_out = p.index_out[l];
    a.flags = p.flags[l];
    a.keep = p.keep[l];
  } else {
    a.index = p.index[l];
  }
  a.f = p.f[p.parity[l] & 1];
  attn_mfma_body<D, TILE_LOG2, false, GATED>(a);
}

// Image and text workgroup counts of a launch.
void set_groups(AttnArgs& a, int tile) {
  const int gpb = (tile == 16) ? 4 : 1;   // 64-query groups per image block
  if (a.dense) {
    a.n_text_groups = (a.seq + 63) / 64;    // every group runs natural-order rows
    a.groups_per_tile = 1;
    a.groups_per_bh = a.n_text_groups;
  } else {
    a.n_text_groups = (a.f.n_text + 63) / 64;
    a.groups_per_tile = gpb;
    a.groups_per_bh = a.n_text_groups + a.n_tiles * gpb;
  }
}

}  // namespace

hipError_t launch_attn_mfma_layers(const AttnLayers& p0, int n_layers, int head_dim, int tile, hipStream_t s) {
  const bool gated = p0.a.gated != 0;
  if (n_layers < 1 || n_layers > kAttnLayersMax || p0.a.dense || (head_dim != 64 && head_dim != 128) ||
      (tile != 8 && tile != 16) || (gated && tile != 8) || p0.a.f.tile_log2 != (tile == 8 ? 3 : 4))
    return hipErrorInvalidValue;
  AttnLayers p = p0;
  set_groups(p.a, tile);
  // Several layers never fit the CUs at once: the chunk-count priorities
  // stay off (they only pay when the whole grid is resident).
  p.a.equalize = 0;
  const int64_t per_layer = (int64_t)p.a.batch * p.a.heads * p.a.groups_per_bh;
  if (per_layer <= 0) return hipSuccess;
  const dim3 grid((unsigned)per_layer, (unsigned)n_layers), block(256);
  if (head_dim == 64) {
    if (gated) hipLaunchKernelGGL((k_attn_mfma_layers<64, 3, true>), grid, block, 0, s, p);
    else if (tile == 8) hipLaunchKernelGGL((k_attn_mfma_layers<64, 3, false>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((k_attn_mfma_layers<64, 4, false>), grid, block, 0, s, p);
  } else {
    if (gated) hipLaunchKernelGGL((k_attn_mfma_layers<128, 3, true>), grid, block, 0, s, p);
    else if (tile == 8) hipLaunchKernelGGL((k_attn_mfma_layers<128, 3, false>), grid, block, 0, s, p);
    else hipLaunchKernelGGL((k_attn_mfma_layers<128, 4, false>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_attn_mfma(const AttnArgs& a0, int head_dim, int tile, hipStream_t s) {
  AttnArgs a = a0;
  set_groups(a, tile);
  const int64_t total = (int64_t)a.batch * a.heads * a.groups_per_bh;
  if (total <= 0) return hipSuccess;
  // Resident workgroups per CU: four waves each, four (D 64), three (D 128
  // with one V buffer) or two (gated D 128) waves per SIMD.
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();   // a failed query only leaves the priorities off
    cus = 0;
  }
  const int slots = head_dim == 64 ? 4 : (a.gated && !a.dense) ? 2 : 3;
  a.equalize = cus > 0 && total <= (int64_t)slots * cus ? 1 : 0;
  const dim3 grid((unsigned)total), block(256);
  const bool big = !a.dense && tile == 16;
  if (a.gated && (a.dense || big)) return hipErrorInvalidValue;   // gated: 8x8 blocks only
  if (head_dim == 64) {
    if (a.dense) hipLaunchKernelGGL((k_attn_mfma<64, 3, true, false>), grid, block, 0, s, a);
    else if (a.gated) hipLaunchKernelGGL((k_attn_mfma<64, 3, false, true>), grid, block, 0, s, a);
    else if (big) hipLaunchKernelGGL((k_attn_mfma<64, 4, false, false>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<64, 3, false, false>), grid, block, 0, s, a);
  } else {
    if (a.dense) hipLaunchKernelGGL((k_attn_mfma<128, 3, true, false>), grid, block, 0, s, a);
    else if (a.gated) hipLaunchKernelGGL((k_attn_mfma<128, 3, false, true>), grid, block, 0, s, a);
    else if (big) hipLaunchKernelGGL((k_attn_mfma<128, 4, false, false>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_attn_mfma<128, 3, false, false>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ssba
