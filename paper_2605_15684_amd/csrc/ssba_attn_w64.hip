// SSBA attention forward, bf16, head_dim 64: one wave per 64 query rows.
//
// Specialised path for the 1024-px class shapes (8x8-token blocks, so one
// query block is exactly 64 rows) and for natural-order rows (text queries,
// dense control).  Computes the attend step of Algorithm 1 like the generic
// kernel; it differs only in how data reaches the matrix cores.
//
// At head_dim 64 a 64x64 block pair costs about the same in MFMA cycles,
// softmax VALU cycles and bytes moved, so every byte of K/V is fetched once
// per query block:
//   * a workgroup is one wave that owns all 64 query rows;
//   * K goes from memory straight into MFMA operand registers (no LDS);
//   * V is copied by DMA (global_load_lds_dwordx4) into a per-wave LDS buffer
//     and read back with ds_read_b64_tr_b16, which hands each lane 4 keys of
//     one channel;
//   * products use v_mfma_f32_32x32x16_bf16 in the transposed orientation
//     (S^T = K Q^T, O^T = V^T P^T), so each lane holds 16 keys of one query
//     per 32-key block, and a row max or sum needs one exchange with lane ^ 32;
//   * the next 64-key chunk is in flight while the current one is computed.
//
// Register layouts of v_mfma_f32_32x32x16_bf16 (lane l, hw = l / 32):
//   A[i][k]: lane holds row i = l % 32, k = 8 hw + e  (e = 0..7)
//   B[k][j]: lane holds col j = l % 32, k = 8 hw + e
//   D[i][j]: lane holds col j = l % 32, rows i = 8 (r / 4) + 4 hw + r % 4 (r = 0..15)
// In S^T the lane therefore holds, for query 32 qb + l % 32, the keys
// 32 kb + 8 (r / 4) + 4 hw + r % 4.  The 16-key step ks of P V contracts
// keys 16 ks + 8 (e / 4) + 4 hw + e % 4 for element e: exactly the lane's own
// probabilities, so P^T never leaves its registers.
//
// V tile in LDS: 64 rows (keys) of 128 bytes; 16-byte column chunk c of key k
// sits at chunk c ^ (4 * ((k >> 1) & 1)), which spreads both the DMA writes
// and the transposing reads evenly over the LDS banks.
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

constexpr int D = 64;
constexpr int KC = 64;                 // keys per chunk
constexpr float kRescaleSlack = 8.0f;  // rescale only when the max grows by > 2^8
constexpr int VBUF = KC * D * 2;       // bytes per V buffer (8 KB)
// s_waitcnt immediate (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4, lgkmcnt 11:8): wait for every outstanding vector memory operation,
// leave the other counters alone.
constexpr int kWaitVm0 = 0x0F70;

// Where one wave's keys come from.
struct Plan {
  int img_chunks;    // leading chunks drawn from kept blocks (8x8 = 64 keys each)
  int n_chunks;      // total chunks
  int natural_end;   // > 0: keys are rows [0, natural_end) in order
};

// Element offsets (from the (batch, head) base) of the rows one chunk needs:
// K rows of keys lane % 32 and lane % 32 + 32, and V rows of keys
// 8 m + lane / 8 (m = 0..7).  Absent keys (ragged tails, invalid block ids)
// read a valid row instead; their scores are masked, so they contribute
// exactly zero.
struct Rows {
  int k0, k1;
  int v[8];
};

__device__ __forceinline__ void natural_rows(int base, int end, int st, int lane, Rows& rw) {
  const int kk = lane & 31, vk = lane >> 3;
  const int last = end - 1;
  rw.k0 = min(base + kk, last) * st;
  rw.k1 = min(base + kk + 32, last) * st;
#pragma unroll
  for (int m = 0; m < 8; ++m) rw.v[m] = min(base + 8 * m + vk, last) * st;
}

// The 64 keys of 8x8 block j of the shifted frame, slot s = 8 * sr + sc.
__device__ __forceinline__ void block_rows(const AttnArgs& a, int j, int st, int lane, Rows& rw) {
  const int kk = lane & 31, vk = lane >> 3;
  const int ty = j / a.f.nx, tx = j - ty * a.f.nx;
  const int y0 = ty * 8 - a.f.sy, x0 = tx * 8 - a.f.sx;
  int x = x0 + (kk & 7);
  x += x < 0 ? a.f.grid_w : 0;
  int y = y0 + (kk >> 3), y1 = y + 4;
  y += y < 0 ? a.f.grid_h : 0;
  y1 += y1 < 0 ? a.f.grid_h : 0;
  rw.k0 = (a.f.n_text + y * a.f.grid_w + x) * st;
  rw.k1 = (a.f.n_text + y1 * a.f.grid_w + x) * st;
  int xv = x0 + vk;
  xv += xv < 0 ? a.f.grid_w : 0;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    int ym = y0 + m;
    ym += ym < 0 ? a.f.grid_h : 0;
    rw.v[m] = (a.f.n_text + ym * a.f.grid_w + xv) * st;
  }
}

// Issue one chunk: 8 x 16 B of K into operand registers and 8 x 1 KB of V by
// DMA into `vbuf` (lane l of DMA m fills bytes [16 l, 16 l + 16) of its KB:
// key 8 m + l / 8, physical chunk l % 8).  Always 16 memory instructions.
__device__ __forceinline__ void issue_chunk(bf16x8 (&kr)[2][4], char* vbuf, const u16* kbase,
                                            const u16* vbase, const Rows& rw, int hw, int vcol) {
  const u16* k0 = kbase + rw.k0 + 8 * hw;
  const u16* k1 = kbase + rw.k1 + 8 * hw;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) kr[0][ks] = *reinterpret_cast<const bf16x8*>(k0 + 16 * ks);
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) kr[1][ks] = *reinterpret_cast<const bf16x8*>(k1 + 16 * ks);
#pragma unroll
  for (int m = 0; m < 8; ++m)
    __builtin_amdgcn_global_load_lds(vbase + rw.v[m] + vcol, vbuf + 1024 * m, 16, 0, 0);
}

__device__ __forceinline__ float swap_max(float v) { return fmaxf(v, __shfl_xor(v, 32)); }
__device__ __forceinline__ float swap_sum(float v) { return v + __shfl_xor(v, 32); }

// Two fp32 -> two bf16 (round to nearest even) in one 32-bit word.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{lo, hi}, bf16x2));
}

__global__ void __launch_bounds__(64) k_attn_w64(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char vA[VBUF];
  __shared__ __attribute__((aligned(16))) char vB[VBUF];
  __shared__ __attribute__((aligned(16))) uint4 qlds[8 * 64];   // Q^T operands, [qb * 4 + ks][lane]

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

  const int lane = threadIdx.x;
  const int hw = lane >> 5, l32 = lane & 31;

  Plan p;
  int qrow[2];
  int listv = 0;   // lane e holds kept block id number e (image groups)
  if (r < a.n_text_groups) {   // natural order: text rows, or every row (dense)
    const int end = a.dense ? a.seq : a.f.n_text;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      const int q = r * 64 + 32 * qb + l32;
      qrow[qb] = q < end ? q : -1;
    }
    p.img_chunks = 0;
    p.natural_end = a.seq;
    p.n_chunks = (a.seq + KC - 1) / KC;
  } else {
    const int i = r - a.n_text_groups;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) qrow[qb] = frame_row(a.f, i, 32 * qb + l32);
    const int32_t* list = a.index + (bh * (int64_t)a.n_tiles + i) * (a.n_tiles + 1);
    const int count = min(max(list[0], 0), min(a.n_tiles, 64));
    const int e = lane < count ? list[1 + lane] : 0;
    listv = (unsigned)e < (unsigned)a.n_tiles ? e : -1;
    p.img_chunks = count;
    p.natural_end = 0;
    p.n_chunks = p.img_chunks + (a.f.n_text + KC - 1) / KC;
  }

  // Rows of chunk c; returns how many of its keys (a prefix) are real.
  auto rows_of = [&](int c, Rows& rw) -> int {
    if (c < p.img_chunks) {
      const int j = __builtin_amdgcn_readlane(listv, c);
      block_rows(a, j >= 0 ? j : 0, st, lane, rw);
      return j >= 0 ? KC : 0;
    }
    const int base = p.natural_end ? c * KC : (c - p.img_chunks) * KC;
    const int end = p.natural_end ? p.natural_end : a.f.n_text;
    natural_rows(base, end, st, lane, rw);
    return min(end - base, KC);
  };

  // Q^T operands [qb][ks]: query 32 qb + l32, channels 16 ks + 8 hw + [0, 8).
  // Parked in LDS in operand order (each lane reads back its own 16 bytes), so
  // they do not occupy registers across the key loop.
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      qlds[(qb * 4 + ks) * 64 + lane] =
          *reinterpret_cast<const uint4*>(qbase + max(qrow[qb], 0) * st + 16 * ks + 8 * hw);

  // V copy: lane l of each 1 KB DMA fills key 8 m + l / 8, physical chunk
  // l % 8, which holds logical chunk (l % 8) ^ (4 * ((l >> 4) & 1)).
  const int vcol = 8 * ((lane & 7) ^ (4 * ((lane >> 4) & 1)));
  // Transposing reads: 16-lane group G = lane / 16, i = lane % 16 points at key
  // 16 ks + 8 r' + 4 hw + i / 4, channels 32 db + 16 (G % 2) + 4 (i % 4).
  const int G = lane >> 4, li = lane & 15;
  int roff[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
    roff[db] = (4 * hw + (li >> 2)) * 128 + 64 * (db ^ ((li >> 3) & 1)) + 32 * (G & 1) + 8 * (li & 3);

  floatx16 oacc[2][2];   // [db][qb]
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) oacc[db][qb] = floatx16{};
  float m_run[2] = {-1e30f, -1e30f}, l_run[2] = {0.f, 0.f};
  const float c2 = a.scale_log2;
  const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};

  // Chunk pipeline.  Per chunk c: wait until chunk c has landed (K in `kr`,
  // V in LDS buffer c & 1); read its V operands from LDS; compute S^T for both
  // query halves; then issue chunk c + 1 (K into `kr`, V by DMA into the other
  // buffer) and finish softmax and P V while it is in flight.  Nothing after
  // the issue reads memory, so one wait per chunk is enough.
  bf16x8 kr[2][4];
  int nv_cur = 0;
  if (p.n_chunks > 0) {
    Rows rw;
    nv_cur = rows_of(0, rw);
    issue_chunk(kr, vA, kbase, vbase, rw, hw, vcol);
  }
  for (int c = 0; c < p.n_chunks; ++c) {
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    const char* vc = (c & 1) ? vB : vA;

    // V^T operands [ks][db]: keys 16 ks + 8 (e / 4) + 4 hw + e % 4, channel
    // 32 db + lane % 32.
    bf16x8 vop[4][2];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int db = 0; db < 2; ++db) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vc + roff[db] + 2048 * ks));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vc + roff[db] + 2048 * ks + 1024));
        const s16x8 v8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        vop[ks][db] = __builtin_bit_cast(bf16x8, v8);
      }

    // S^T[qb][kb] = K_kb . Q_qb^T  (keys 32 kb + 8 (r / 4) + 4 hw + r % 4)
    floatx16 sc[2][2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        sc[qb][kb] = floatx16{};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          sc[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              kr[kb][ks], __builtin_bit_cast(bf16x8, qlds[(qb * 4 + ks) * 64 + lane]), sc[qb][kb], 0, 0, 0);
      }

    const int nvc = nv_cur;
    if (c + 1 < p.n_chunks) {
      Rows rw;
      nv_cur = rows_of(c + 1, rw);
      issue_chunk(kr, (c & 1) ? vA : vB, kbase, vbase, rw, hw, vcol);
    }

#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      if (nvc < KC) {   // rare: ragged tail or invalid block id
        int lim = nvc - 4 * hw;
        asm volatile("" : "+v"(lim));
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int rr = 0; rr < 16; ++rr)
            if (32 * kb + 8 * (rr >> 2) + (rr & 3) >= lim) sc[qb][kb][rr] = -INFINITY;
      }
      // Online softmax (log2 domain, lazy rescale).
      float mx = fmaxf(sc[qb][0][0], sc[qb][1][0]);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) mx = fmaxf(mx, sc[qb][kb][rr]);
      mx = swap_max(mx) * c2;
      const bool grow = mx > m_run[qb] + kRescaleSlack;
      if (__any(grow)) {
        const float m_new = grow ? mx : m_run[qb];
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < 2; ++db) oacc[db][qb] *= alpha;
      }
      const float mneg = -m_run[qb];
      uint32_t pk[2][8];   // [kb] bf16 pairs of the lane's 16 probabilities
      float ls0 = 0.f, ls1 = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int rr = 0; rr < 16; rr += 2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][kb][rr], c2, mneg));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[qb][kb][rr + 1], c2, mneg));
          const uint32_t w = pack2(p0, p1);
          pk[kb][rr >> 1] = w;
          if (rr & 2) ls1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), one2, ls1, false);
          else        ls0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), one2, ls0, false);
        }
      l_run[qb] += ls0 + ls1;

      // O^T[db][qb] += V^T . P^T over 4 key steps of 16.
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint32_t* w = &pk[ks >> 1][4 * (ks & 1)];
        const bf16x8 pb = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
#pragma unroll
        for (int db = 0; db < 2; ++db)
          oacc[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[ks][db], pb, oacc[db][qb], 0, 0, 0);
      }
    }
  }

  // Epilogue: O = O^T / l, 4 consecutive channels per store.
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const float l = swap_sum(l_run[qb]);
    const float inv = l > 0.f ? 1.0f / l : 0.f;
    if (qrow[qb] < 0) continue;
    u16* orow = obase + qrow[qb] * st;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint2 w = make_uint2(pack2(oacc[db][qb][4 * j] * inv, oacc[db][qb][4 * j + 1] * inv),
                                   pack2(oacc[db][qb][4 * j + 2] * inv, oacc[db][qb][4 * j + 3] * inv));
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j + 4 * hw) = w;
      }
  }
}

}  // namespace

bool w64_supported(int head_dim, int tile, bool dense, int n_tiles, int64_t span) {
  // 32-bit element offsets inside one (batch, head); at most 64 kept blocks.
  return head_dim == 64 && (dense || (tile == 8 && n_tiles <= 64)) && span < ((int64_t)1 << 31);
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
  hipLaunchKernelGGL(k_attn_w64, dim3((unsigned)total), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace ssba
