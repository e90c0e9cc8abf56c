// Internal declarations shared by the SSBA host library and its HIP kernels.
// Not part of the public ABI (include/ssba.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ssba.h"

namespace ssba {

// Shifted block frame of one SSBA call (Section 2.2.2).  The image grid is
// rolled by (sy, sx) and cut into tile x tile blocks; block t = (ty, tx) and
// slot s map back to the original image token through row_of().
struct Frame {
  int grid_h, grid_w;
  int tile_log2;   // tile = 1 << tile_log2
  int nx;          // blocks per grid row
  int sy, sx;      // shift reduced into [0, grid_h) x [0, grid_w)
  int n_text;      // image rows start here
};

// Sequence row (text first) of slot s of block t in the shifted frame.
__host__ __device__ __forceinline__ int frame_row(const Frame& f, int t, int s) {
  const int tile = 1 << f.tile_log2;
  const int ty = t / f.nx, tx = t - ty * f.nx;
  int y = (ty << f.tile_log2) + (s >> f.tile_log2) - f.sy;
  int x = (tx << f.tile_log2) + (s & (tile - 1)) - f.sx;
  y += (y < 0) ? f.grid_h : 0;
  x += (x < 0) ? f.grid_w : 0;
  return f.n_text + y * f.grid_w + x;
}

// Ranking key of the top-k gate: an unsigned integer whose order is the
// gate's order on affinities.  -0 is folded onto +0 and every NaN onto key 0,
// below all numbers; equal keys are then ordered by ascending block index.
__device__ __forceinline__ uint64_t rank_key(double s) {
  if (s != s) return 0;
  if (s == 0.0) s = 0.0;
  const uint64_t u = (uint64_t)__double_as_longlong(s);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Top-k selection over one wave (lane = block id < tb): true in the lanes of
// the `keep` blocks ranked first by (key descending, block id ascending).
// Radix select: the keep-th largest key is found bit by bit from the top
// with wave ballots; keys above it are kept and, of the keys equal to it,
// the lowest block ids fill the remaining places.  The search stops early
// once exactly `keep` keys lie at or above the bits decided so far: that set
// is then the answer.  Invalid lanes count as key 0, which no candidate
// (always >= 1) reaches.
__device__ __forceinline__ bool wave_topk(uint64_t key, bool valid, int keep, int lane) {
  const uint64_t k = valid ? key : 0;
  uint64_t thr = 0;
#pragma unroll 4
  for (int bit = 63; bit >= 0; --bit) {
    const uint64_t cand = thr | (1ull << bit);
    const int n = __popcll(__builtin_amdgcn_ballot_w64(k >= cand));
    if (n >= keep) {
      thr = cand;
      if (n == keep) break;
    }
  }
  const bool gt = valid && k > thr, eq = valid && k == thr;
  const int need = keep - __popcll(__builtin_amdgcn_ballot_w64(gt));
  const int before = __popcll(__builtin_amdgcn_ballot_w64(eq) & ((1ull << lane) - 1ull));
  return gt || (eq && before < need);
}

// Everything an attention launch needs; passed by value as a kernel argument.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  const int32_t* index;  // [B][H][T_b][1 + T_b]; unused by dense launches
  int64_t sb, sh, st;    // element strides (channel stride 1)
  int batch, heads, seq;  // seq = T = n_text + grid_h * grid_w
  int n_tiles;           // T_b
  Frame f;
  float scale_log2;      // softmax scale * log2(e)
  float scale;           // softmax scale
  int n_text_groups;     // leading workgroups that run text query rows (dense rows)
  int groups_per_tile;   // image workgroups per query block (tile^2 / rows per group)
  int groups_per_bh;     // workgroups per (batch, head)
  int dense;             // 1: every row attends every key in natural order
  // Gated launches compute the top-k gate of each image block in the kernel
  // from the pooled sums and write the index rows and status flags.
  int gated;
  int keep;
  const double* kb;      // [B][H][D][T_b] pooled key sums
  int32_t* index_out;    // [B][H][T_b][1 + T_b]
  int32_t* flags;        // [B][H][T_b]
  // Optional (MFMA kernels): natural-log log-sum-exp of each row's scaled
  // scores, [B][H][T] fp32, for the backward pass.
  float* lse;
  // MFMA kernels, set by their launcher: 1 when every workgroup of the grid
  // is resident at once, so the waves are prioritised by the chunks they
  // have left (see k_attn_mfma).
  int equalize;
};

// Attention of up to kAttnLayersMax layers of one shape in one launch (the
// layer driver): layer y reads q/k/v[y] and writes o[y] in frame
// f[parity[y]]; a gated launch (a.gated) reads kb[y], writes index_out[y]
// and flags[y] and keeps keep[y] blocks, an ungated one reads index[y];
// every other field is a's.
constexpr int kAttnLayersMax = 32;
struct AttnLayers {
  AttnArgs a;
  Frame f[2];
  const void* q[kAttnLayersMax];
  const void* k[kAttnLayersMax];
  const void* v[kAttnLayersMax];
  void* o[kAttnLayersMax];
  const int32_t* index[kAttnLayersMax];
  const double* kb[kAttnLayersMax];
  int32_t* index_out[kAttnLayersMax];
  int32_t* flags[kAttnLayersMax];
  int keep[kAttnLayersMax];
  int parity[kAttnLayersMax];
};

struct IndexArgs {
  const void* q;
  const void* k;
  int32_t* index;
  double* qb;            // [B][H][T_b][D] pooled sums
  double* kb;
  int32_t* flags;        // [B][H][T_b]
  double* srows;         // [B][H][T_b][T_b] per-head affinity rows (head-shared gate)
  int64_t sb, sh, st;
  int batch, heads, head_dim, n_tiles, keep, win_h, win_w, ny;
  Frame f;
};

// Everything the backward kernels need.
struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;
  void* dq;
  void* dk;
  void* dv;
  const float* lse;      // [B][H][T] natural-log log-sum-exp from the forward
  float* lse2;           // [B][H][T] scratch: lse * log2(e)
  float* delta;          // [B][H][T] scratch: rowsum(dO * O)
  const int32_t* index;  // [B][H][T_b][1 + T_b]
  unsigned long long* kmask;  // [B][H][T_b] scratch: kept blocks of each query block as bits
  int32_t* korder;            // [B][H][T_b] scratch: key blocks in the key-side kernel's order
  int64_t sb, sh, st;
  int batch, heads, seq, n_tiles, n_text_groups;
  Frame f;
  float scale, scale_log2;
};

// The pooled-key pre-pass of up to kPoolLayersMax layers in one launch (the
// layer driver): layer y pools K at k[y] into kb[y] in the frame
// f[parity[y]] (the shift alternates sign between layers); every other
// field is a's.
constexpr int kPoolLayersMax = 32;
struct PoolLayers {
  IndexArgs a;
  Frame f[2];
  const void* k[kPoolLayersMax];
  double* kb[kPoolLayersMax];
  int parity[kPoolLayersMax];
};

// The rotary pre-pass of the fused call (bf16, 8x8 blocks): rotated Q and K
// written to q_out / k_out and the pooled sums of the rotated keys to a.kb.
// inv_freq[i] = theta^(-i / (D/4)) for the D/4 pairs of a half.
struct RopeArgs {
  IndexArgs a;
  void* q_out;
  void* k_out;
  double inv_freq[32];
  int n_text_groups;   // workgroups per (batch, head) that copy text rows
};
hipError_t launch_rope_pool_keys(const RopeArgs& r, hipStream_t s);

// The head-shared top-k gate of up to kIndexLayersMax layers of one shape,
// each step one launch (the layer driver): layer y reads q/k[y], writes its
// pooled sums to qb/kb[y], its per-head rows to srows[y], its index and
// flags to index/flags[y], keeps keep[y] blocks, in frame f[parity[y]];
// every other field is a's.
constexpr int kIndexLayersMax = 32;
struct IndexLayers {
  IndexArgs a;
  Frame f[2];
  const void* q[kIndexLayersMax];
  const void* k[kIndexLayersMax];
  int32_t* index[kIndexLayersMax];
  double* qb[kIndexLayersMax];
  double* kb[kIndexLayersMax];
  int32_t* flags[kIndexLayersMax];
  double* srows[kIndexLayersMax];
  int keep[kIndexLayersMax];
  int parity[kIndexLayersMax];
};

// Launchers (each returns hipGetLastError() of its launch).
hipError_t launch_pool(const IndexArgs& a, int dtype, hipStream_t s);
// Pooled key sums only (bf16, 8x8 blocks): the pre-pass of the gated attention
// kernel, which forms the pooled query sums itself.
hipError_t launch_pool_keys(const IndexArgs& a, hipStream_t s);
// The same for n_layers <= kPoolLayersMax layers of one shape.
hipError_t launch_pool_keys_layers(const PoolLayers& p, int n_layers, hipStream_t s);
hipError_t launch_gate_topk(const IndexArgs& a, hipStream_t s);
// The head-shared gate (bf16, 8x8 or 16x16 blocks, T_b <= 64) of
// n_layers <= kIndexLayersMax layers: pooling, affinity rows, ranking.
hipError_t launch_topk_shared_layers(const IndexLayers& p, int n_layers, hipStream_t s);
// Head-shared top-k gate: per-head affinity rows, then their sum over heads.
hipError_t launch_gate_topk_shared(const IndexArgs& a, hipStream_t s);
hipError_t launch_gate_static(const IndexArgs& a, int gate, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
// Four-wave MFMA kernel: head_dim 64 / 128, 8x8 / 16x16 blocks, dense control;
// gated launches (a.gated) need 8x8 blocks.
bool mfma_supported(int head_dim, int tile, bool dense, int n_tiles, int seq, int64_t span);
hipError_t launch_attn_mfma(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
// Attention (bf16, D 64 or 128; 8x8 blocks when gated, 8x8 or 16x16 with an
// index) of n_layers <= kAttnLayersMax layers, on shapes mfma_supported takes.
hipError_t launch_attn_mfma_layers(const AttnLayers& p, int n_layers, int head_dim, int tile, hipStream_t s);
const char* mfma_kernel_name(int head_dim, int tile, bool dense, bool gated);
// Backward: bf16, 8x8 or 16x16 blocks, head_dim 64 / 128, at most 64 blocks.
bool bwd_supported(int head_dim, int tile, int n_tiles, int dtype);
hipError_t launch_backward(const BwdArgs& a, int head_dim, hipStream_t s);
// Name of the kernel launch_attn_bf16 / launch_attn_f32 would run.
const char* attn_kernel_name(const AttnArgs& a, int head_dim, int tile, int dtype);

}  // namespace ssba
