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
};

struct IndexArgs {
  const void* q;
  const void* k;
  int32_t* index;
  double* qb;            // [B][H][T_b][D] pooled sums
  double* kb;
  int32_t* flags;        // [B][H][T_b]
  int64_t sb, sh, st;
  int batch, heads, head_dim, n_tiles, keep, win_h, win_w, ny;
  Frame f;
};

// Launchers (each returns hipGetLastError() of its launch).
hipError_t launch_pool(const IndexArgs& a, int dtype, hipStream_t s);
hipError_t launch_gate_topk(const IndexArgs& a, hipStream_t s);
hipError_t launch_gate_static(const IndexArgs& a, int gate, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
// One-wave-per-64-rows bf16 kernel for head_dim 64 (8x8 blocks or dense).
bool mfma_supported(int head_dim, int tile, bool dense, int n_tiles, int seq, int64_t span);
hipError_t launch_attn_mfma(const AttnArgs& a, int head_dim, int tile, hipStream_t s);
const char* mfma_kernel_name(int head_dim, int tile, bool dense);
// Name of the kernel launch_attn_bf16 / launch_attn_f32 would run.
const char* attn_kernel_name(const AttnArgs& a, int head_dim, int tile, int dtype);

}  // namespace ssba
