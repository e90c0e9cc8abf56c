// Host-side kernel selection: which attention and backward kernels a
// descriptor's shape is served by, and their names as profilers show them.
// Host code only (no kernels), so the argument-checking and dispatch layer
// can also be built and exercised on a CPU.
#include "ssba_common.h"

namespace ssba {

namespace {
constexpr int kMfmaChunk = 64;   // keys per chunk of the MFMA attention kernels
}  // namespace

const char* mfma_kernel_name(int head_dim, int tile, bool dense, bool gated) {
  static const char* const names[2][2][2] = {
      {{"k_attn_mfma<64, 3, false, false>", "k_attn_mfma<64, 3, true, false>"},
       {"k_attn_mfma<64, 4, false, false>", "k_attn_mfma<64, 4, true, false>"}},
      {{"k_attn_mfma<128, 3, false, false>", "k_attn_mfma<128, 3, true, false>"},
       {"k_attn_mfma<128, 4, false, false>", "k_attn_mfma<128, 4, true, false>"}}};
  if (gated && !dense) return head_dim == 64 ? "k_attn_mfma<64, 3, false, true>" : "k_attn_mfma<128, 3, false, true>";
  // The dense control runs natural-order rows only; it uses the 8x8 shape.
  const int ti = (!dense && tile == 16) ? 1 : 0;
  return names[head_dim == 64 ? 0 : 1][ti][dense ? 1 : 0];
}

bool mfma_supported(int head_dim, int tile, bool dense, int n_tiles, int seq, int64_t span) {
  // 32-bit byte offsets inside one (batch, head); at most 64 kept blocks;
  // natural-order chunks need at least one full chunk of rows.
  return (head_dim == 64 || head_dim == 128) && (dense || ((tile == 8 || tile == 16) && n_tiles <= 64)) &&
         seq >= kMfmaChunk && 2 * span < ((int64_t)1 << 32);
}

const char* attn_kernel_name(const AttnArgs& a, int head_dim, int tile, int dtype) {
  if (dtype == SSBA_DT_F32) return head_dim == 64 ? "k_attn_f32<64>" : "k_attn_f32<128>";
  if (mfma_supported(head_dim, tile, a.dense != 0, a.n_tiles, a.seq, (int64_t)a.seq * a.st))
    return mfma_kernel_name(head_dim, tile, a.dense != 0, a.gated != 0);
  static const char* const names[2][3] = {
      {"k_attn_bf16<64, 2>", "k_attn_bf16<64, 3>", "k_attn_bf16<64, 4>"},
      {"k_attn_bf16<128, 2>", "k_attn_bf16<128, 3>", "k_attn_bf16<128, 4>"}};
  return names[head_dim == 64 ? 0 : 1][tile == 4 ? 0 : tile == 8 ? 1 : 2];
}

bool bwd_supported(int head_dim, int tile, int n_tiles, int dtype) {
  return dtype == SSBA_DT_BF16 && (head_dim == 64 || head_dim == 128) && (tile == 8 || tile == 16) &&
         n_tiles <= 64;
}

}  // namespace ssba
