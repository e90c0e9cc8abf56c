// C ABI of the SSBA forward library: argument validation, workspace sizing and
// dispatch to the gfx950 kernels.  See include/ssba.h for the contract.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <vector>

#include "ssba.h"
#include "ssba_common.h"

namespace {

using ssba::AttnArgs;
using ssba::Frame;
using ssba::IndexArgs;

constexpr int kMaxTiles = 1024;  // one gate workgroup ranks a whole row

bool is_topk(int gate) { return gate == SSBA_GATE_TOPK || gate == SSBA_GATE_TOPK_SHARED; }

int ilog2(int v) {
  int l = 0;
  while ((1 << l) < v) ++l;
  return l;
}

int mod(int a, int m) {
  const int r = a % m;
  return r < 0 ? r + m : r;
}

struct Shape {
  int64_t sb, sh, st;
  int n_tiles, ny, nx, seq;
  Frame f;
};

// Structural checks shared by every entry point (no pointers).  The dense
// path ignores the gate fields (gate, keep, window).
ssba_status check_desc(const ssba_desc* d, Shape* out, bool gate_fields = true) {
  if (!d) return SSBA_ERR_ARG;
  if (d->batch < 1 || d->heads < 1 || d->grid_h < 1 || d->grid_w < 1 || d->n_text < 0)
    return SSBA_ERR_SHAPE;
  if (d->dtype != SSBA_DT_BF16 && d->dtype != SSBA_DT_F32) return SSBA_ERR_ARG;
  if (gate_fields && d->gate != SSBA_GATE_TOPK && d->gate != SSBA_GATE_WINDOW &&
      d->gate != SSBA_GATE_DENSE && d->gate != SSBA_GATE_TOPK_SHARED)
    return SSBA_ERR_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return SSBA_ERR_UNSUPPORTED;
  if (d->tile != 4 && d->tile != 8 && d->tile != 16) return SSBA_ERR_UNSUPPORTED;
  if (d->grid_h % d->tile || d->grid_w % d->tile) return SSBA_ERR_SHAPE;
  if (!(std::isfinite(d->softmax_scale))) return SSBA_ERR_ARG;
  const int64_t t_img = (int64_t)d->grid_h * d->grid_w;
  const int64_t seq = d->n_text + t_img;
  if (seq > (int64_t)1 << 30) return SSBA_ERR_UNSUPPORTED;
  const int64_t n_tiles = t_img / ((int64_t)d->tile * d->tile);
  if (n_tiles > kMaxTiles) return SSBA_ERR_UNSUPPORTED;
  const int ny = d->grid_h / d->tile, nx = d->grid_w / d->tile;
  if (gate_fields && is_topk(d->gate) && (d->keep < 1 || d->keep > n_tiles)) return SSBA_ERR_ARG;
  if (gate_fields && d->gate == SSBA_GATE_WINDOW &&
      (d->win_h < 1 || d->win_w < 1 || ny % d->win_h || nx % d->win_w))
    return SSBA_ERR_ARG;
  int64_t sb = d->stride_b, sh = d->stride_h, st = d->stride_t;
  if (sb == 0 && sh == 0 && st == 0) {
    st = d->head_dim;
    sh = seq * st;
    sb = (int64_t)d->heads * sh;
  } else if (sb < 1 || sh < 1 || st < d->head_dim) {
    return SSBA_ERR_SHAPE;
  }
  // 16-byte vector loads in the bf16 kernel need 8-element aligned rows.
  if (d->dtype == SSBA_DT_BF16 && ((sb | sh | st) & 7)) return SSBA_ERR_UNSUPPORTED;
  // Element offsets must stay inside int64 and row indices inside int32.
  const double span = (double)(d->batch - 1) * sb + (double)(d->heads - 1) * sh + (double)seq * st;
  if (span > 9.0e18) return SSBA_ERR_SHAPE;
  // Workspace byte counts (index, pooled sums, per-head affinity rows) must
  // not wrap around size_t, and a launch covers every (batch, head) pair's
  // query groups with fewer than 2^31 workgroups.
  const double pairs = (double)d->batch * d->heads;
  if (pairs * (double)n_tiles * (double)(n_tiles + 1) * 8.0 > 9.0e18 ||
      pairs * (double)n_tiles * (double)d->head_dim * 16.0 > 9.0e18)
    return SSBA_ERR_SHAPE;
  if (pairs * (double)(seq / 64 + 1 + n_tiles * 4) >= 2147483648.0) return SSBA_ERR_UNSUPPORTED;
  if (out) {
    out->sb = sb;
    out->sh = sh;
    out->st = st;
    out->n_tiles = (int)n_tiles;
    out->ny = ny;
    out->nx = nx;
    out->seq = (int)seq;
    out->f.grid_h = d->grid_h;
    out->f.grid_w = d->grid_w;
    out->f.tile_log2 = ilog2(d->tile);
    out->f.nx = nx;
    out->f.sy = mod(d->shift_y, d->grid_h);
    out->f.sx = mod(d->shift_x, d->grid_w);
    out->f.n_text = d->n_text;
  }
  return SSBA_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Byte count passed by the entry points without a size argument: the caller
// vouches for the buffer, nothing is checked.
constexpr size_t kUnchecked = SIZE_MAX;

size_t index_bytes_of(const ssba_desc* d, const Shape& s) {
  return (size_t)4 * d->batch * d->heads * s.n_tiles * (s.n_tiles + 1);
}

// Scratch layout: [pooled q_b | pooled k_b] (top-k gates), [per-head
// affinity rows] (head-shared gate), then the status flags.
size_t flags_offset_of(const ssba_desc* d, const Shape& s) {
  const size_t rows = (size_t)d->batch * d->heads * s.n_tiles;
  size_t off = 0;
  if (is_topk(d->gate)) off += (size_t)16 * rows * d->head_dim;
  if (d->gate == SSBA_GATE_TOPK_SHARED) off += (size_t)8 * rows * s.n_tiles;
  return off;
}

size_t scratch_bytes_of(const ssba_desc* d, const Shape& s) {
  return flags_offset_of(d, s) + (size_t)4 * d->batch * d->heads * s.n_tiles;
}

// Backward scratch: lse2 and D ([B][H][T] fp32 each), then each query
// block's kept blocks as a 64-bit mask ([B][H][T_b]), then the key blocks in
// the key-side kernel's order (int32 [B][H][T_b]); every region 256-byte
// aligned.
struct BwdScratch {
  size_t lse2, delta, kmask, korder, total;
};

BwdScratch bwd_scratch(const ssba_desc* d, const Shape& s) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t rows = (size_t)d->batch * d->heads * s.seq;
  BwdScratch w;
  w.lse2 = 0;
  w.delta = up(4 * rows);
  w.kmask = w.delta + up(4 * rows);
  w.korder = w.kmask + up((size_t)8 * d->batch * d->heads * s.n_tiles);
  w.total = w.korder + up((size_t)4 * d->batch * d->heads * s.n_tiles);
  return w;
}

// Per-layer scratch slices of the layer driver start 256-byte aligned.
size_t layer_scratch_stride(const ssba_desc* d, const Shape& s) {
  return (scratch_bytes_of(d, s) + 255) / 256 * 256;
}

AttnArgs attn_args(const ssba_desc* d, const Shape& s, const void* q, const void* k, const void* v,
                   const int32_t* index, void* o, bool dense) {
  AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.index = index;
  a.sb = s.sb;
  a.sh = s.sh;
  a.st = s.st;
  a.batch = d->batch;
  a.heads = d->heads;
  a.seq = s.seq;
  a.n_tiles = s.n_tiles;
  a.f = s.f;
  const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.0f / std::sqrt((float)d->head_dim);
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.dense = dense ? 1 : 0;
  return a;
}

ssba_status run_attention(const ssba_desc* d, const void* q, const void* k, const void* v,
                          const int32_t* index, size_t index_bytes, void* o, void* stream, bool dense) {
  Shape s;
  ssba_status st = check_desc(d, &s, !dense);
  if (st != SSBA_OK) return st;
  if (!q || !k || !v || !o || (!dense && !index)) return SSBA_ERR_ARG;
  const size_t al = d->dtype == SSBA_DT_BF16 ? 16 : 4;
  if (!aligned(q, al) || !aligned(k, al) || !aligned(v, al) || !aligned(o, al) || !aligned(index, 4))
    return SSBA_ERR_ARG;
  if (!dense && index_bytes < index_bytes_of(d, s)) return SSBA_ERR_WORKSPACE;
  const AttnArgs a = attn_args(d, s, q, k, v, index, o, dense);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t e = d->dtype == SSBA_DT_BF16 ? ssba::launch_attn_bf16(a, d->head_dim, d->tile, hs)
                                          : ssba::launch_attn_f32(a, d->head_dim, d->tile, hs);
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

}  // namespace

extern "C" {

int ssba_abi_version(void) { return SSBA_ABI_VERSION; }

const char* ssba_status_str(ssba_status s) {
  switch (s) {
    case SSBA_OK: return "ok";
    case SSBA_ERR_ARG: return "invalid argument";
    case SSBA_ERR_SHAPE: return "invalid shape";
    case SSBA_ERR_UNSUPPORTED: return "unsupported configuration";
    case SSBA_ERR_WORKSPACE: return "workspace too small";
    case SSBA_ERR_NONFINITE: return "non-finite block affinity";
    case SSBA_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

ssba_status ssba_workspace_size(const ssba_desc* d, size_t* index_bytes, size_t* scratch_bytes) {
  Shape s;
  const ssba_status st = check_desc(d, &s);
  if (st != SSBA_OK) return st;
  if (index_bytes) *index_bytes = index_bytes_of(d, s);
  if (scratch_bytes) *scratch_bytes = scratch_bytes_of(d, s);
  return SSBA_OK;
}

}  // extern "C"

namespace {

IndexArgs index_args(const ssba_desc* d, const Shape& s, const void* q, const void* k, int32_t* index,
                     void* scratch) {
  IndexArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q;
  a.k = k;
  a.index = index;
  const size_t pooled = (size_t)d->batch * d->heads * s.n_tiles * d->head_dim;
  double* base = static_cast<double*>(scratch);
  if (is_topk(d->gate)) {
    a.qb = base;
    a.kb = base + pooled;
  }
  if (d->gate == SSBA_GATE_TOPK_SHARED) a.srows = base + 2 * pooled;
  a.flags = reinterpret_cast<int32_t*>(static_cast<char*>(scratch) + flags_offset_of(d, s));
  a.sb = s.sb;
  a.sh = s.sh;
  a.st = s.st;
  a.batch = d->batch;
  a.heads = d->heads;
  a.head_dim = d->head_dim;
  a.n_tiles = s.n_tiles;
  a.keep = d->keep;
  a.win_h = d->win_h;
  a.win_w = d->win_w;
  a.ny = s.ny;
  a.f = s.f;
  return a;
}

// Shapes whose top-k gate can run inside the attention kernel.
bool gated_supported(const ssba_desc* d, const Shape& s) {
  return d->dtype == SSBA_DT_BF16 && d->tile == 8 &&
         ssba::mfma_supported(d->head_dim, 8, false, s.n_tiles, s.seq, (int64_t)s.seq * s.st);
}

// Checks shared by the two launches of the fused top-k form; `attention`
// for the gated attention launch (Q, V, O and the index too).
ssba_status check_fused(const ssba_desc* d, Shape* s, const void* q, const void* k, const void* v,
                        const int32_t* index, size_t index_bytes, const void* scratch, size_t scratch_bytes,
                        const void* o, bool attention) {
  ssba_status st = check_desc(d, s);
  if (st != SSBA_OK) return st;
  if (d->gate != SSBA_GATE_TOPK || !gated_supported(d, *s)) return SSBA_ERR_UNSUPPORTED;
  if (!k || !scratch || !aligned(k, 16) || !aligned(scratch, 16)) return SSBA_ERR_ARG;
  if (attention && (!q || !v || !o || !index || !aligned(q, 16) || !aligned(v, 16) || !aligned(o, 16) ||
                    !aligned(index, 4)))
    return SSBA_ERR_ARG;
  if (scratch_bytes < scratch_bytes_of(d, *s) || (attention && index_bytes < index_bytes_of(d, *s)))
    return SSBA_ERR_WORKSPACE;
  return SSBA_OK;
}

}  // namespace

extern "C" {

ssba_status ssba_build_index_ex(const ssba_desc* d, const void* q, const void* k, int32_t* index,
                                size_t index_bytes, void* scratch, size_t scratch_bytes, void* stream) {
  Shape s;
  const ssba_status st = check_desc(d, &s);
  if (st != SSBA_OK) return st;
  if (!index || !scratch || !aligned(index, 4) || !aligned(scratch, 16)) return SSBA_ERR_ARG;
  const bool topk = is_topk(d->gate);
  if (topk) {
    const size_t al = d->dtype == SSBA_DT_BF16 ? 16 : 4;
    if (!q || !k || !aligned(q, al) || !aligned(k, al)) return SSBA_ERR_ARG;
  }
  if (index_bytes < index_bytes_of(d, s) || scratch_bytes < scratch_bytes_of(d, s)) return SSBA_ERR_WORKSPACE;
  const IndexArgs a = index_args(d, s, q, k, index, scratch);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (topk) {
    e = ssba::launch_pool(a, d->dtype, hs);
    if (e == hipSuccess)
      e = d->gate == SSBA_GATE_TOPK ? ssba::launch_gate_topk(a, hs) : ssba::launch_gate_topk_shared(a, hs);
  } else {
    e = ssba::launch_gate_static(a, d->gate, hs);
  }
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_build_index(const ssba_desc* d, const void* q, const void* k, int32_t* index,
                             void* scratch, void* stream) {
  return ssba_build_index_ex(d, q, k, index, kUnchecked, scratch, kUnchecked, stream);
}

ssba_status ssba_forward_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                            const int32_t* index, size_t index_bytes, void* o, void* stream) {
  return run_attention(d, q, k, v, index, index_bytes, o, stream, false);
}

ssba_status ssba_forward(const ssba_desc* d, const void* q, const void* k, const void* v,
                         const int32_t* index, void* o, void* stream) {
  return run_attention(d, q, k, v, index, kUnchecked, o, stream, false);
}

ssba_status ssba_forward_dense(const ssba_desc* d, const void* q, const void* k, const void* v,
                               void* o, void* stream) {
  return run_attention(d, q, k, v, nullptr, kUnchecked, o, stream, true);
}

ssba_status ssba_pool_keys_ex(const ssba_desc* d, const void* k, void* scratch, size_t scratch_bytes,
                              void* stream) {
  Shape s;
  const ssba_status st = check_fused(d, &s, nullptr, k, nullptr, nullptr, 0, scratch, scratch_bytes, nullptr,
                                     false);
  if (st != SSBA_OK) return st;
  const IndexArgs ia = index_args(d, s, nullptr, k, nullptr, scratch);
  return ssba::launch_pool_keys(ia, static_cast<hipStream_t>(stream)) == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_forward_gated_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                  int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                  void* o, void* stream) {
  Shape s;
  const ssba_status st = check_fused(d, &s, q, k, v, index, index_bytes, scratch, scratch_bytes, o, true);
  if (st != SSBA_OK) return st;
  // Each block's pooled query sum is formed in the kernel from its own Q
  // rows; the pooled key sums come from ssba_pool_keys_ex.
  const IndexArgs ia = index_args(d, s, q, k, index, scratch);
  AttnArgs aa = attn_args(d, s, q, k, v, nullptr, o, false);
  aa.gated = 1;
  aa.keep = d->keep;
  aa.kb = ia.kb;
  aa.index_out = index;
  aa.flags = ia.flags;
  const hipError_t e = ssba::launch_attn_bf16(aa, d->head_dim, d->tile, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_forward_topk_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                 int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                 void* o, void* stream) {
  Shape s;
  ssba_status st = check_desc(d, &s);
  if (st != SSBA_OK) return st;
  if (!is_topk(d->gate)) return SSBA_ERR_ARG;
  if (!q || !k || !v || !o || !index || !scratch) return SSBA_ERR_ARG;
  const size_t al = d->dtype == SSBA_DT_BF16 ? 16 : 4;
  if (!aligned(q, al) || !aligned(k, al) || !aligned(v, al) || !aligned(o, al) || !aligned(index, 4) ||
      !aligned(scratch, 16))
    return SSBA_ERR_ARG;
  if (index_bytes < index_bytes_of(d, s) || scratch_bytes < scratch_bytes_of(d, s)) return SSBA_ERR_WORKSPACE;
  if (d->gate != SSBA_GATE_TOPK || !gated_supported(d, s)) {   // the two calls, same results
    st = ssba_build_index_ex(d, q, k, index, index_bytes, scratch, scratch_bytes, stream);
    return st != SSBA_OK ? st : ssba_forward_ex(d, q, k, v, index, index_bytes, o, stream);
  }
  // Pooled key sums, then the attention kernel, which gates each block and attends.
  st = ssba_pool_keys_ex(d, k, scratch, scratch_bytes, stream);
  return st != SSBA_OK ? st : ssba_forward_gated_ex(d, q, k, v, index, index_bytes, scratch, scratch_bytes, o, stream);
}

ssba_status ssba_rope_pool_keys_ex(const ssba_desc* d, const void* q, const void* k, void* q_rope, void* k_rope,
                                  float theta, void* scratch, size_t scratch_bytes, void* stream) {
  Shape s;
  const ssba_status st = check_fused(d, &s, nullptr, k, nullptr, nullptr, 0, scratch, scratch_bytes, nullptr,
                                     false);
  if (st != SSBA_OK) return st;
  if (!q || !q_rope || !k_rope || !aligned(q, 16) || !aligned(q_rope, 16) || !aligned(k_rope, 16))
    return SSBA_ERR_ARG;
  if (!std::isfinite(theta)) return SSBA_ERR_ARG;
  const double base = theta > 0.f ? (double)theta : 10000.0;   // <= 0: the default base
  ssba::RopeArgs r;
  std::memset(&r, 0, sizeof(r));
  r.a = index_args(d, s, q, k, nullptr, scratch);
  r.q_out = q_rope;
  r.k_out = k_rope;
  const int pairs = d->head_dim / 4;
  for (int i = 0; i < pairs; ++i) r.inv_freq[i] = std::pow(base, -(double)i / (double)pairs);
  r.n_text_groups = (d->n_text + 63) / 64;
  return ssba::launch_rope_pool_keys(r, static_cast<hipStream_t>(stream)) == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_forward_topk_rope_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                     void* q_rope, void* k_rope, float theta, int32_t* index, size_t index_bytes,
                                     void* scratch, size_t scratch_bytes, void* o, void* stream) {
  Shape s;
  const ssba_status st = check_fused(d, &s, q, k, v, index, index_bytes, scratch, scratch_bytes, o, true);
  if (st != SSBA_OK) return st;
  const ssba_status sr = ssba_rope_pool_keys_ex(d, q, k, q_rope, k_rope, theta, scratch, scratch_bytes, stream);
  if (sr != SSBA_OK) return sr;
  return ssba_forward_gated_ex(d, q_rope, k_rope, v, index, index_bytes, scratch, scratch_bytes, o, stream);
}

ssba_status ssba_forward_topk(const ssba_desc* d, const void* q, const void* k, const void* v,
                              int32_t* index, void* scratch, void* o, void* stream) {
  return ssba_forward_topk_ex(d, q, k, v, index, kUnchecked, scratch, kUnchecked, o, stream);
}

const char* ssba_forward_kernel(const ssba_desc* d, int mode) {
  Shape s;
  const bool dense = mode == 1;
  if (mode < 0 || mode > 2 || check_desc(d, &s, !dense) != SSBA_OK) return nullptr;
  if (mode == 2 && !is_topk(d->gate)) return nullptr;
  AttnArgs a = attn_args(d, s, nullptr, nullptr, nullptr, nullptr, nullptr, dense);
  a.gated = (mode == 2 && d->gate == SSBA_GATE_TOPK && gated_supported(d, s)) ? 1 : 0;
  return ssba::attn_kernel_name(a, d->head_dim, d->tile, d->dtype);
}

ssba_status ssba_forward_train_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                  const int32_t* index, size_t index_bytes, void* o, float* lse,
                                  void* stream) {
  Shape s;
  const ssba_status st = check_desc(d, &s, false);
  if (st != SSBA_OK) return st;
  if (d->dtype != SSBA_DT_BF16 ||
      !ssba::mfma_supported(d->head_dim, d->tile, false, s.n_tiles, s.seq, (int64_t)s.seq * s.st))
    return SSBA_ERR_UNSUPPORTED;
  if (!q || !k || !v || !o || !index || !lse) return SSBA_ERR_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) || !aligned(index, 4) ||
      !aligned(lse, 4))
    return SSBA_ERR_ARG;
  if (index_bytes < index_bytes_of(d, s)) return SSBA_ERR_WORKSPACE;
  AttnArgs a = attn_args(d, s, q, k, v, index, o, false);
  a.lse = lse;
  const hipError_t e = ssba::launch_attn_bf16(a, d->head_dim, d->tile, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_forward_train(const ssba_desc* d, const void* q, const void* k, const void* v,
                               const int32_t* index, void* o, float* lse, void* stream) {
  return ssba_forward_train_ex(d, q, k, v, index, kUnchecked, o, lse, stream);
}

ssba_status ssba_backward_workspace_size(const ssba_desc* d, size_t* scratch_bytes) {
  Shape s;
  const ssba_status st = check_desc(d, &s, false);
  if (st != SSBA_OK) return st;
  if (scratch_bytes) *scratch_bytes = bwd_scratch(d, s).total;
  return SSBA_OK;
}

ssba_status ssba_backward_ex(const ssba_desc* d, const void* q, const void* k, const void* v, const void* o,
                             const void* dout, const float* lse, const int32_t* index, size_t index_bytes,
                             void* dq, void* dk, void* dv, void* scratch, size_t scratch_bytes, void* stream) {
  Shape s;
  const ssba_status st = check_desc(d, &s, false);
  if (st != SSBA_OK) return st;
  if (!ssba::bwd_supported(d->head_dim, d->tile, s.n_tiles, d->dtype) ||
      !ssba::mfma_supported(d->head_dim, d->tile, false, s.n_tiles, s.seq, (int64_t)s.seq * s.st))
    return SSBA_ERR_UNSUPPORTED;
  const void* t16[] = {q, k, v, o, dout, dq, dk, dv};
  for (const void* p : t16)
    if (!p || !aligned(p, 16)) return SSBA_ERR_ARG;
  if (!lse || !index || !scratch || !aligned(lse, 4) || !aligned(index, 4) || !aligned(scratch, 256))
    return SSBA_ERR_ARG;
  const BwdScratch w = bwd_scratch(d, s);
  if (index_bytes < index_bytes_of(d, s) || scratch_bytes < w.total) return SSBA_ERR_WORKSPACE;
  ssba::BwdArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.dout = dout;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.lse = lse;
  char* base = static_cast<char*>(scratch);
  a.lse2 = reinterpret_cast<float*>(base + w.lse2);
  a.delta = reinterpret_cast<float*>(base + w.delta);
  a.kmask = reinterpret_cast<unsigned long long*>(base + w.kmask);
  a.korder = reinterpret_cast<int32_t*>(base + w.korder);
  a.index = index;
  a.sb = s.sb;
  a.sh = s.sh;
  a.st = s.st;
  a.batch = d->batch;
  a.heads = d->heads;
  a.seq = s.seq;
  a.n_tiles = s.n_tiles;
  a.f = s.f;
  const float scale = d->softmax_scale > 0.f ? d->softmax_scale : 1.0f / std::sqrt((float)d->head_dim);
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  const hipError_t e = ssba::launch_backward(a, d->head_dim, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}

ssba_status ssba_backward(const ssba_desc* d, const void* q, const void* k, const void* v, const void* o,
                          const void* dout, const float* lse, const int32_t* index, void* dq, void* dk,
                          void* dv, void* scratch, void* stream) {
  return ssba_backward_ex(d, q, k, v, o, dout, lse, index, kUnchecked, dq, dk, dv, scratch, kUnchecked,
                          stream);
}

ssba_status ssba_layers_workspace_size(const ssba_desc* d, int n_layers, size_t* index_bytes,
                                       size_t* scratch_bytes) {
  if (!d || n_layers < 1) return SSBA_ERR_ARG;
  ssba_desc base = *d;
  if (is_topk(base.gate)) base.keep = 1;   // per-layer keeps are checked by the layer driver
  Shape s;
  const ssba_status st = check_desc(&base, &s);
  if (st != SSBA_OK) return st;
  if (index_bytes) *index_bytes = (size_t)n_layers * index_bytes_of(&base, s);
  if (scratch_bytes) *scratch_bytes = (size_t)n_layers * layer_scratch_stride(&base, s);
  return SSBA_OK;
}

ssba_status ssba_forward_layers_ex(const ssba_desc* d, const ssba_layer* layers, int n_layers,
                                   int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                   void* stream) {
  if (!d || !layers || n_layers < 1) return SSBA_ERR_ARG;
  ssba_desc base = *d;
  if (is_topk(base.gate)) base.keep = 1;
  Shape s;
  ssba_status st = check_desc(&base, &s);
  if (st != SSBA_OK) return st;
  if (!index || !scratch || !aligned(index, 4) || !aligned(scratch, 16)) return SSBA_ERR_ARG;
  // Every layer is checked before the first launch.
  const size_t al = d->dtype == SSBA_DT_BF16 ? 16 : 4;
  for (int l = 0; l < n_layers; ++l) {
    const ssba_layer& L = layers[l];
    if (L.skip) continue;
    if (!L.q || !L.k || !L.v || !L.o || !aligned(L.q, al) || !aligned(L.k, al) || !aligned(L.v, al) ||
        !aligned(L.o, al))
      return SSBA_ERR_ARG;
    if (is_topk(d->gate) && (L.keep < 1 || L.keep > s.n_tiles)) return SSBA_ERR_ARG;
  }
  const size_t idx_bytes = index_bytes_of(&base, s);
  const size_t idx_elems = idx_bytes / sizeof(int32_t);
  const size_t scr_stride = layer_scratch_stride(&base, s);
  if (index_bytes / idx_bytes < (size_t)n_layers || scratch_bytes / scr_stride < (size_t)n_layers)
    return SSBA_ERR_WORKSPACE;
  if (d->gate == SSBA_GATE_TOPK && gated_supported(&base, s)) {
    // The fused form, batched over layers: one launch pools the keys of up
    // to 32 layers into their scratch slices, then one launch runs those
    // layers' gated attention (grid y = layer), each reading its slice.
    // Every workgroup does what it does in one ssba_forward_topk call per
    // layer, so the indices, flags and outputs are the same bits.
    static_assert(ssba::kPoolLayersMax == ssba::kAttnLayersMax, "one chunk of layers per launch pair");
    ssba_desc odd = base;
    odd.shift_y = -d->shift_y;
    odd.shift_x = -d->shift_x;
    Shape so;
    st = check_desc(&odd, &so);
    if (st != SSBA_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    ssba::PoolLayers p;
    ssba::AttnLayers at;
    for (int l0 = 0; l0 < n_layers;) {
      std::memset(&p, 0, sizeof(p));
      std::memset(&at, 0, sizeof(at));
      p.a = index_args(&base, s, nullptr, nullptr, nullptr, scratch);
      p.f[0] = at.f[0] = s.f;
      p.f[1] = at.f[1] = so.f;
      at.a = attn_args(&base, s, nullptr, nullptr, nullptr, nullptr, nullptr, false);
      at.a.gated = 1;
      int np = 0, l1 = l0;
      for (; l1 < n_layers && np < ssba::kPoolLayersMax; ++l1) {
        const ssba_layer& L = layers[l1];
        if (L.skip) continue;
        const IndexArgs ia = index_args(&base, s, nullptr, nullptr, nullptr,
                                        static_cast<char*>(scratch) + (size_t)l1 * scr_stride);
        p.k[np] = L.k;
        p.kb[np] = ia.kb;
        p.parity[np] = at.parity[np] = l1 & 1;
        at.q[np] = L.q;
        at.k[np] = L.k;
        at.v[np] = L.v;
        at.o[np] = L.o;
        at.kb[np] = ia.kb;
        at.index_out[np] = index + (size_t)l1 * idx_elems;
        at.flags[np] = ia.flags;
        at.keep[np] = L.keep;
        ++np;
      }
      if (np > 0 && (ssba::launch_pool_keys_layers(p, np, hs) != hipSuccess ||
                     ssba::launch_attn_mfma_layers(at, np, d->head_dim, 8, hs) != hipSuccess))
        return SSBA_ERR_HIP;
      l0 = l1;
    }
    return SSBA_OK;
  }
  int cached[2] = {-1, -1};   // static gates: the layer whose index serves each parity
  if (d->dtype == SSBA_DT_BF16 &&
      ssba::mfma_supported(d->head_dim, d->tile, false, s.n_tiles, s.seq, (int64_t)s.seq * s.st)) {
    // Each layer's index as one call per layer builds it (the head-shared
    // top-k gate of up to 32 layers in one launch per step, a static gate
    // once per offset parity), then the attention of those layers in one
    // launch (grid y = layer) reading their indices: the same bits as one
    // call per layer.
    static_assert(ssba::kIndexLayersMax == ssba::kAttnLayersMax, "one chunk of layers per launch group");
    ssba_desc odd = base;
    odd.shift_y = -d->shift_y;
    odd.shift_x = -d->shift_x;
    Shape so;
    st = check_desc(&odd, &so);
    if (st != SSBA_OK) return st;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    const bool shared = d->gate == SSBA_GATE_TOPK_SHARED;
    ssba::AttnLayers at;
    ssba::IndexLayers ix;
    for (int l0 = 0; l0 < n_layers;) {
      std::memset(&at, 0, sizeof(at));
      std::memset(&ix, 0, sizeof(ix));
      at.f[0] = ix.f[0] = s.f;
      at.f[1] = ix.f[1] = so.f;
      at.a = attn_args(&base, s, nullptr, nullptr, nullptr, nullptr, nullptr, false);
      ix.a = index_args(&base, s, nullptr, nullptr, nullptr, scratch);
      int np = 0, l1 = l0;
      for (; l1 < n_layers && np < ssba::kAttnLayersMax; ++l1) {
        const ssba_layer& L = layers[l1];
        if (L.skip) continue;
        int32_t* il = index + (size_t)l1 * idx_elems;
        void* sl = static_cast<char*>(scratch) + (size_t)l1 * scr_stride;
        const int par = l1 & 1;
        if (shared) {
          const IndexArgs ia = index_args(&base, s, L.q, L.k, il, sl);
          ix.q[np] = L.q;
          ix.k[np] = L.k;
          ix.index[np] = il;
          ix.qb[np] = ia.qb;
          ix.kb[np] = ia.kb;
          ix.flags[np] = ia.flags;
          ix.srows[np] = ia.srows;
          ix.keep[np] = L.keep;
          ix.parity[np] = par;
          at.index[np] = il;
        } else {
          if (cached[par] < 0) {
            const ssba_desc& dl = par ? odd : base;
            st = ssba_build_index_ex(&dl, nullptr, nullptr, il, idx_bytes, sl, scr_stride, stream);
            if (st != SSBA_OK) return st;
            cached[par] = l1;
          }
          at.index[np] = index + (size_t)cached[par] * idx_elems;
        }
        at.q[np] = L.q;
        at.k[np] = L.k;
        at.v[np] = L.v;
        at.o[np] = L.o;
        at.parity[np] = par;
        ++np;
      }
      if (np > 0 && ((shared && ssba::launch_topk_shared_layers(ix, np, hs) != hipSuccess) ||
                     ssba::launch_attn_mfma_layers(at, np, d->head_dim, d->tile, hs) != hipSuccess))
        return SSBA_ERR_HIP;
      l0 = l1;
    }
    return SSBA_OK;
  }
  for (int l = 0; l < n_layers; ++l) {
    const ssba_layer& L = layers[l];
    if (L.skip) continue;
    ssba_desc dl = base;
    if (l & 1) {   // Section 2.2.2: the offset alternates sign between layers
      dl.shift_y = -d->shift_y;
      dl.shift_x = -d->shift_x;
    }
    int32_t* il = index + (size_t)l * idx_elems;
    void* sl = static_cast<char*>(scratch) + (size_t)l * scr_stride;
    if (is_topk(d->gate)) {
      dl.keep = L.keep;
      st = ssba_forward_topk_ex(&dl, L.q, L.k, L.v, il, idx_bytes, sl, scr_stride, L.o, stream);
    } else {
      const int par = l & 1;
      if (cached[par] < 0) {
        st = ssba_build_index_ex(&dl, nullptr, nullptr, il, idx_bytes, sl, scr_stride, stream);
        if (st != SSBA_OK) return st;
        cached[par] = l;
      }
      st = ssba_forward_ex(&dl, L.q, L.k, L.v, index + (size_t)cached[par] * idx_elems, idx_bytes, L.o, stream);
    }
    if (st != SSBA_OK) return st;
  }
  return SSBA_OK;
}

ssba_status ssba_forward_layers(const ssba_desc* d, const ssba_layer* layers, int n_layers,
                                int32_t* index, void* scratch, void* stream) {
  return ssba_forward_layers_ex(d, layers, n_layers, index, kUnchecked, scratch, kUnchecked, stream);
}

ssba_status ssba_read_device_status_ex(const ssba_desc* d, const void* scratch, size_t scratch_bytes,
                                       ssba_status* out, void* stream) {
  if (!d) return SSBA_ERR_ARG;
  ssba_desc base = *d;   // the flags do not depend on keep
  if (is_topk(base.gate) && base.keep < 1) base.keep = 1;
  Shape s;
  const ssba_status st = check_desc(&base, &s);
  if (st != SSBA_OK) return st;
  if (!scratch || !out || !aligned(scratch, 8)) return SSBA_ERR_ARG;
  if (scratch_bytes < scratch_bytes_of(&base, s)) return SSBA_ERR_WORKSPACE;
  const size_t n = (size_t)d->batch * d->heads * s.n_tiles;
  const int32_t* flags =
      reinterpret_cast<const int32_t*>(static_cast<const char*>(scratch) + flags_offset_of(&base, s));
  std::vector<int32_t> host(n);
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(host.data(), flags, n * sizeof(int32_t), hipMemcpyDeviceToHost, hs) != hipSuccess)
    return SSBA_ERR_HIP;
  if (hipStreamSynchronize(hs) != hipSuccess) return SSBA_ERR_HIP;
  int32_t any = 0;
  for (int32_t f : host) any |= f;
  *out = any ? SSBA_ERR_NONFINITE : SSBA_OK;
  return SSBA_OK;
}

ssba_status ssba_read_device_status(const ssba_desc* d, const void* scratch, ssba_status* out,
                                    void* stream) {
  return ssba_read_device_status_ex(d, scratch, kUnchecked, out, stream);
}

}  // extern "C"
