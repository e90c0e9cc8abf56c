// Recording stand-ins for the kernel launchers of the SSBA library, for a CPU
// build of its host layer (argument checks, workspace arithmetic, dispatch,
// the layer-stack driver) under AddressSanitizer and
// UndefinedBehaviorSanitizer.  Each records what it was given and launches
// nothing.
#include "ssba_common.h"
#include "stub_log.h"

std::vector<StubCall>& stub_calls() {
  static std::vector<StubCall> calls;
  return calls;
}

namespace ssba {

namespace {
hipError_t rec_index(const char* what, const IndexArgs& a) {
  stub_calls().push_back({what, a.index, a.qb, a.flags, nullptr, a.keep, a.f.sy, a.f.sx, 0});
  return hipSuccess;
}
hipError_t rec_attn(const char* what, const AttnArgs& a) {
  stub_calls().push_back({what, a.gated ? a.index_out : a.index, a.kb, a.flags, a.o, a.keep, a.f.sy, a.f.sx,
                          a.gated});
  return hipSuccess;
}
}  // namespace

hipError_t launch_pool(const IndexArgs& a, int, hipStream_t) { return rec_index("pool", a); }
hipError_t launch_pool_keys(const IndexArgs& a, hipStream_t) { return rec_index("pool_keys", a); }
// The rotary pre-pass: its pooled-key sums, rotated Q (in `out`) and the
// first inverse frequency's bits in `keep` (inv_freq[0] is 1).
hipError_t launch_rope_pool_keys(const RopeArgs& r, hipStream_t) {
  stub_calls().push_back({"rope", r.k_out, r.a.kb, nullptr, r.q_out, (int)r.inv_freq[0], r.a.f.sy, r.a.f.sx,
                          r.n_text_groups});
  return hipSuccess;
}
// One record per layer: its pooled-key slice, parity (in keep) and frame offsets.
hipError_t launch_pool_keys_layers(const PoolLayers& p, int n_layers, hipStream_t) {
  if (n_layers < 1 || n_layers > kPoolLayersMax) return hipErrorInvalidValue;
  for (int i = 0; i < n_layers; ++i) {
    const Frame& f = p.f[p.parity[i] & 1];
    stub_calls().push_back({"pool_keys_layers", p.k[i], p.kb[i], nullptr, nullptr, p.parity[i], f.sy, f.sx, 0});
  }
  return hipSuccess;
}
hipError_t launch_gate_topk(const IndexArgs& a, hipStream_t) { return rec_index("gate_topk", a); }
hipError_t launch_gate_topk_shared(const IndexArgs& a, hipStream_t) { return rec_index("gate_shared", a); }
hipError_t launch_gate_static(const IndexArgs& a, int, hipStream_t) { return rec_index("gate_static", a); }
// One record per layer: its index, pooled sums, flags, keep and frame offsets.
hipError_t launch_topk_shared_layers(const IndexLayers& p, int n_layers, hipStream_t) {
  if (n_layers < 1 || n_layers > kIndexLayersMax) return hipErrorInvalidValue;
  for (int i = 0; i < n_layers; ++i) {
    const Frame& f = p.f[p.parity[i] & 1];
    stub_calls().push_back({"shared_layers", p.index[i], p.qb[i], p.flags[i], p.srows[i], p.keep[i], f.sy, f.sx, 0});
  }
  return hipSuccess;
}
hipError_t launch_attn_bf16(const AttnArgs& a, int, int, hipStream_t) { return rec_attn("attn_bf16", a); }
hipError_t launch_attn_f32(const AttnArgs& a, int, int, hipStream_t) { return rec_attn("attn_f32", a); }
hipError_t launch_attn_mfma(const AttnArgs& a, int, int, hipStream_t) { return rec_attn("attn_mfma", a); }
// One record per layer, as rec_attn would make for that layer's own launch.
hipError_t launch_attn_mfma_layers(const AttnLayers& p, int n_layers, int, int, hipStream_t) {
  if (n_layers < 1 || n_layers > kAttnLayersMax) return hipErrorInvalidValue;
  for (int i = 0; i < n_layers; ++i) {
    const Frame& f = p.f[p.parity[i] & 1];
    if (p.a.gated)
      stub_calls().push_back({"attn_layers", p.index_out[i], p.kb[i], p.flags[i], p.o[i], p.keep[i], f.sy, f.sx, 1});
    else
      stub_calls().push_back({"attn_layers", p.index[i], nullptr, nullptr, p.o[i], 0, f.sy, f.sx, 0});
  }
  return hipSuccess;
}
hipError_t launch_backward(const BwdArgs& a, int, hipStream_t) {
  stub_calls().push_back({"backward", a.index, a.lse2, a.kmask, a.korder, 0, a.f.sy, a.f.sx, 0});
  return hipSuccess;
}

}  // namespace ssba
