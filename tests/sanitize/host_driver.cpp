// Exercises the host layer of the SSBA library (argument checks, workspace
// arithmetic, dispatch and the layer-stack driver) with the kernel launchers
// replaced by recording stand-ins.  Built for the CPU under AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_host_sanitize.py.  Prints "ok"
// and exits 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "ssba.h"
#include "stub_log.h"

#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
      return 1;                                                          \
    }                                                                    \
  } while (0)

namespace {

ssba_desc base_desc() {
  ssba_desc d;
  std::memset(&d, 0, sizeof d);
  d.batch = 1;
  d.heads = 16;
  d.head_dim = 64;
  d.grid_h = 64;
  d.grid_w = 64;
  d.tile = 8;
  d.shift_y = 4;
  d.shift_x = 4;
  d.gate = SSBA_GATE_TOPK;
  d.keep = 10;
  d.win_h = 1;
  d.win_w = 1;
  d.dtype = SSBA_DT_BF16;
  return d;
}

// Real host memory, so an access the library made through these pointers
// (it must make none) would be seen by the address sanitizer.
struct Buffers {
  std::vector<uint64_t> q, k, v, o, index, scratch;
  explicit Buffers(size_t tensor_bytes, size_t index_bytes, size_t scratch_bytes)
      : q(tensor_bytes / 8 + 2), k(tensor_bytes / 8 + 2), v(tensor_bytes / 8 + 2), o(tensor_bytes / 8 + 2),
        index(index_bytes / 8 + 2), scratch(scratch_bytes / 8 + 2) {}
};

uint64_t rng_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {
  rng_state ^= rng_state << 13;
  rng_state ^= rng_state >> 7;
  rng_state ^= rng_state << 17;
  return rng_state;
}
int32_t pick(const int32_t* v, int n) { return v[next() % (uint64_t)n]; }

}  // namespace

int main() {
  CHECK(ssba_abi_version() == SSBA_ABI_VERSION);
  for (int s = 0; s < 8; ++s) CHECK(ssba_status_str((ssba_status)s) != nullptr);

  // ---- workspace sizes against their stated formulas ----------------------
  {
    const int32_t tiles[] = {4, 8, 16};
    const int32_t dims[] = {64, 128};
    const int32_t gates[] = {SSBA_GATE_TOPK, SSBA_GATE_WINDOW, SSBA_GATE_DENSE, SSBA_GATE_TOPK_SHARED};
    for (int n = 0; n < 400; ++n) {
      ssba_desc d = base_desc();
      d.batch = 1 + (int32_t)(next() % 4);
      d.heads = 1 + (int32_t)(next() % 24);
      d.tile = pick(tiles, 3);
      d.head_dim = pick(dims, 2);
      d.grid_h = d.tile * (1 + (int32_t)(next() % 8));
      d.grid_w = d.tile * (1 + (int32_t)(next() % 8));
      d.n_text = (int32_t)(next() % 300);
      d.gate = pick(gates, 4);
      const size_t tb = (size_t)(d.grid_h / d.tile) * (size_t)(d.grid_w / d.tile);
      d.keep = 1 + (int32_t)(next() % tb);
      size_t ib = 0, sb = 0;
      CHECK(ssba_workspace_size(&d, &ib, &sb) == SSBA_OK);
      const size_t rows = (size_t)d.batch * d.heads * tb;
      CHECK(ib == 4 * rows * (tb + 1));
      size_t want = 4 * rows;
      if (d.gate == SSBA_GATE_TOPK || d.gate == SSBA_GATE_TOPK_SHARED) want += 16 * rows * d.head_dim;
      if (d.gate == SSBA_GATE_TOPK_SHARED) want += 8 * rows * tb;
      CHECK(sb == want);
    }
  }

  // ---- each entry point: arguments, short buffers, exact buffers ----------
  ssba_desc d = base_desc();
  size_t ib = 0, sb = 0;
  CHECK(ssba_workspace_size(&d, &ib, &sb) == SSBA_OK);
  const size_t tensor = (size_t)16 * 4096 * 64 * 2;
  {
    Buffers b(tensor, ib, sb);
    int32_t* idx = reinterpret_cast<int32_t*>(b.index.data());
    void* scr = b.scratch.data();
    stub_calls().clear();
    CHECK(ssba_build_index_ex(&d, b.q.data(), b.k.data(), idx, ib - 1, scr, sb, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_build_index_ex(&d, b.q.data(), b.k.data(), idx, ib, scr, sb - 4, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(stub_calls().empty());
    CHECK(ssba_build_index_ex(&d, b.q.data(), b.k.data(), idx, ib, scr, sb, nullptr) == SSBA_OK);
    CHECK(stub_calls().size() == 2);
    CHECK(std::strcmp(stub_calls()[0].what, "pool") == 0 && std::strcmp(stub_calls()[1].what, "gate_topk") == 0);
    // flags follow the pooled sums: 16 * B * H * T_b * D bytes in
    CHECK(stub_calls()[1].flags == static_cast<char*>(scr) + (size_t)16 * 16 * 64 * 64);
    CHECK(stub_calls()[1].index == idx);

    stub_calls().clear();
    CHECK(ssba_forward_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib - 1, b.o.data(), nullptr) ==
          SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib, b.o.data(), nullptr) == SSBA_OK);
    CHECK(stub_calls().size() == 1 && stub_calls()[0].out == b.o.data());

    stub_calls().clear();
    CHECK(ssba_forward_topk_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib, scr, sb - 1, b.o.data(),
                               nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_topk_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib, scr, sb, b.o.data(), nullptr) ==
          SSBA_OK);
    CHECK(stub_calls().size() == 2 && stub_calls()[1].gated == 1 && stub_calls()[1].index == idx);
    // the fused call pools the keys only; the attention kernel gets their sums
    CHECK(std::strcmp(stub_calls()[0].what, "pool_keys") == 0);
    CHECK(stub_calls()[1].scratch == static_cast<char*>(scr) + (size_t)8 * 16 * 64 * 64);

    // the same two launches one at a time
    stub_calls().clear();
    CHECK(ssba_pool_keys_ex(&d, b.k.data(), scr, sb - 1, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_gated_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib - 1, scr, sb, b.o.data(),
                                nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(stub_calls().empty());
    CHECK(ssba_pool_keys_ex(&d, b.k.data(), scr, sb, nullptr) == SSBA_OK);
    CHECK(ssba_forward_gated_ex(&d, b.q.data(), b.k.data(), b.v.data(), idx, ib, scr, sb, b.o.data(), nullptr) ==
          SSBA_OK);
    CHECK(stub_calls().size() == 2 && std::strcmp(stub_calls()[0].what, "pool_keys") == 0);
    CHECK(stub_calls()[1].gated == 1 && stub_calls()[1].index == idx &&
          stub_calls()[1].scratch == static_cast<char*>(scr) + (size_t)8 * 16 * 64 * 64);

    // the rotary form: pre-pass, then the gated attention on the rotated Q and K
    {
      Buffers rb(tensor, 0, 0);
      stub_calls().clear();
      CHECK(ssba_forward_topk_rope_ex(&d, b.q.data(), b.k.data(), b.v.data(), rb.q.data(), rb.k.data(), 0.f, idx,
                                      ib, scr, sb - 1, b.o.data(), nullptr) == SSBA_ERR_WORKSPACE);
      const float nan = std::numeric_limits<float>::quiet_NaN();
      CHECK(ssba_forward_topk_rope_ex(&d, b.q.data(), b.k.data(), b.v.data(), rb.q.data(), rb.k.data(), nan, idx,
                                      ib, scr, sb, b.o.data(), nullptr) == SSBA_ERR_ARG);
      CHECK(ssba_rope_pool_keys_ex(&d, b.q.data(), b.k.data(), nullptr, rb.k.data(), 0.f, scr, sb, nullptr) ==
            SSBA_ERR_ARG);
      CHECK(stub_calls().empty());
      CHECK(ssba_forward_topk_rope_ex(&d, b.q.data(), b.k.data(), b.v.data(), rb.q.data(), rb.k.data(), 0.f, idx,
                                      ib, scr, sb, b.o.data(), nullptr) == SSBA_OK);
      CHECK(stub_calls().size() == 2 && std::strcmp(stub_calls()[0].what, "rope") == 0);
      CHECK(stub_calls()[0].out == rb.q.data() && stub_calls()[0].index == rb.k.data());
      CHECK(stub_calls()[0].scratch == static_cast<char*>(scr) + (size_t)8 * 16 * 64 * 64);
      CHECK(stub_calls()[0].keep == 1 && stub_calls()[0].gated == 0);   // inv_freq[0] = 1, no text rows
      CHECK(stub_calls()[1].gated == 1 && stub_calls()[1].index == idx &&
            stub_calls()[1].scratch == stub_calls()[0].scratch);
    }

    // misaligned and missing pointers
    CHECK(ssba_forward_ex(&d, static_cast<char*>(static_cast<void*>(b.q.data())) + 2, b.k.data(), b.v.data(), idx,
                          ib, b.o.data(), nullptr) == SSBA_ERR_ARG);
    CHECK(ssba_forward_topk_ex(&d, nullptr, b.k.data(), b.v.data(), idx, ib, scr, sb, b.o.data(), nullptr) ==
          SSBA_ERR_ARG);
    ssba_status st;
    CHECK(ssba_read_device_status_ex(&d, scr, sb - 1, &st, nullptr) == SSBA_ERR_WORKSPACE);
  }

  // ---- backward ------------------------------------------------------------
  {
    size_t bsb = 0;
    CHECK(ssba_backward_workspace_size(&d, &bsb) == SSBA_OK);
    const size_t up = (4 * 16 * 4096 + 255) / 256 * 256;
    const size_t mask_bytes = (8 * 16 * 64 + 255) / 256 * 256;
    CHECK(bsb == 2 * up + mask_bytes + (4 * 16 * 64 + 255) / 256 * 256);
    Buffers b(tensor, ib, bsb + 256);
    // 256-byte aligned scratch inside the vector
    char* raw = reinterpret_cast<char*>(b.scratch.data());
    void* scr = raw + (256 - reinterpret_cast<uintptr_t>(raw) % 256) % 256;
    int32_t* idx = reinterpret_cast<int32_t*>(b.index.data());
    std::vector<float> lse(16 * 4096);
    stub_calls().clear();
    CHECK(ssba_backward_ex(&d, b.q.data(), b.k.data(), b.v.data(), b.o.data(), b.o.data(), lse.data(), idx, ib,
                           b.q.data(), b.k.data(), b.v.data(), scr, bsb - 1, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_backward_ex(&d, b.q.data(), b.k.data(), b.v.data(), b.o.data(), b.o.data(), lse.data(), idx, ib,
                           b.q.data(), b.k.data(), b.v.data(), scr, bsb, nullptr) == SSBA_OK);
    CHECK(stub_calls().size() == 1 && stub_calls()[0].scratch == scr);
    CHECK(stub_calls()[0].flags == static_cast<char*>(scr) + 2 * up);
    CHECK(stub_calls()[0].out == static_cast<char*>(scr) + 2 * up + mask_bytes);
  }

  // ---- layer stack: slices, offsets, skipped layers, index cache ----------
  {
    const int L = 5;
    size_t lib = 0, lsb = 0;
    CHECK(ssba_layers_workspace_size(&d, L, &lib, &lsb) == SSBA_OK);
    CHECK(lib == (size_t)L * ib);
    const size_t stride = lsb / L;
    CHECK(stride % 256 == 0 && stride >= sb);
    Buffers b(tensor, lib, lsb);
    ssba_layer layers[L];
    std::memset(layers, 0, sizeof layers);
    for (int l = 0; l < L; ++l) {
      layers[l].q = b.q.data();
      layers[l].k = b.k.data();
      layers[l].v = b.v.data();
      layers[l].o = b.o.data();
      layers[l].keep = 3 + l;
    }
    layers[2].skip = 1;
    int32_t* idx = reinterpret_cast<int32_t*>(b.index.data());
    char* scr = reinterpret_cast<char*>(b.scratch.data());
    stub_calls().clear();
    CHECK(ssba_forward_layers_ex(&d, layers, L, idx, lib - 1, scr, lsb, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(ssba_forward_layers_ex(&d, layers, L, idx, lib, scr, lsb - 1, nullptr) == SSBA_ERR_WORKSPACE);
    CHECK(stub_calls().empty());
    CHECK(ssba_forward_layers_ex(&d, layers, L, idx, lib, scr, lsb, nullptr) == SSBA_OK);
    // four layers ran: one pooling launch over their keys, then one gated
    // attention launch over the same layers
    CHECK(stub_calls().size() == 8);
    const int ran[] = {0, 1, 3, 4};
    const size_t pooled = (size_t)8 * 16 * 64 * 64;   // the pooled key sums follow 8 B H T_b D bytes of q sums
    for (int i = 0; i < 4; ++i) {
      const int l = ran[i];
      const StubCall& pre = stub_calls()[i];
      CHECK(std::strcmp(pre.what, "pool_keys_layers") == 0 && pre.index == layers[l].k);
      CHECK(pre.scratch == scr + (size_t)l * stride + pooled && pre.keep == (l & 1));
      const StubCall& att = stub_calls()[4 + i];
      CHECK(std::strcmp(att.what, "attn_layers") == 0 && att.out == layers[l].o);
      CHECK(att.gated == 1 && att.keep == 3 + l);
      CHECK(att.flags == scr + (size_t)l * stride + 2 * pooled);
      CHECK(att.index == idx + (size_t)l * (ib / 4));
      CHECK(att.scratch == pre.scratch);
      // offsets alternate sign: +4 on even layers, -4 (reduced: 60) on odd ones
      CHECK(att.sy == ((l & 1) ? 60 : 4) && att.sx == att.sy);
      CHECK(pre.sy == att.sy && pre.sx == att.sx);
    }
    // more layers than one pre-pass launch takes: launches of at most 32
    {
      const int LL = 70;
      size_t lib2 = 0, lsb2 = 0;
      CHECK(ssba_layers_workspace_size(&d, LL, &lib2, &lsb2) == SSBA_OK);
      Buffers b2(tensor, lib2, lsb2);
      std::vector<ssba_layer> many(LL);
      for (int l = 0; l < LL; ++l) {
        many[l] = layers[0];
        many[l].keep = 1 + l % 64;
        many[l].skip = (l % 5 == 4) ? 1 : 0;
      }
      stub_calls().clear();
      CHECK(ssba_forward_layers_ex(&d, many.data(), LL, reinterpret_cast<int32_t*>(b2.index.data()), lib2,
                                   b2.scratch.data(), lsb2, nullptr) == SSBA_OK);
      int pre = 0, att = 0, run = 0, longest = 0;
      for (const StubCall& c : stub_calls()) {
        if (std::strcmp(c.what, "pool_keys_layers") == 0) {
          ++pre;
          ++run;
          longest = run > longest ? run : longest;
        } else {
          ++att;
          run = 0;
        }
      }
      CHECK(pre == 56 && att == 56 && longest == 32);
    }
    // static gate: the index is built once per offset parity
    ssba_desc w = d;
    w.gate = SSBA_GATE_WINDOW;
    w.win_h = 2;
    w.win_w = 2;
    size_t wib = 0, wsb = 0;
    CHECK(ssba_layers_workspace_size(&w, L, &wib, &wsb) == SSBA_OK);
    stub_calls().clear();
    CHECK(ssba_forward_layers_ex(&w, layers, L, idx, wib, scr, wsb, nullptr) == SSBA_OK);
    int gates = 0, attn = 0;
    for (const StubCall& c : stub_calls()) {
      if (std::strcmp(c.what, "gate_static") == 0) ++gates;
      if (std::strncmp(c.what, "attn", 4) == 0) {
        ++attn;
        CHECK(c.index == idx || c.index == idx + wib / L / 4);   // the slices of layers 0 and 1
      }
    }
    CHECK(gates == 2 && attn == 4);
    // head-shared top-k gate: one launch group builds every running layer's
    // index in its own slice, then one attention launch reads them
    ssba_desc sh = d;
    sh.gate = SSBA_GATE_TOPK_SHARED;
    size_t sib = 0, ssb = 0;
    CHECK(ssba_layers_workspace_size(&sh, L, &sib, &ssb) == SSBA_OK);
    Buffers bs(tensor, sib, ssb);
    int32_t* sidx = reinterpret_cast<int32_t*>(bs.index.data());
    char* sscr = reinterpret_cast<char*>(bs.scratch.data());
    stub_calls().clear();
    CHECK(ssba_forward_layers_ex(&sh, layers, L, sidx, sib, sscr, ssb, nullptr) == SSBA_OK);
    CHECK(stub_calls().size() == 8);
    const size_t sstride = ssb / L;
    for (int i = 0; i < 4; ++i) {
      const int l = ran[i];
      const StubCall& g = stub_calls()[i];
      CHECK(std::strcmp(g.what, "shared_layers") == 0 && g.keep == 3 + l);
      CHECK(g.index == sidx + (size_t)l * (sib / L / 4) && g.scratch == sscr + (size_t)l * sstride);
      // q sums, k sums, then the per-head rows (8 B H T_b T_b), then the flags
      CHECK(g.out == sscr + (size_t)l * sstride + 2 * pooled);
      CHECK(g.flags == sscr + (size_t)l * sstride + 2 * pooled + (size_t)8 * 16 * 64 * 64);
      CHECK(g.sy == ((l & 1) ? 60 : 4));
      const StubCall& att = stub_calls()[4 + i];
      CHECK(std::strcmp(att.what, "attn_layers") == 0 && att.gated == 0);
      CHECK(att.index == g.index && att.out == layers[l].o && att.sy == g.sy);
    }
  }

  // ---- descriptors at the edges: rejected or sized without wrapping -------
  {
    const int32_t big[] = {1, 2, 7, 64, 1 << 15, 1 << 20, 1 << 30, 2147483647, 0, -1, -2147483647 - 1};
    const int32_t tiles[] = {4, 8, 16, 3, 0, -8};
    const int32_t dims[] = {64, 128, 96, 0};
    for (int n = 0; n < 20000; ++n) {
      ssba_desc e = base_desc();
      e.batch = pick(big, 11);
      e.heads = pick(big, 11);
      e.tile = pick(tiles, 6);
      e.head_dim = pick(dims, 4);
      e.grid_h = pick(big, 11);
      e.grid_w = pick(big, 11);
      e.n_text = pick(big, 11);
      e.shift_y = pick(big, 11);
      e.shift_x = pick(big, 11);
      e.keep = pick(big, 11);
      e.gate = (int32_t)(next() % 5);
      e.win_h = pick(big, 11);
      e.win_w = pick(big, 11);
      if (next() % 2) {
        e.stride_b = (int64_t)pick(big, 11);
        e.stride_h = (int64_t)pick(big, 11);
        e.stride_t = (int64_t)pick(big, 11) * 8;
      }
      size_t eib = 0, esb = 0;
      const ssba_status st = ssba_workspace_size(&e, &eib, &esb);
      if (st != SSBA_OK) continue;
      // accepted: the sizes are the formulas evaluated without wrapping
      const long double tb = (long double)(e.grid_h / e.tile) * (long double)(e.grid_w / e.tile);
      const long double rows = (long double)e.batch * e.heads * tb;
      CHECK((long double)eib == 4.0L * rows * (tb + 1.0L));
      CHECK((long double)esb >= 4.0L * rows);
      // and a one-byte-short index is rejected by every index consumer
      stub_calls().clear();
      void* fake = reinterpret_cast<void*>(static_cast<uintptr_t>(0x100000));
      CHECK(ssba_forward_ex(&e, fake, fake, fake, static_cast<int32_t*>(fake), eib - 1, fake, nullptr) !=
            SSBA_OK);
      CHECK(stub_calls().empty());
    }
  }

  std::printf("ok\n");
  return 0;
}
