// Call log of the recording launcher stand-ins (tests/sanitize/stub_launch.cpp).
#pragma once

#include <vector>

struct StubCall {
  const char* what;       // launcher name
  const void* index;      // index read or written (the layer pre-pass: the keys pooled)
  const void* scratch;    // pooled sums (q for the gates, k for the attention and the layer pre-pass), backward lse2
  const void* flags;      // status flags (gates) / kept-block masks (backward)
  const void* out;        // attention output (backward: the key-side order)
  int keep, sy, sx, gated;
};

std::vector<StubCall>& stub_calls();
