// ssba_forward_topk_noalloc: the top-k gate and attention call
// (ssba_forward_topk) with its scratch taken from a fixed device array instead
// of a caller buffer, for callers that cannot allocate device memory.
//
// The array lives in this file.  Each device holds its own copy, from module
// load until the process ends; its device address is looked up once per
// device (hipGetSymbolAddress, with that device current) and cached.  The
// name of the array is a host-side stand-in, never a device address: only the
// looked-up pointer reaches the kernels.  No part of the scratch has to start
// at zero (the pooling kernel writes every pooled sum, the gate every status
// flag), so nothing is cleared.  Calls that overlap on one device share the
// array and race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ssba.h"

namespace {

constexpr size_t kScratchBytes = SSBA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_lock;
void* g_ptr[kMaxDevices];   // device address of `scratch` per device, once looked up

// Device address of this device's array (looked up on first use).
ssba_status device_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SSBA_ERR_HIP;
  std::lock_guard<std::mutex> guard(g_lock);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SSBA_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return SSBA_OK;
}

}  // namespace

extern "C" {

ssba_status ssba_forward_topk_noalloc(const ssba_desc* d, const void* q, const void* k, const void* v,
                                      int32_t* index, size_t index_bytes, void* o, void* hip_stream) {
  size_t need = 0;
  ssba_status st = ssba_workspace_size(d, nullptr, &need);
  if (st != SSBA_OK) return st;
  if (d->gate != SSBA_GATE_TOPK && d->gate != SSBA_GATE_TOPK_SHARED) return SSBA_ERR_ARG;
  if (need > kScratchBytes) return SSBA_ERR_WORKSPACE;
  void* s = nullptr;
  st = device_scratch(&s);
  if (st != SSBA_OK) return st;
  return ssba_forward_topk_ex(d, q, k, v, index, index_bytes, s, kScratchBytes, o, hip_stream);
}

}  // extern "C"
