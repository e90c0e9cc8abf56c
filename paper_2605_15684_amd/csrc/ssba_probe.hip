// MFMA throughput probe (measurement helper, not part of the attention path):
// back-to-back v_mfma_f32_32x32x16_bf16 on four independent accumulator
// chains per wave, four waves per workgroup.
#include <hip/hip_runtime.h>

#include "ssba_probe.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__global__ void __launch_bounds__(256) k_probe_mfma(int iters, float* sink) {
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)((threadIdx.x + e) & 15));
    b[e] = (__bf16)(1e-3f * (float)((threadIdx.x * 3 + e) & 15));
  }
  floatx16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = floatx16{};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j & 3], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" ssba_status ssba_probe_mfma(int32_t blocks, int32_t iters, float* sink, void* hip_stream) {
  if (!sink || blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 20)) return SSBA_ERR_ARG;
  hipLaunchKernelGGL(k_probe_mfma, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(hip_stream),
                     iters, sink);
  return hipGetLastError() == hipSuccess ? SSBA_OK : SSBA_ERR_HIP;
}
