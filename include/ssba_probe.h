/*
 * ssba_probe.h -- measurement helper of the SSBA library for AMD Instinct
 * MI355X (gfx950): the MFMA throughput the chip sustains in this process, as
 * the reference a kernel's measured rate is compared with (besides the
 * published 2.5 PFLOP/s dense bf16 peak, which assumes the 2.4 GHz clock).
 * Not part of the attention path.
 */
#ifndef SSBA_PROBE_H_
#define SSBA_PROBE_H_

#include "ssba.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Launches `blocks` workgroups of four waves; every wave issues `iters` x 8
 * v_mfma_f32_32x32x16_bf16 instructions (32768 flops each) on four
 * independent accumulator chains, with nothing else in the loop, and writes
 * one float per thread to `sink` (device memory of blocks * 256 floats,
 * owned by the caller; the values carry no meaning, they only keep the work
 * alive).  The caller times the launch on `hip_stream`; the work is
 * blocks * 4 * iters * 8 * 32768 flops.  Errors: SSBA_ERR_ARG for a NULL
 * sink or blocks, iters outside [1, 2^20]; SSBA_ERR_HIP if the launch
 * fails.  Asynchronous. */
ssba_status ssba_probe_mfma(int32_t blocks, int32_t iters, float* sink, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* SSBA_PROBE_H_ */
