/*
 * ssba_haar.h -- C ABI of the multi-level 2-D Haar transform pair of the Tiny
 * DWT-Distilled VAE (ElasticDiT, Section 2.3.1) for AMD Instinct MI355X
 * (gfx950), in the same library as ssba.h.
 *
 * The encoder injects a single 2-D Haar kernel bank {LL, HL, LH, HH} level
 * after level (the DWT equation: level l holds 4C channels at H/2^l x W/2^l);
 * the decoder inverts the pyramid, adding a residual to each reconstructed
 * level (the IWT equation).  The bank is the orthonormal Haar bank: for the
 * 2 x 2 cell a = x[2i][2j], b = x[2i][2j+1], c = x[2i+1][2j], d = x[2i+1][2j+1]
 *   LL = (a + b + c + d) / 2    HL = (a - b + c - d) / 2
 *   LH = (a + b - c - d) / 2    HH = (a - b - c + d) / 2
 * (HL high-pass along the width, LH along the height); the inverse uses the
 * same four combinations.  Arithmetic is fp32; bf16 tensors are rounded to
 * nearest even on store only, so level l is computed from the unrounded LL
 * of level l - 1 and the inverse rounds only its output.
 *
 * Layouts (contiguous, 16-byte aligned, dtype d->dtype):
 *   x:         [N][C][H][W]
 *   level l:   [N][4C][H >> l][W >> l], channel 4 c + band, bands in the
 *              order LL, HL, LH, HH (l = 1 .. levels)
 *   residual l (inverse only, optional): [N][C][H >> l][W >> l], added to the
 *              reconstruction of LL^(l); residual 0 is added to the output.
 * Ownership, streams and errors as in ssba.h: the caller owns every buffer,
 * calls are asynchronous on `hip_stream`, and every check happens before
 * anything is launched.
 */
#ifndef SSBA_HAAR_H_
#define SSBA_HAAR_H_

#include "ssba.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ssba_haar_desc {
  int32_t n, c, h, w;  /* input planes; h a multiple of 2^levels, w a multiple of 8 */
  int32_t levels;      /* 1 .. 3                                                  */
  int32_t dtype;       /* ssba_dtype of every tensor (SSBA_DT_BF16 or SSBA_DT_F32) */
} ssba_haar_desc;

/* Forward multi-level transform (the DWT equation): writes levels[l - 1] for
 * l = 1 .. d->levels.  Every level's four bands are stored, including the LL
 * band that the next level transforms further. */
ssba_status ssba_haar_dwt(const ssba_haar_desc* d, const void* x, void* const* levels,
                          void* hip_stream);

/* Inverse pyramid (the IWT equation): LL^(l-1) = IWT(LL^(l), HL^(l), LH^(l),
 * HH^(l)) + residual[l - 1] from l = d->levels down to 1, where only the
 * coarsest level's LL band and every level's HL, LH and HH bands are read;
 * writes LL^(0) to x.  `residuals` may be NULL, and so may any of its
 * d->levels entries (no residual at that level); all NULL inverts
 * ssba_haar_dwt up to fp32 rounding. */
ssba_status ssba_haar_iwt(const ssba_haar_desc* d, const void* const* levels,
                          const void* const* residuals, void* x, void* hip_stream);

/* Name of the kernel the forward (inverse = 0) or inverse (inverse = 1) call
 * launches, as profilers show it (e.g. "k_haar_dwt<unsigned short, 3>"); NULL
 * for an invalid descriptor.  Static storage; launches nothing. */
const char* ssba_haar_kernel_name(const ssba_haar_desc* d, int inverse);

#ifdef __cplusplus
}
#endif
#endif /* SSBA_HAAR_H_ */
