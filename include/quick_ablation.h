/*
 * quick_ablation.h -- ablation entry point of libquick.so (measurement of the
 * method's central design choice; not used by the GEMM entry points).
 *
 * The paper (Section 3.1, Section 3.2) argues that writing the dequantized
 * weights to shared memory (LDS) and loading them back as matrix-instruction
 * fragments -- the conventional mixed-precision GEMM design -- costs extra
 * LDS traffic and bank conflicts, and that loading the reordered weights
 * straight into the fragment registers removes it.  This entry point runs
 * the same 64 x 256 tiled kernel (data-parallel, one workgroup per tile) in
 * three forms so the difference can be measured on gfx950:
 *   mode 0  dequantized weights go straight to the fragment registers
 *           (the method; identical to the library's 64 x 32 tiled kernel);
 *   mode 1  each wave first writes its k-group of dequantized weights to an
 *           LDS tile [column][channel] with rows padded by 16 bytes, then
 *           reads the fragments back (conflict-free write-back);
 *   mode 2  the same with unpadded 256-byte rows, so the 16 columns of a
 *           fragment access fall on the same LDS banks (naive write-back).
 * All three compute the same result as quick_w4a16_gemm (the fragments hold
 * the same binary16 values).
 */
#ifndef QUICK_ABLATION_H
#define QUICK_ABLATION_H

#include <stdint.h>

#include "quick.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Arguments, layouts, alignment and errors as quick_w4a16_gemm (group fixed
 * at 128); `mode` 0, 1 or 2 as above (INVALID_ARG otherwise).  Uses no
 * workspace; asynchronous on `stream`. */
int quick_ablation_gemm(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
                        int64_t M, int64_t N, int64_t K, int mode, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QUICK_ABLATION_H */
