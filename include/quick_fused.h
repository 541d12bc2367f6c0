/*
 * quick_fused.h -- W4A16 GEMMs of libquick.so with a fused output epilogue.
 *
 * The GEMM is that of quick_w4a16_gemm (paper, Section 2.1 and Section 2.3:
 * W = (q - z) * s per group of 128 input channels, y = x . W, weights
 * reordered offline as in Section 3.1 and Section 3.2).  The epilogue is
 * applied to the fp32 accumulators before the single rounding to f16, so a
 * bias add or the gated activation of a feed-forward layer costs no extra
 * pass over y and no intermediate rounding:
 *   h[m][n] = x . W [m][n] + bias[n]                      (bias optional)
 *   QUICK_ACT_NONE:       y[m][n] = h[m][n]                (y: M x N)
 *   QUICK_ACT_SILU_GATE:  y[m][16t + i] = silu(h[m][32t + i]) * h[m][32t + 16 + i]
 *                         for i < 16                       (y: M x N/2)
 * with silu(a) = a / (1 + e^-a) in fp32.  The gated form expects a fused
 * gate/up weight matrix whose packed columns alternate in 16-column tiles,
 * gate tile t at columns 32t .. 32t+15 and the matching up tile at
 * 32t+16 .. 32t+31; quick_interleave_gate_up builds that column order from
 * the two unpacked matrices before quick_pack_weights.
 */
#ifndef QUICK_FUSED_H
#define QUICK_FUSED_H

#include <stddef.h>
#include <stdint.h>

#include "quick.h"

#ifdef __cplusplus
extern "C" {
#endif

#define QUICK_ACT_NONE 0
#define QUICK_ACT_SILU_GATE 1

typedef struct quick_epilogue {
    const void* bias;  /* device, f16 [N] in packed column order (grouped:
                          [E][N], expert e's at e*N), 8-byte aligned; NULL =
                          no bias                                            */
    int activation;    /* QUICK_ACT_NONE or QUICK_ACT_SILU_GATE              */
} quick_epilogue_t;

/* quick_w4a16_gemm_ex with an epilogue (epi NULL = none).  With
 * QUICK_ACT_SILU_GATE, N (the packed columns) must be a multiple of 32
 * (SHAPE otherwise) and y is M x N/2.  The gated form needs each gate tile
 * and its up tile in one wave: an automatic configuration is adjusted for
 * it; an explicit cfg that cannot hold them (stream kernel with one n-tile
 * per wave, tiled kernel with 16-column waves and no K split) is
 * INVALID_ARG, as is the reserved variant 4.
 * The workspace a caller passes must hold quick_fused_workspace_bytes().
 * Other arguments, errors and the workspace contract as quick_w4a16_gemm_ex;
 * also INVALID_ARG for an unknown activation, ALIGNMENT for the bias. */
int quick_w4a16_gemm_fused(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
                           int64_t M, int64_t N, int64_t K, int64_t group, void* stream,
                           const quick_epilogue_t* epi, const quick_config_t* cfg, void* workspace,
                           size_t workspace_bytes);

/* quick_w4a16_grouped_gemm_ex (quick_grouped.h) with an epilogue; the bias
 * is per expert ([E][N]).  A bias with an explicit split-K configuration
 * (variant 2, split_k > 1) is INVALID_ARG: the split-K reduction pass does
 * not know a row's expert. */
int quick_w4a16_grouped_gemm_fused(const void* x, const int32_t* rows, const int32_t* offsets, const void* packed,
                                   const void* scales, const void* zeros, void* y, int64_t T, int64_t R, int64_t E,
                                   int64_t N, int64_t K, int64_t group, void* stream, const quick_epilogue_t* epi,
                                   const quick_config_t* cfg, void* workspace, size_t workspace_bytes);

/* Workspace bytes the two calls above need (0 when none, or for invalid
 * arguments). */
size_t quick_fused_workspace_bytes(int64_t M, int64_t N, int64_t K, const quick_config_t* cfg,
                                   const quick_epilogue_t* epi);
size_t quick_grouped_fused_workspace_bytes(int64_t R, int64_t E, int64_t N, int64_t K, const quick_config_t* cfg,
                                           const quick_epilogue_t* epi);

/* Host, offline: the K x 2*Nh column order the gated form expects, from the
 * unpacked gate and up matrices (each q [K][Nh], z and s [K/group][Nh], in
 * the layouts quick_pack_weights takes).  Output column 32t + i is gate
 * column 16t + i for i < 16 and up column 16t + i - 16 otherwise; q, z, s
 * (caller-owned, [K][2Nh] and [K/group][2Nh]) are fully overwritten.
 * Errors: INVALID_ARG (NULL), UNSUPPORTED (group != 128), SHAPE (K % 128,
 * Nh % 16, non-positive sizes). */
int quick_interleave_gate_up(const uint8_t* q_gate, const uint8_t* z_gate, const uint16_t* s_gate,
                             const uint8_t* q_up, const uint8_t* z_up, const uint16_t* s_up, int64_t K, int64_t Nh,
                             int64_t group, uint8_t* q, uint8_t* z, uint16_t* s);

#ifdef __cplusplus
}
#endif

#endif /* QUICK_FUSED_H */
