/*
 * quick_grouped.h -- grouped (mixture-of-experts) W4A16 GEMM of libquick.so.
 *
 * A mixture-of-experts feed-forward layer applies, to every routed token
 * row, the weights of the expert the row was routed to.  Per element this is
 * the same operation as quick_w4a16_gemm (paper, Section 2.1 and
 * Section 2.3: W = (q - z) * s per group of 128 input channels, y = x . W,
 * with the weights reordered offline as in Section 3.1 and Section 3.2), but
 * over E weight matrices in one launch, so that all experts' tiles share the
 * chip instead of one small GEMM per expert.  The routed rows are gathered
 * from the token activations inside the kernel's activation load, and the
 * per-expert row counts are read from device memory by the kernel itself
 * (no host synchronization to learn them).
 *
 * Results are those of quick_w4a16_gemm applied expert by expert to the
 * gathered rows: fp32 accumulation, one final round-to-nearest-even to f16,
 * each weight dequantized with a single rounding; deterministic run to run.
 */
#ifndef QUICK_GROUPED_H
#define QUICK_GROUPED_H

#include <stddef.h>
#include <stdint.h>

#include "quick.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Most experts one call accepts. */
#define QUICK_MAX_EXPERTS 512

/* y[r][:] = x[rows[r]][:] . W_e  for every routed row r, where e is the
 * expert with offsets[e] <= r < offsets[e+1].
 *   x        device, f16 [T][K] token activations, 16-byte aligned
 *   rows     device, int32 [R] token row of each routed row (0 <= rows[r] < T),
 *            4-byte aligned; NULL means rows[r] = r (then T >= R)
 *   offsets  device, int32 [E+1], non-decreasing, offsets[0] = 0,
 *            offsets[E] = R; expert e owns routed rows offsets[e] ..
 *            offsets[e+1]-1 (an expert may own none), 4-byte aligned
 *   packed, scales, zeros
 *            device, the E experts' packed buffers from quick_pack_weights
 *            (each expert K x N) stored back to back: expert e's packed
 *            weights start at byte e*K*N/2, its scales at e*K*N/64 and its
 *            zero points at e*K*N/256; alignment as quick_w4a16_gemm
 *   y        device, f16 [R][N], 8-byte aligned; must not overlap the inputs
 *   T, R, E  token rows of x, routed rows (rows of y), experts (1..512)
 *   N, K     every expert's output columns and input channels (N % 16 == 0,
 *            K % 128 == 0); group must be 128
 * R == 0 is a valid no-op.  Asynchronous on `stream` (hipStream_t as void*,
 * NULL = default stream); the library's internal workspace is used as by
 * quick_w4a16_gemm (including its graph-capture rule).  When the automatic choice takes 128-row tiles (about
 * 96 or more routed rows per expert), the GEMM runs as two launches on
 * `stream`: each expert's whole 128-row tiles, and a remainder of at least
 * 64 rows, with those tiles; then the shorter remainders with 32-row tiles,
 * so that a remainder of a few rows does not pay for a full-height tile.  rows and offsets are read on the device only: values
 * that break the contract above (out-of-range tokens or offsets,
 * decreasing offsets) are clamped into range, so the kernel stays inside
 * every buffer, but the affected rows of y are then unspecified.
 * Errors (checked before anything is enqueued): INVALID_ARG (NULL buffer),
 * SHAPE (negative sizes, E outside 1..512, K or N not multiples, T == 0 with
 * R > 0, rows NULL with T < R, 32-bit limits as quick_w4a16_gemm per
 * expert), UNSUPPORTED (group != 128), ALIGNMENT, HIP, CAPTURE. */
int quick_w4a16_grouped_gemm(const void* x, const int32_t* rows, const int32_t* offsets, const void* packed,
                             const void* scales, const void* zeros, void* y, int64_t T, int64_t R, int64_t E,
                             int64_t N, int64_t K, int64_t group, void* stream);

/* Same with an explicit kernel choice and optional caller workspace (same
 * workspace contract as quick_w4a16_gemm_ex).  cfg: variant 0 = automatic,
 * 2 = one workgroup per (tile, K slice) with split_k K slices (0 = 1),
 * 3 = stream-K over split_k resident workgroups (a multiple of 8, 0 = all
 * resident); (tile_m, tile_n) one of (16, 16), (16, 32), (32, 16),
 * (32, 32), (64, 32), (128, 32), 0 = automatic; variant 1 (the stream
 * kernel) is not available here (INVALID_ARG).  A cfg with every field 0
 * is the automatic choice (including its two-launch form); any other cfg
 * runs as one launch. */
int quick_w4a16_grouped_gemm_ex(const void* x, const int32_t* rows, const int32_t* offsets, const void* packed,
                                const void* scales, const void* zeros, void* y, int64_t T, int64_t R, int64_t E,
                                int64_t N, int64_t K, int64_t group, void* stream, const quick_config_t* cfg,
                                void* workspace, size_t workspace_bytes);

/* Workspace bytes quick_w4a16_grouped_gemm_ex needs (cfg NULL = automatic
 * choice; for its two-launch form, the larger of the two launches' needs);
 * 0 when none, or for invalid arguments. */
size_t quick_grouped_workspace_bytes(int64_t R, int64_t E, int64_t N, int64_t K, const quick_config_t* cfg);

/* The automatic choice for R routed rows over E experts (for the two-launch
 * form, the first launch's configuration).
 * Errors: INVALID_ARG (NULL cfg), SHAPE. */
int quick_grouped_select_config(int64_t R, int64_t E, int64_t N, int64_t K, quick_config_t* cfg);

#ifdef __cplusplus
}
#endif

#endif /* QUICK_GROUPED_H */
