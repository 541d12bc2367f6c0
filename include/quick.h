/*
 * quick.h -- C ABI of the MI355X (gfx950) W4A16 mixed-precision GEMM library.
 *
 * The operation (paper, Section 2.1 and Section 2.3): weights are stored as
 * 4-bit unsigned integers q with one zero point z (4-bit) and one scale s
 * (binary16) per group of 128 consecutive input channels of an output
 * column; they are dequantized to W = (q - z) * s and multiplied by binary16
 * activations x, y = x . W.  Following Section 3.1 and Section 3.2 the static
 * weights are reordered once, offline (quick_pack_weights), so that the GEMM
 * kernels load them from memory straight into the registers of the gfx950
 * matrix-instruction operand and dequantize them there, without ever writing
 * dequantized weights to shared memory (LDS).
 *
 * Conventions shared by every entry point:
 *  - Every function returns a quick status code (QUICK_OK == 0) and never
 *    throws.  All validation happens before any write or launch: on an error
 *    nothing has been written and nothing has been enqueued.
 *  - Every buffer is owned by the caller.  The library keeps no pointer to a
 *    caller buffer after the call returns.
 *  - Matrices are dense and row-major.  "f16" means IEEE binary16 bit
 *    patterns stored in uint16_t.
 *  - Only group == 128 is supported (QUICK_ERR_UNSUPPORTED otherwise);
 *    K must be a multiple of 128 and N a multiple of 16 (QUICK_ERR_SHAPE).
 *  - 32-bit limits (the kernels address their buffers with 32-bit offsets):
 *    packed weights K*N/2 < 2^32 bytes, M*K < 2^31 activation elements,
 *    M*N < 2^31 output elements and M <= 2^24; larger shapes are
 *    QUICK_ERR_SHAPE.
 */
#ifndef QUICK_H
#define QUICK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define QUICK_OK 0
#define QUICK_ERR_INVALID_ARG 1  /* null pointer, bad config field          */
#define QUICK_ERR_SHAPE 2        /* M < 0, K % 128, N % 16, K or N <= 0,
                                    a 32-bit limit exceeded                  */
#define QUICK_ERR_UNSUPPORTED 3  /* group != 128                             */
#define QUICK_ERR_RANGE 4        /* a q or z value above 15                  */
#define QUICK_ERR_ALIGNMENT 5    /* device pointer not aligned (see below)   */
#define QUICK_ERR_HIP 6          /* HIP runtime error (launch, allocation)   */
#define QUICK_ERR_WORKSPACE 7    /* caller workspace missing or too small    */
#define QUICK_ERR_IO 8           /* tune table file unreadable / malformed   */
#define QUICK_ERR_CAPTURE 9      /* internal workspace would have to be
                                    allocated or grown on a capturing stream */

/* Human-readable name of a status code (static storage, never NULL). */
const char* quick_status_string(int status);

/* Identifier of the packed weight layout produced by quick_pack_weights.
 * 1 == "QPK16": units of 16 output columns x 128 input channels, 1 KiB of
 * packed weights each, ordered for the 16x16x32 f16 matrix instruction. */
int quick_pack_format_version(void);

/* ---- offline packing (host memory, no device work, reentrant) --------- */

/* Byte sizes of the three packed buffers for a K x N weight matrix:
 * packed weights K*N/2, packed zero points K*N/256, packed scales K*N/64.
 * Any output pointer may be NULL.  Errors: SHAPE, UNSUPPORTED. */
int quick_packed_sizes(int64_t K, int64_t N, int64_t group,
                       size_t* packed_bytes, size_t* zeros_bytes, size_t* scales_bytes);

/* Offline reorder of the static quantized weights (Section 3.1, 3.2).
 *   q      [K][N]          uint8, one 4-bit value (0..15) per byte
 *   z      [K/group][N]    uint8, zero points 0..15
 *   s      [K/group][N]    f16 scales
 * Outputs (host memory, sizes from quick_packed_sizes, fully overwritten):
 *   packed  QPK16 weights: for n-tile nt = n/16 and k-group kg = k/128 the
 *           1 KiB unit ((nt*K/128 + kg)) holds 64 lanes x 4 words; lane
 *           16*((k%32)/8) + n%16, word (k%128)/32, and inside the word the
 *           element e = k%8 sits in nibble e/2 (even e) or 4 + e/2 (odd e),
 *           so that masking the word and its 8-bit shift with 0x000F000F and
 *           0x00F000F0 yields element pairs (0,1), (2,3), (4,5), (6,7).
 *   zeros   uint32 word (nt*K/128 + kg)*2 + (n%16)/8 holds z in nibble n%8.
 *   scales  f16 at (nt*K/128 + kg)*16 + n%16.
 * Errors: INVALID_ARG (NULL), SHAPE, UNSUPPORTED, RANGE (value > 15; the
 * outputs are then left untouched). */
int quick_pack_weights(const uint8_t* q, const uint8_t* z, const uint16_t* s,
                       int64_t K, int64_t N, int64_t group,
                       void* packed, void* scales, void* zeros);

/* Exact inverse of quick_pack_weights (host memory). */
int quick_unpack_weights(const void* packed, const void* scales, const void* zeros,
                         int64_t K, int64_t N, int64_t group,
                         uint8_t* q, uint8_t* z, uint16_t* s);

/* ---- the GEMM (device memory, asynchronous) --------------------------- */

/* y[M][N] (f16) = x[M][K] (f16) . W, W the dequantized packed weights.
 * Accumulation is fp32 throughout (also across split-K partials); the one
 * final rounding to f16 is round-to-nearest-even.  Each weight is
 * dequantized to f16 as (q - z) * s with an exact subtraction and a single
 * rounding of the product.
 *   x, packed      device pointers, 16-byte aligned
 *   scales         device pointer, 2-byte aligned
 *   zeros          device pointer, 4-byte aligned
 *   y              device pointer, 8-byte aligned; must not overlap inputs
 *   stream         hipStream_t passed as void*, NULL = default stream
 * M == 0 is a valid no-op.  The call returns after enqueueing; results are
 * visible after the stream is synchronized.  The library may use an internal
 * device workspace (split-K partial sums, stream-K partial tiles, the sliced
 * stream kernel's partial columns, and arrival counters), one per (device,
 * stream), allocated on first need (its counters cleared on `stream`) and
 * grown when a larger plan needs more; a grown-out buffer is retired but not
 * freed, so graphs captured earlier keep valid pointers.  Nothing is ever
 * freed before process exit.  Calls on one stream are ordered; calls on
 * different streams use different workspaces.
 * HIP graph capture: a call on a capturing stream never allocates, clears or
 * synchronizes; when its plan needs more internal workspace than the
 * stream's buffer holds (e.g. the first call on that stream) it enqueues
 * nothing and returns QUICK_ERR_CAPTURE.  Warm the stream up with the same
 * shapes before capturing, or pass a workspace (quick_w4a16_gemm_ex).  The
 * captured launches keep using the capture stream's buffer: replays must not
 * overlap other work that uses it (eager calls on that stream or replays of
 * other graphs captured on it).
 * Errors: INVALID_ARG, SHAPE, UNSUPPORTED, ALIGNMENT, HIP, CAPTURE. */
int quick_w4a16_gemm(const void* x, const void* packed, const void* scales,
                     const void* zeros, void* y, int64_t M, int64_t N, int64_t K,
                     int64_t group, void* stream);

/* Kernel selection for quick_w4a16_gemm_ex (tests, benchmarks, tuning).
 * Zero in any field means "choose automatically". */
typedef struct quick_config {
    int variant;   /* 0 auto, 1 = stream kernel (small M), 2 = tiled kernel,
                      3 = tiled kernel with the stream-K schedule (resident
                      workgroups run the whole rounds of tiles, then share
                      the remaining tiles x k-groups work equally),
                      4 = reserved (rejected with INVALID_ARG),
                      5 = sliced stream kernel (M <= 16: the 8 waves of a
                      workgroup split 128 or 256 columns, workgroups split
                      K into slices of at most 2048 channels whose rows of x
                      they stage in LDS once; N/128 <= 4096),
                      6 = tiled kernel on the 32x32x16 matrix instruction
                      (waves of 32 columns: two n-tiles per instruction),
                      7 = the same with the stream-K schedule              */
    int split_k;   /* variants 2, 6: K slices across workgroups; variant 1:
                      waves per workgroup (1, 2, 4, 8); variants 3, 7: resident
                      workgroups, a multiple of 8 up to 4096 (clamped to the
                      number of tile x 128-channel units); variant 5: K
                      slices (raised to at least
                      ceil(K/2048), at most K/128); 0 = auto                */
    int tile_m;    /* tiled kernel rows per workgroup: 16, 32, 64 or 128
                      (variant 5: must be 0);
                      supported (tile_m, tile_n) pairs, variants 2, 3:
                      (16|32|64|128, 16|32); variants 6, 7:
                      (32|64|128, 32)                                        */
    int tile_n;    /* tiled kernel columns per wave: 16 or 32
                      stream kernels (variants 1, 5): n-tiles per wave: 1 or
                      2                                                      */
} quick_config_t;

/* Leading bytes of a workspace that hold stream-K arrival counters. */
#define QUICK_WORKSPACE_COUNTER_BYTES 16384

/* Same contract as quick_w4a16_gemm with an explicit kernel choice.
 * workspace/workspace_bytes: optional caller-owned device buffer (16-byte
 * aligned) for split-K partial sums, stream-K partial tiles or the sliced
 * stream kernel's per-slice partial columns; when NULL the
 * internal workspace is used.  Its first QUICK_WORKSPACE_COUNTER_BYTES hold
 * arrival counters that must be zero before the buffer's first use (e.g.
 * allocate it zero-filled); every call leaves them zero.  Calls that share a
 * workspace must be ordered (same stream).
 * Errors as quick_w4a16_gemm, plus INVALID_ARG for an unsupported config
 * and WORKSPACE when the caller buffer is smaller than
 * quick_workspace_bytes(). */
int quick_w4a16_gemm_ex(const void* x, const void* packed, const void* scales,
                        const void* zeros, void* y, int64_t M, int64_t N, int64_t K,
                        int64_t group, void* stream, const quick_config_t* cfg,
                        void* workspace, size_t workspace_bytes);

/* ---- allocation-free variant ----------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, automatic kernel choice (including a loaded tune table) and
 * results as quick_w4a16_gemm, but the split-K / stream-K / sliced-kernel
 * workspace is a fixed library array of QUICK_SCRATCH_BYTES per GPU (a
 * static device array, held on every GPU the library runs on until the
 * process ends) instead of an allocation: the call itself never allocates,
 * frees or synchronizes.  The first call on a device looks the array up and
 * enqueues one small kernel on `stream` that zeroes its arrival counters
 * (every GEMM leaves them zero again).
 * All calls on one GPU share that GPU's array, which keeps the last call's
 * contents: calls that may run at the same time on one GPU (different
 * streams, or graph replays that overlap other such calls) race and give
 * wrong results.  Order them on one stream.
 * Errors: as quick_w4a16_gemm (no CAPTURE: nothing is allocated), plus
 * WORKSPACE when the shape's plan needs more than QUICK_SCRATCH_BYTES
 * (quick_workspace_bytes(M, N, K, NULL) tells beforehand). */
#define QUICK_SCRATCH_BYTES ((size_t)80 << 20)
int quick_w4a16_gemm_noalloc(const void* x, const void* packed, const void* scales,
                             const void* zeros, void* y, int64_t M, int64_t N, int64_t K,
                             int64_t group, void* stream);

/* Workspace bytes quick_w4a16_gemm_ex needs for this shape and config
 * (cfg NULL = automatic choice); 0 when no workspace is used. */
size_t quick_workspace_bytes(int64_t M, int64_t N, int64_t K, const quick_config_t* cfg);

/* The configuration the automatic heuristic picks for a shape (for logs and
 * benchmarks).  Errors: INVALID_ARG (NULL cfg), SHAPE. */
int quick_select_config(int64_t M, int64_t N, int64_t K, quick_config_t* cfg);

/* ---- per-shape autotuning (the paper leaves split-K / tile choice as a
 * tuning knob; Section 5 names autotuning as future work) ---------------- */

/* Times every supported kernel configuration for this shape on the caller's
 * buffers (same arguments and contract as quick_w4a16_gemm; y is
 * overwritten, the last write coming from the best configuration) and
 * records the fastest in the process-wide tune table.  Each configuration's
 * max(20, copies) launches are captured as one HIP graph on a private
 * stream (which first waits for `stream`) and timed with HIP events as the
 * fastest of three replays, so the host's per-launch cost does not enter
 * the timing of short kernels.  The table is keyed by (M, N, K).  From
 * then on quick_w4a16_gemm, and the
 * automatic choice of quick_w4a16_gemm_ex / quick_workspace_bytes /
 * quick_select_config, use the recorded configuration for that shape on
 * every device.  The timed launches rotate through temporary device copies
 * of packed, scales and zeros spanning at least 512 MB (twice the 256 MB
 * Infinity Cache, at most 64 copies), so that each launch streams its
 * weights from HBM as in a forward pass; when that memory cannot be
 * allocated, they repeat the caller's buffers.
 * Blocking: waits for its own work; takes tens of milliseconds to a few
 * hundred; allocates and frees the copies and allocates a workspace for its
 * private stream (kept until process exit), so not for use under graph
 * capture (QUICK_ERR_CAPTURE when `stream` is capturing).  `best` (may be NULL) receives the
 * configuration recorded.  M == 0 records nothing.
 * Errors: as quick_w4a16_gemm, plus CAPTURE. */
int quick_tune(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
               int64_t M, int64_t N, int64_t K, int64_t group, void* stream, quick_config_t* best);

/* Persist / restore the tune table as text: a header line "quick-tune 1"
 * then one line "M N K variant split_k tile_m tile_n" per shape.  Loading
 * validates every line first and then merges (later entries replace
 * earlier ones for the same shape); on any malformed line nothing is loaded.
 * Errors: INVALID_ARG (NULL path), IO (cannot open / malformed). */
int quick_tune_table_save(const char* path);
int quick_tune_table_load(const char* path);
/* Number of shapes in the tune table; quick_tune_table_clear empties it. */
int quick_tune_table_size(void);
void quick_tune_table_clear(void);

#ifdef __cplusplus
}
#endif

#endif /* QUICK_H */
