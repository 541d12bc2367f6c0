// Types and launch functions shared by the parts of quick_gemm.hip, which the
// build compiles as separate translation units in parallel: the host part
// (validation, plans, workspace, tuning, the C ABI), the stream-kernel part
// and the tiled-kernel part (each instantiates and launches its kernels).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace quick {

typedef uint32_t lu4_t __attribute__((ext_vector_type(4)));

// Output epilogue applied to the fp32 accumulators before the single
// rounding to f16: an optional per-column bias, then either nothing or the
// gated SiLU of a fused gate/up projection whose packed columns alternate
// in 16-column tiles (gate tile t at packed columns 32t .. 32t+15, the
// matching up tile at 32t+16 .. 32t+31):
//   y[m][16t + i] = silu(h[m][32t + i]) * h[m][32t + 16 + i],
//   silu(a) = a / (1 + e^-a),  h = x . W (+ bias).
struct Epi {
    const uint16_t* bias;  // f16 [N] in packed column order, or null
    int act;               // 0 none, 1 gated SiLU (output has N/2 columns)
};

// Grouped (mixture-of-experts) form: E experts' packed weights back to back,
// routed row r of the output multiplies token rows[r] of x (row r when rows
// is null) with the weights of the expert e whose range
// [offsets[e], offsets[e+1]) holds r.  The per-expert row counts live only
// in device memory: each workgroup derives the tile list from them.
struct GroupArgs {
    const int* rows;     // [routed] token row of each routed row, or null
    const int* offsets;  // [experts + 1] first routed row of each expert
    int experts;
    int routed;          // rows of y
    // Which of each expert's rows this launch covers.  0: all.  With
    // `unit` rows per full tile: 1 = the leading whole tiles, plus the
    // remainder when it holds at least `keep` rows; 2 = the rest (a
    // remainder of fewer than `keep` rows), for a launch with shorter tiles.
    int part;
    int unit;
    int keep;
};

// A launch configuration, complete once finish_plan has run.
struct Plan {
    int variant;
    int split;  // stream: waves per workgroup; tiled: k splits; stream-K: workgroups;
                // sliced stream: K slices
    int bm;     // tiled: rows per workgroup
    int wn;     // tiled: columns per wave; stream kernels: n-tiles per wave
    int kgps;   // tiled split-K and sliced stream: k-groups per slice
};

// Stream-kernel part.
int launch_stream(const Plan& pl, const uint16_t* x, const lu4_t* pw, const uint16_t* ps, const uint32_t* pz,
                  uint16_t* y, int M, int N, int K, hipStream_t st, const Epi& epi);
int launch_kstream(const Plan& pl, const uint16_t* x, const lu4_t* pw, const uint16_t* ps, const uint32_t* pz,
                   uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi);

// Tiled-kernel part.  ga == nullptr: the plain GEMM; otherwise the grouped
// form (M = token rows).
int launch_tiled(const Plan& pl, const uint16_t* x, const lu4_t* pw, const uint16_t* ps, const uint32_t* pz,
                 uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi,
                 const GroupArgs* ga = nullptr);
// Workgroups of the tiled kernel (mfma32: its 32x32x16 form) resident at
// once on the current device.
int tiled_resident(int bm, int wn, bool mfma32 = false);
// The tiled kernel on the 32x32x16 instruction (plans of variants 6 and 7).
int launch_tiled32(const Plan& pl, const uint16_t* x, const lu4_t* pw, const uint16_t* ps, const uint32_t* pz,
                   uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi);
// The 64 x 256 data-parallel tiled kernel with the write-back mode of the
// ablation (0 direct, 1 padded LDS rows, 2 unpadded LDS rows).
int launch_ablation(const uint16_t* x, const lu4_t* pw, const uint16_t* ps, const uint32_t* pz, uint16_t* y,
                    int M, int N, int K, int mode, hipStream_t st);

}  // namespace quick
