// W4A16 GEMM kernels for gfx950 (MI355X) and the GEMM entry points of the
// C ABI.
//
// y[M][N] = x[M][K] . W,  W[k][n] = (q[k][n] - z[k/128][n]) * s[k/128][n]
// (paper, Section 2.1 and Section 2.3), with the weights in the QPK16 packed
// layout produced offline by quick_pack_weights (Section 3.1, 3.2).
//
// Common scheme of both kernels:
//  * One 16-byte load per lane fetches a lane's share of a 1 KiB packed
//    unit (16 columns x 128 input channels): 4 words, one per 32-wide k step
//    of the 16x16x32 f16 matrix instruction.  The words go straight into
//    VGPRs; dequantized weights never touch LDS (Section 3.1).
//  * Dequantization in VGPRs with packed f16 arithmetic (Section 2.3):
//    masking the word and its 8-bit shift with 0x000F000F / 0x00F000F0 and
//    OR-ing the binary16 pattern of 1024 yields f16 pairs 1024+q (low
//    nibbles) and 1024+16q (high nibbles); subtracting 1024+z, or fused
//    multiply-adding with 1/16 and -(64+z), gives q-z exactly, and one f16
//    multiply by s gives the weight with a single rounding.  The nibble order
//    inside the word (Section 3.2's dequant-aware reorder) makes the four f16
//    pairs come out in k order, i.e. already in operand-register order.
//  * The dequantized weights are the instruction's A operand (rows = output
//    columns n) and the activations its B operand (columns = rows m of x), so
//    each lane ends with 4 consecutive n of one output row in its 4
//    accumulators and stores them as one 8-byte write.
//  * fp32 accumulation everywhere, including split-K partial sums, and one
//    final round-to-nearest-even to f16.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <type_traits>
#include <utility>
#include <vector>

#include "quick.h"
#include "quick_ablation.h"
#include "quick_fused.h"
#include "quick_grouped.h"
#include "quick_internal.h"
#include "quick_launch.h"

// The build compiles this file as three translation units in parallel
// (QUICK_PART 0: host code and the C ABI; 1: stream-kernel launches; 2:
// tiled-kernel launches); without QUICK_PART it is the whole library.
#if !defined(QUICK_PART)
#define QUICK_HOST 1
#define QUICK_STREAM 1
#define QUICK_TILED 1
#else
#define QUICK_HOST (QUICK_PART == 0)
#define QUICK_STREAM (QUICK_PART == 1)
#define QUICK_TILED (QUICK_PART == 2)
#endif

namespace {

using quick::Epi;
using quick::GroupArgs;
using quick::Plan;

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u2_t __attribute__((ext_vector_type(2)));


template <class To, class From>
__device__ __forceinline__ To bits_as(const From& v)
{
    static_assert(sizeof(To) == sizeof(From), "size mismatch");
    return __builtin_bit_cast(To, v);
}

// Per (column, k-group) constants of the dequantizer, as f16x2 bit patterns:
// zlo = (1024+z, 1024+z), zhi = (-(64+z), -(64+z)), ss = (s, s).
struct Deq {
    uint32_t zlo, zhi, ss;
};

// Same from the 32-bit word holding this column's scale and its neighbour's
// (columns 2i, 2i+1): `sel` picks the half (0x01000100 low, 0x03020302 high)
// and duplicates it.
__device__ __forceinline__ Deq make_deq_pair(uint32_t s_pair, uint32_t sel, uint32_t z)
{
    const uint32_t a = 0x6400u | z;
    const uint32_t b = 0xD400u + (z << 4);
    Deq d;
    d.zlo = a | (a << 16);
    d.zhi = b | (b << 16);
    d.ss = __builtin_amdgcn_perm(s_pair, s_pair, sel);
    return d;
}

__device__ __forceinline__ Deq make_deq(uint32_t s_bits, uint32_t z)
{
    const uint32_t a = 0x6400u | z;          // binary16 of 1024 + z
    const uint32_t b = 0xD400u + (z << 4);   // binary16 of -(64 + z), ulp 1/16
    Deq d;
    d.zlo = a | (a << 16);
    d.zhi = b | (b << 16);
    d.ss = s_bits | (s_bits << 16);
    return d;
}

// (a & mask) | bits in one VALU instruction.  gfx9 VOP3 encodings take no
// literal constants, so the compiler otherwise splits this into an AND and an
// OR with literals; the mask is passed in an SGPR, the OR pattern in a VGPR.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t mask, uint32_t bits)
{
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(mask), "v"(bits));
    return r;
}

// Eight weights of one packed word -> the 8 f16 operand values, k order.
__device__ __forceinline__ h8_t dequant8(uint32_t w, const Deq& d)
{
#pragma clang fp contract(off)
    const uint32_t lo = 0x000F000Fu, hi = 0x00F000F0u, one024 = 0x64006400u;
    const uint32_t w8 = w >> 8;
    const h2_t h0 = bits_as<h2_t>(and_or(w, lo, one024));   // 1024 + q(e0), 1024 + q(e1)
    const h2_t h1 = bits_as<h2_t>(and_or(w, hi, one024));   // 1024 + 16 q(e2), ... q(e3)
    const h2_t h2 = bits_as<h2_t>(and_or(w8, lo, one024));  // e4, e5
    const h2_t h3 = bits_as<h2_t>(and_or(w8, hi, one024));  // e6, e7
    const h2_t zlo = bits_as<h2_t>(d.zlo);
    const h2_t zhi = bits_as<h2_t>(d.zhi);
    const h2_t ss = bits_as<h2_t>(d.ss);
    const h2_t sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f};
    const h2_t d0 = (h0 - zlo) * ss;
    const h2_t d1 = __builtin_elementwise_fma(h1, sixteenth, zhi) * ss;
    const h2_t d2 = (h2 - zlo) * ss;
    const h2_t d3 = __builtin_elementwise_fma(h3, sixteenth, zhi) * ss;
    h8_t r = {d0[0], d0[1], d1[0], d1[1], d2[0], d2[1], d3[0], d3[1]};
    return r;
}

__device__ __forceinline__ f4_t mfma16(const h8_t& a, const h8_t& b, const f4_t& c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// 4 fp32 -> 4 f16 (round to nearest even), stored as one 8-byte write.
__device__ __forceinline__ void store_h4(uint16_t* dst, const f4_t& v)
{
    const _Float16 a = (_Float16)v[0], b = (_Float16)v[1], c = (_Float16)v[2], e = (_Float16)v[3];
    u2_t o;
    o[0] = (uint32_t)bits_as<uint16_t>(a) | ((uint32_t)bits_as<uint16_t>(b) << 16);
    o[1] = (uint32_t)bits_as<uint16_t>(c) | ((uint32_t)bits_as<uint16_t>(e) << 16);
    *reinterpret_cast<u2_t*>(dst) = o;
}

__device__ __forceinline__ f4_t add_bias(f4_t v, const uint16_t* bias, int n)
{
    if (bias) {
        const u2_t b = *reinterpret_cast<const u2_t*>(bias + n);
        v[0] += (float)bits_as<_Float16>((uint16_t)(b[0] & 0xFFFFu));
        v[1] += (float)bits_as<_Float16>((uint16_t)(b[0] >> 16));
        v[2] += (float)bits_as<_Float16>((uint16_t)(b[1] & 0xFFFFu));
        v[3] += (float)bits_as<_Float16>((uint16_t)(b[1] >> 16));
    }
    return v;
}

__device__ __forceinline__ f4_t silu_gate(const f4_t& a, const f4_t& b)
{
    f4_t r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = a[i] / (1.f + __expf(-a[i])) * b[i];
    return r;
}

// Store 4 consecutive packed columns n .. n+3 of row m (act == 0), or, for
// the gated form, the gate quad at n (n % 32 < 16) with its up quad `u` at
// n + 16 as output columns n/32*16 + n%32 .. +3; N = packed columns.
__device__ __forceinline__ void store_out(uint16_t* y, const Epi& e, int64_t m, int N, int n, f4_t v)
{
    v = add_bias(v, e.bias, n);
    store_h4(y + m * N + n, v);
}
__device__ __forceinline__ void store_gated(uint16_t* y, const Epi& e, int64_t m, int N, int n, f4_t gate, f4_t up)
{
    gate = add_bias(gate, e.bias, n);
    up = add_bias(up, e.bias, n + 16);
    store_h4(y + m * (N / 2) + (n >> 5) * 16 + (n & 15), silu_gate(gate, up));
}

// Raw buffer loads: a wave-uniform 128-bit descriptor (base, byte size) in
// SGPRs, a per-lane byte offset in a VGPR and a wave-uniform byte offset in an
// SGPR, so per-iteration address arithmetic is scalar.  Offsets at or beyond
// the size read as zero instead of faulting.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRawBufferWord3 = 0x00020000;  // gfx9 raw (untyped, unswizzled) buffer

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kRawBufferWord3);
}
__device__ __forceinline__ u4_t ld128(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return bits_as<u4_t>(__builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ uint32_t ld32(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}
// 16 bytes per lane from a buffer straight into LDS: lane L of the wave
// writes bytes [16L, 16L+16) after the wave-uniform LDS address `dst`.
__device__ __forceinline__ void dma16(rsrc_t r, void* dst, uint32_t voff, uint32_t soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, voff, soff, 0, 0);
}
// Wait until every outstanding memory operation of this wave has completed.
__device__ __forceinline__ void wait_all() { __builtin_amdgcn_s_waitcnt(0); }
// Wait until at most V vector-memory loads of this wave are outstanding
// (V clamped to the 6-bit counter; gfx9 encoding: vmcnt in bits 3:0 and
// 15:14, expcnt and lgkmcnt left at their maxima).
template <int V>
__device__ __forceinline__ void wait_vm()
{
    constexpr int v = V < 63 ? V : 63;
    __builtin_amdgcn_s_waitcnt(0x0F70 | (v & 15) | ((v >> 4) << 14));
}
// f(std::integral_constant<int, n>{}) for a wave-uniform 0 <= n <= N: code
// specialised on a count known only at run time.
template <int N, class F>
__device__ __forceinline__ void with_count(int n, F&& f)
{
    if constexpr (N == 0) {
        f(std::integral_constant<int, 0>{});
    } else {
        if (n >= N) f(std::integral_constant<int, N>{});
        else with_count<N - 1>(n, f);
    }
}
// Workgroup execution barrier without memory-fence semantics.  Used where
// explicit counter waits before it already order the memory traffic: every
// LDS-DMA a wave issued for the next stage has completed (vmcnt wait) and
// every LDS read of a stage that another wave may overwrite after the
// barrier has returned its data (lgkmcnt wait, wait_lds()).
__device__ __forceinline__ void barrier() { __builtin_amdgcn_s_barrier(); }
// Wait until every LDS read of this wave has returned (lgkmcnt 0; vmcnt and
// expcnt left at their maxima).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Scheduling fence: no instruction moves across it.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
__device__ __forceinline__ uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ uint32_t ld16(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return (uint32_t)(uint16_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}

// ---------------------------------------------------------------------------
// Stream kernel (small M, bandwidth-bound).
//
// A workgroup owns NPW n-tiles (16 columns each) and the whole K range; its
// WAVES waves split the k-groups between them (in-workgroup split-K, no
// partial sums leave the workgroup).  Each wave streams its packed units from
// HBM with one 16-byte load per lane and unit through a ring of D register
// stages, so D-1 k-groups of weights are in flight while one is dequantized
// and multiplied; a short k-range (activations in LDS) instead runs as one
// pass specialised on its unit count with a few units requested ahead.  At
// the end the waves' fp32 partial tiles are summed through LDS in wave order
// (deterministic) and stored.
//
// Activation fragments (B operand, MT blocks of 16 rows):
//  * XL: the wave first copies its own k-range of all M rows of x into its
//    slice of LDS with the 16-byte LDS-DMA load (rows contiguous, row stride
//    = the slice width), waits for it (the copy is issued before the weight
//    loads, so the wait lets those stay in flight), and then reads fragments
//    with LDS reads; lanes of rows >= M read row M-1 (broadcast).  No
//    barrier: a wave only reads what it copied.  Used when all waves' slices
//    fit in 64 KiB.
//  * otherwise the fragments are 16-byte buffer loads from global memory
//    (they are small and shared by every workgroup, so they hit in cache),
//    one k-group ahead.
// ---------------------------------------------------------------------------
// Per-wave LDS slice of the stream kernel's staged activations: M rows of
// the wave's k-range (at most ceil(KG/WAVES) k-groups of 256 bytes per row),
// rounded up to whole 1 KiB copy instructions.
__host__ __device__ constexpr uint32_t stream_slice_bytes(int M, int KG, int WAVES)
{
    return (uint32_t)((M * ((KG + WAVES - 1) / WAVES) * 256 + 1023) / 1024 * 1024);
}

template <int NPW>
struct WStage {
    u4_t w[NPW];
    uint32_t s[NPW];
    uint32_t z[NPW];
};

// Longest per-wave k-range (units) the stream kernel runs as one specialised
// pass, and the units that pass keeps requested ahead of the one it
// multiplies.
constexpr int kStreamSinglePass = 16;
constexpr int kStreamLookahead = 4;

template <int MT, int NPW, int WAVES, int D, bool XL>
__global__ void __launch_bounds__(64 * WAVES)
stream_kernel(const uint16_t* __restrict__ x, const u4_t* __restrict__ pw,
              const uint16_t* __restrict__ ps, const uint32_t* __restrict__ pz,
              uint16_t* __restrict__ y, int M, int N, int K, Epi epi)
{
    static_assert(D % 2 == 0, "ring depth must be even (activation double buffer parity)");
    static_assert(!XL || 3 * NPW * D <= 63, "the slice-copy waits count the ring's loads within the 6-bit vmcnt");
    extern __shared__ __attribute__((aligned(16))) uint8_t xlds[];
    const int KG = K >> 7;
    const int NT = N >> 4;
    const int lane = threadIdx.x & 63;
    // wave index as a scalar: everything derived from it (k range, buffer
    // offsets) stays in SGPRs
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = lane & 15;
    const int g = lane >> 4;
    const int nt0 = blockIdx.x * NPW;
    const int kb = (KG * wave) / WAVES;
    const int ke = (KG * (wave + 1)) / WAVES;
    const int nk = ke - kb;

    const rsrc_t rw = make_rsrc(pw, (uint32_t)((size_t)K * N / 2));
    const rsrc_t rs = make_rsrc(ps, (uint32_t)((size_t)K * N / 64));
    const rsrc_t rz = make_rsrc(pz, (uint32_t)((size_t)K * N / 256));
    const rsrc_t rx = make_rsrc(x, (uint32_t)((size_t)M * K * 2));

    // Column tiles past the end of N and activation rows past M are clamped
    // to valid ones instead of masked: an output row of the instruction
    // depends only on its own weight row (n) and an output column only on
    // its own activation column (m), and those outputs are never stored.
    uint32_t ubase[NPW];  // first unit of each n-tile, wave-uniform
#pragma unroll
    for (int p = 0; p < NPW; ++p) ubase[p] = (uint32_t)min(nt0 + p, NT - 1) * KG;
    const uint32_t vw = lane * 16;
    const uint32_t vs = c * 2;
    const uint32_t vz = (c >> 3) * 4;

    // activation fragment source per 16-row block: global byte offset of
    // (row, channel 8*g) [global path] or LDS offset inside the wave's slice
    // [XL path]
    uint32_t vx[MT];
    // this wave's slice: M rows x nk*256 bytes, at a fixed per-wave stride
    // that is a 1 KiB multiple, so the last copy instruction's extra lanes
    // stay inside the wave's own slice
    uint8_t* xslice = xlds + (size_t)wave * stream_slice_bytes(M, KG, WAVES);
    const uint32_t xrow = (uint32_t)nk * 256;         // slice row stride
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int row = min(mt * 16 + c, M - 1);
        vx[mt] = XL ? (uint32_t)(row * xrow + g * 16) : (uint32_t)(row * K + g * 8) * 2;
    }

    if constexpr (XL) {
        // copy rows 0..M-1, channels kb*128 .. ke*128 into the slice: 16 bytes
        // per lane, slice byte b = row*xrow + q*16 <- x[row][kb*128 + 8q ..]
        const int chunks = M * nk * 16;   // 16-byte chunks in the slice
        for (int i0 = 0; i0 < chunks; i0 += 64) {
            const int idx = min(i0 + lane, chunks - 1);
            const int row = idx / (nk * 16);
            const int q = idx - row * nk * 16;
            const uint32_t src = (uint32_t)(row * K + kb * 128 + q * 8) * 2;
            // the last instruction may have fewer than 64 chunks: its extra
            // lanes repeat the final chunk into the slice's padding
            dma16(rx, xslice + (size_t)i0 * 16, src, 0);
        }
    }

    f4_t acc[NPW][MT];
#pragma unroll
    for (int p = 0; p < NPW; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[p][mt] = f4_t{0.f, 0.f, 0.f, 0.f};

    WStage<NPW> ring[D];
    u4_t xf[2][MT][4];

    auto load_w = [&](WStage<NPW>& st, int kg) {
#pragma unroll
        for (int p = 0; p < NPW; ++p) {
            const uint32_t u = uniform(ubase[p] + kg);
            st.w[p] = ld128(rw, vw, u * 1024u);
            st.s[p] = ld16(rs, vs, u * 32u);
            st.z[p] = ld32(rz, vz, u * 8u);
        }
    };
    auto load_x = [&](u4_t (&xb)[MT][4], int kg) {
        if constexpr (XL) {
            const int kl = kg - kb;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    xb[mt][j] = *reinterpret_cast<const u4_t*>(xslice + vx[mt] + kl * 256 + j * 64);
        } else {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int j = 0; j < 4; ++j) xb[mt][j] = ld128(rx, vx[mt] + j * 64, uniform(kg * 256u));
        }
    };
    auto compute = [&](const WStage<NPW>& st, const u4_t (&xb)[MT][4]) {
        Deq d[NPW];
#pragma unroll
        for (int p = 0; p < NPW; ++p) d[p] = make_deq(st.s[p], (st.z[p] >> (4 * (c & 7))) & 15u);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int p = 0; p < NPW; ++p) {
                const h8_t a = dequant8(st.w[p][j], d[p]);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[p][mt] = mfma16(a, bits_as<h8_t>(xb[mt][j]), acc[p][mt]);
            }
        }
    };

    if (XL && nk <= kStreamSinglePass) {
        // A short k-range: one pass, specialised on the unit count so that
        // every load is unconditional.  The compiler's wait before each unit
        // then covers only that unit's loads, and units are multiplied as
        // they land instead of after the last one.
        with_count<kStreamSinglePass>(nk, [&](auto nkc) {
            constexpr int NKC = decltype(nkc)::value;
            // LA units ahead: requests beyond that would only queue behind
            // the bandwidth-bound ones already in flight while holding back
            // the first multiplications (in-order issue)
            constexpr int LA = NKC < kStreamLookahead ? NKC : kStreamLookahead;
            constexpr int R = LA + 1;  // stages live at once
            WStage<NPW> sring[R];
#pragma unroll
            for (int i = 0; i < LA; ++i) {
                load_w(sring[i], kb + i);
                sched_fence();  // issue stage by stage, so each unit's loads land together
            }
            if constexpr (NKC > 0) {
                // the slice copy was issued before these 3 * NPW * LA loads
                wait_vm<3 * NPW * LA>();
                load_x(xf[0], kb);
#pragma unroll
                for (int i = 0; i < NKC; ++i) {
                    if (i + 1 < NKC) load_x(xf[(i + 1) & 1], kb + i + 1);
                    compute(sring[i % R], xf[i & 1]);
                    if (i + LA < NKC) load_w(sring[(i + LA) % R], kb + i + LA);
                    // no work of a later unit moves up here, where it would
                    // wait for that unit's loads
                    sched_fence();
                }
            }
        });
    } else {
        // one trip of the ring: unit k0 + i is multiplied while unit
        // k0 + i + D is requested
        auto trip = [&](int k0) {
#pragma unroll
            for (int i = 0; i < D; ++i) {
                load_x(xf[(i + 1) & 1], k0 + i + 1);
                compute(ring[i], xf[i & 1]);
                load_w(ring[i], k0 + i + D);
                // keep each refill where it is: the scheduler would otherwise
                // sink all of them to the end of the trip and issue them in
                // one burst that the next trip then waits for
                sched_fence();
            }
        };
        int kg = kb;
        if (nk >= 2 * D) {
            // At least one full trip.  Unconditional requests, the first
            // activation fragments ahead of the weights, and the first trip
            // peeled: the loop is then entered in the state it loops back in
            // (D stages in flight), and the compiler's wait analysis keeps
            // D-1 stages in flight from the first unit on.
            if constexpr (!XL) load_x(xf[0], kb);
#pragma unroll
            for (int i = 0; i < D; ++i) load_w(ring[i], kb + i);
            if constexpr (XL) {
                wait_vm<3 * NPW * D>();  // the slice copy, issued before these loads, has landed
                load_x(xf[0], kb);
            }
            trip(kg);
            for (kg += D; kg + 2 * D <= ke; kg += D) trip(kg);
        } else {
#pragma unroll
            for (int i = 0; i < D; ++i)
                if (kb + i < ke) load_w(ring[i], kb + i);
            if constexpr (XL) wait_all();  // the slice has landed (weights too, once)
            if (kb < ke) load_x(xf[0], kb);
        }
        // tail
        for (; kg < ke; kg += D) {
#pragma unroll
            for (int i = 0; i < D; ++i) {
                const int k = kg + i;
                if (k < ke) {
                    if (k + 1 < ke) load_x(xf[(i + 1) & 1], k + 1);
                    compute(ring[i], xf[i & 1]);
                    if (k + D < ke) load_w(ring[i], k + D);
                }
            }
        }
    }

    // (gated form: NPW == 2 and nt0 even, so acc[0] / acc[1] are a gate
    // tile and its up tile)
    if constexpr (WAVES == 1) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int m = mt * 16 + c;
            if (m >= M) continue;
            if (NPW == 2 && epi.act) {
                if (nt0 < NT) store_gated(y, epi, m, N, nt0 * 16 + 4 * g, acc[0][mt], acc[NPW - 1][mt]);
                continue;
            }
#pragma unroll
            for (int p = 0; p < NPW; ++p)
                if (nt0 + p < NT) store_out(y, epi, m, N, (nt0 + p) * 16 + 4 * g, acc[p][mt]);
        }
    } else {
        __shared__ f4_t red[WAVES][NPW * MT][64];
#pragma unroll
        for (int p = 0; p < NPW; ++p)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) red[wave][p * MT + mt][lane] = acc[p][mt];
        __syncthreads();
        auto total = [&](int pm, int l) {
            f4_t sum = red[0][pm][l];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) sum += red[w][pm][l];
            return sum;
        };
        if (NPW == 2 && epi.act) {
            for (int item = threadIdx.x; item < MT * 64; item += 64 * WAVES) {
                const int l = item & 63;
                const int mt = item >> 6;
                const int m = mt * 16 + (l & 15);
                if (nt0 >= NT || m >= M) continue;
                store_gated(y, epi, m, N, nt0 * 16 + 4 * (l >> 4), total(mt, l), total((NPW - 1) * MT + mt, l));
            }
        } else {
            for (int item = threadIdx.x; item < NPW * MT * 64; item += 64 * WAVES) {
                const int l = item & 63;
                const int pm = item >> 6;
                const int p = pm / MT;
                const int mt = pm % MT;
                const int m = mt * 16 + (l & 15);
                if (nt0 + p >= NT || m >= M) continue;
                store_out(y, epi, m, N, (nt0 + p) * 16 + 4 * (l >> 4), total(pm, l));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Tiled kernel (large M, matrix-core-bound).
//
// One workgroup of WAVES waves per CU computes a BM x (WAVES*WN) output tile;
// the waves split the columns (each wave WN columns and all BM rows), so
// every packed weight is loaded and dequantized exactly once per workgroup,
// straight into VGPRs (Section 3.1), and the activation tile in LDS is shared
// by all of them (Section 3.3: LDS holds activations only, which leaves room
// for a big tile and a deep ring).
//
// Activations: a ring of NST LDS stages of BM rows x 128 input channels (one
// k-group).  Each stage is filled global -> LDS by the 16-byte LDS-DMA form of
// the buffer load (no staging registers): one instruction moves 4 rows, lane
// L landing at byte 16*L of the instruction's 1 KiB.  Inside a 256-byte row
// the 16-byte chunk holding channels 8*q .. 8*q+7 sits at position
// q ^ (row % 16), so fragment reads of 16 consecutive rows at one chunk index
// hit 16 distinct bank groups.
//
// Weights: one 16-byte load per lane and n-tile per k-group into a ring of
// NST register slots.  k-group k+NST-1 (activations and weights) is requested
// while k-group k is computed; the wait of k-group k only drains the loads
// of k-group k+1 (vector-memory counters retire in issue order), so NST-2
// k-groups stay in flight across the barrier.
//
// Inside a k-group: 4 steps of 32 channels, software-pipelined -- while the
// matrix instructions of step j run, the activation fragments of step j+1
// are read from LDS and the weights of step j+1 are dequantized.  The
// pipeline runs on across k-groups: the wait and the workgroup barrier of
// k-group k come before its last step, whose matrix instructions then cover
// the fragment reads and dequant of k-group k+1's first step.
//
// Tiles are numbered M-fastest and assigned so that consecutive numbers run
// on the same XCD (workgroup ids go to the 8 XCDs round-robin): M-tiles that
// share an N-tile's weights share one L2.  Three schedules:
//  * data-parallel (n_splits == 1): one workgroup per tile; gridDim.x is
//    padded to a multiple of 8 and the extra workgroups exit at once;
//  * split-K (n_splits > 1): one workgroup per (tile, K slice); each writes
//    fp32 partial sums to the workspace and a second kernel adds them in
//    split order;
//  * stream-K (n_splits == 0): gridDim.x resident workgroups run the whole
//    rounds of tiles data-parallel and share the rest of the tiles x
//    k-groups iteration space in equal contiguous ranges, so no round of
//    tiles runs on a partly idle chip.  A tile whose k-groups span
//    several workgroups is finished by the last of them to arrive (per-tile
//    arrival counter): every contributor writes its fp32 partial tile with
//    device-coherent stores, and the last one adds all partials in k order
//    (the same order whoever is last, so results are deterministic), rounds
//    once to f16 and resets the counter.  No workgroup ever waits for
//    another.
// ---------------------------------------------------------------------------
constexpr int kTiledWaves = 8;
constexpr int kTiledStages = 4;
// stream-K workspace: arrival counters (one per workgroup, zero between
// calls), then two fp32 partial-tile slots per workgroup
constexpr int kSkMaxWorkgroups = 4096;
constexpr size_t kSkCounterBytes = QUICK_WORKSPACE_COUNTER_BYTES;
static_assert(kSkCounterBytes >= kSkMaxWorkgroups * sizeof(unsigned), "one counter per workgroup");
constexpr int kCoherentAux = 0x11;  // sc0 sc1: coherent across XCDs, write-through
constexpr int kMaxExperts = QUICK_MAX_EXPERTS;


// WB != 0 builds the write-back ablation of the conventional design (the
// dequantized weights go through an LDS tile and are read back as matrix
// fragments): 1 = rows padded by 16 bytes (conflict-free), 2 = unpadded
// [n][k] rows (same-bank fragment accesses).  Only the ablation library
// launches it; WB = 0 is the method's direct-to-register path.
// GRP builds the grouped form (M is then the number of token rows of x).
// EP builds the output epilogue (bias, gated SiLU); without it the stores
// are plain roundings and the kernel carries none of its code.
template <int BM, int WN, int WB = 0, bool GRP = false, bool EP = false>
__global__ void __launch_bounds__(64 * kTiledWaves, 1)
tiled_kernel(const uint16_t* __restrict__ x, const u4_t* __restrict__ pw,
             const uint16_t* __restrict__ ps, const uint32_t* __restrict__ pz,
             uint16_t* __restrict__ y, float* __restrict__ ws, int M, int N, int K,
             int kg_per_split, int n_mtiles, int n_ntiles, int n_splits, GroupArgs ga, Epi epi)
{
    constexpr int WAVES = kTiledWaves;
    constexpr int NST = kTiledStages;
    constexpr int NP = WN / 16;                   // n-tiles per wave
    constexpr int MTT = BM / 16;                  // 16-row blocks
    constexpr int ROWB = 256;                     // bytes per activation row of a stage
    constexpr int STAGE = BM * ROWB;              // bytes per stage
    // 1 KiB LDS-DMA instructions per stage; wave w issues instructions
    // w, w + WAVES, ...  (for BM = 16 only waves 0..3 have one)
    constexpr int NDMA = STAGE / 1024;
    constexpr int DMA_PER_WAVE = (NDMA + WAVES - 1) / WAVES;   // upper bound per wave
    static_assert(NDMA >= 1 && STAGE % 1024 == 0 && (NDMA % WAVES == 0 || NDMA < WAVES), "DMA split");
    static_assert(2 * (DMA_PER_WAVE + 3 * NP) < 64, "vmcnt range");
    // one LDS object per stage: the compiler can then tell that a DMA into
    // one stage does not alias fragment reads from another, and does not
    // drain in-flight DMAs before every read
    static_assert(NST == 4, "stage objects below");
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s0[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s1[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s2[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s3[STAGE];
    auto stage_ptr = [&](int st) -> uint8_t* {
        return st == 0 ? lds_s0 : st == 1 ? lds_s1 : st == 2 ? lds_s2 : lds_s3;
    };
    // write-back ablation: per wave an [NP*16 columns][128 channels] f16 tile
    constexpr int WB_RS = WB == 1 ? 136 : 128;   // row stride in halves
    constexpr int WB_BYTES = WB ? WAVES * NP * 16 * WB_RS * 2 : 16;
    __shared__ __attribute__((aligned(16))) uint8_t lds_wb[WB_BYTES];

    const int KG = K >> 7;
    const int NT = N >> 4;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = lane & 15;
    const int g = lane >> 4;

    const size_t wbytes = (size_t)K * N / 2;   // packed weights of one expert
    rsrc_t rw = make_rsrc(pw, (uint32_t)wbytes);
    rsrc_t rs = make_rsrc(ps, (uint32_t)(wbytes / 32));
    rsrc_t rz = make_rsrc(pz, (uint32_t)(wbytes / 128));
    const rsrc_t rx = make_rsrc(x, (uint32_t)((size_t)M * K * 2));
    const uint32_t vw = lane * 16;
    const uint32_t vs = c * 2;
    const uint32_t vz = (c >> 3) * 4;
    // this wave's DMA instruction count (wave-uniform)
    const int ndma = NDMA >= WAVES ? DMA_PER_WAVE : (wave < NDMA ? 1 : 0);

    // ---- grouped form: per expert its routed rows [g_lo, g_hi) and the
    // number of BM-row tiles of all experts before it (g_cum).  Offsets are
    // clamped into [0, routed] so that any input stays in bounds.
    constexpr int GE = GRP ? kMaxExperts + 1 : 1;
    __shared__ int g_lo[GE], g_hi[GE], g_cum[GE];
    int n_mt = n_mtiles;  // m-tiles of the tile space
    if constexpr (GRP) {
        if (wave == 0) {
            int carry = 0;
            for (int e0 = 0; e0 < ga.experts; e0 += 64) {
                const int e = e0 + lane;
                int lo = 0, hi = 0;
                if (e < ga.experts) {
                    lo = min(max(ga.offsets[e], 0), ga.routed);
                    hi = min(max(ga.offsets[e + 1], lo), ga.routed);
                    if (ga.part) {
                        const int rem = (hi - lo) % ga.unit;
                        const int lead = rem >= ga.keep ? hi : hi - rem;   // end of part 1
                        if (ga.part == 1) hi = lead;
                        else lo = lead;
                    }
                }
                int t = (hi - lo + BM - 1) / BM;
#pragma unroll
                for (int d = 1; d < 64; d <<= 1) {
                    const int v = __shfl_up(t, d, 64);
                    if (lane >= d) t += v;
                }
                if (e < ga.experts) {
                    g_lo[e] = lo;
                    g_hi[e] = hi;
                    g_cum[e + 1] = carry + t;
                }
                carry += __shfl(t, 63, 64);
            }
            if (lane == 0) g_cum[0] = 0;
        }
        __syncthreads();
        n_mt = uniform(g_cum[ga.experts]);
    }

    const uint16_t* const bias0 = epi.bias;
    // ---- per-tile state
    int m0 = 0;      // first row of the tile
    int mend = M;    // end of the tile's rows (exclusive)
    int ntw = 0;     // first n-tile of this wave
    uint32_t ubase[NP];
    uint32_t vx[DMA_PER_WAVE];
    // tile t of the tile space: M-fastest (grouped: expert, then n-tile, then
    // the expert's m-tiles)
    auto set_tile = [&](int t) __attribute__((always_inline)) {
        int ntile;
        if constexpr (GRP) {
            // the expert whose tiles hold t: the last e with g_cum[e] * n_ntiles <= t
            int lo = 0, hi = ga.experts;
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (g_cum[mid] * n_ntiles <= t) lo = mid;
                else hi = mid;
            }
            const int e = uniform(lo);
            const int local = t - g_cum[e] * n_ntiles;
            const int tiles_e = g_cum[e + 1] - g_cum[e];
            ntile = local / tiles_e;
            m0 = uniform(g_lo[e]) + (local - ntile * tiles_e) * BM;
            mend = uniform(g_hi[e]);
            if (EP && bias0) epi.bias = bias0 + (size_t)e * N;   // bias [E][N]
            rw = make_rsrc(pw + (size_t)e * (wbytes / 16), (uint32_t)wbytes);
            rs = make_rsrc(ps + (size_t)e * (wbytes / 64), (uint32_t)(wbytes / 32));
            rz = make_rsrc(pz + (size_t)e * (wbytes / 512), (uint32_t)(wbytes / 128));
        } else {
            m0 = (t % n_mtiles) * BM;
            ntile = (t / n_mtiles) % n_ntiles;
        }
        // weight units of this wave's n-tiles (clamped; out-of-range tiles
        // are computed on valid data and never stored)
        ntw = ntile * (WAVES * NP) + wave * NP;
#pragma unroll
        for (int p = 0; p < NP; ++p) ubase[p] = (uint32_t)min(ntw + p, NT - 1) * KG;
        // LDS-DMA source offsets: this lane fills row rr of 1 KiB block i at
        // chunk position (lane % 16), i.e. it fetches channel chunk
        // (lane % 16) ^ (rr % 16)
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i) {
            const int rr = (wave + i * WAVES) * 4 + (lane >> 4);
            int row = min(m0 + rr, mend - 1);
            if constexpr (GRP) {
                // gather: the token row of this routed row
                if (ga.rows) row = ga.rows[row];
                row = min(max(row, 0), M - 1);
            }
            vx[i] = ((uint32_t)row * (uint32_t)K + 8 * ((lane & 15) ^ (rr & 15))) * 2;
        }
    };

    u4_t wr[NST][NP];
    uint32_t sr[NST][NP], zr[NST][NP];
    // k-group kg's activations -> LDS stage st and weights -> ring slot st
    auto fetch = [&](int st, int kg) __attribute__((always_inline)) {
        const uint32_t soff = uniform((uint32_t)kg * 256u);
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i)
            if (i < ndma) dma16(rx, stage_ptr(st) + (wave + i * WAVES) * 1024, vx[i], soff);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const uint32_t u = uniform(ubase[p] + kg);
            wr[st][p] = ld128(rw, vw, u * 1024u);
            sr[st][p] = ld16(rs, vs, u * 32u);
            zr[st][p] = ld32(rz, vz, u * 8u);
        }
    };
    // wait until at most `groups` k-groups of loads are still in flight
    // s_waitcnt immediate (gfx9): vmcnt in bits 3:0 and 15:14, expcnt 6:4 and
    // lgkmcnt 11:8 left at their maxima (no wait)
    auto wait_vm = [](auto n) { __builtin_amdgcn_s_waitcnt(0x0F70 | (n & 15) | ((n >> 4) << 14)); };
    constexpr int GL_FULL = DMA_PER_WAVE + 3 * NP;      // loads per k-group, waves with DMA
    constexpr int GL_NODMA = 3 * NP;                    // waves without (BM = 16, waves 4..7)
    auto wait_groups = [&](int groups) {
        if (ndma == DMA_PER_WAVE) {
            if (groups >= 2) wait_vm(std::integral_constant<int, 2 * GL_FULL>{});
            else if (groups == 1) wait_vm(std::integral_constant<int, GL_FULL>{});
            else wait_vm(std::integral_constant<int, 0>{});
        } else {
            if (groups >= 2) wait_vm(std::integral_constant<int, 2 * GL_NODMA>{});
            else if (groups == 1) wait_vm(std::integral_constant<int, GL_NODMA>{});
            else wait_vm(std::integral_constant<int, 0>{});
        }
    };

    f4_t acc[NP][MTT];

    // fragment read inside a stage: row mt*16 + c, chunk (4j+g) ^ c
    auto bfrag = [&](int st, int mt, int j) -> h8_t {
        const uint8_t* src = stage_ptr(st) + (mt * 16 + c) * ROWB + (((4 * j + g) ^ c) << 4);
        return bits_as<h8_t>(*reinterpret_cast<const u4_t*>(src));
    };

    // write-back ablation: this lane's 8 channels of step j, column 16p + c
    auto wb_at = [&](int p, int j) -> uint8_t* {
        return lds_wb + ((size_t)(wave * NP * 16 + p * 16 + c) * WB_RS + 32 * j + 8 * g) * 2;
    };

    // Fragments carried from one k-group to the next: the barrier of a
    // k-group sits before its last k-step, and that step's matrix
    // instructions cover the LDS fragment reads and the dequant of the next
    // k-group's first step, so no k-group starts with the matrix units
    // waiting on LDS latency behind a barrier.
    h8_t fa[2][NP];    // weights (A operand), double-buffered over k-steps
    h8_t fb[2][MTT];   // activations (B operand)
    Deq dcur[NP];      // dequant constants of the current k-group
    auto make_d = [&](int st, Deq (&d)[NP]) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < NP; ++p) d[p] = make_deq(sr[st][p], (zr[st][p] >> (4 * (c & 7))) & 15u);
        if constexpr (WB != 0) {
            // the conventional order: dequantize the whole k-group of weights
            // into the LDS tile first (same-wave LDS operations stay ordered)
#pragma unroll
            for (int p = 0; p < NP; ++p)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    *reinterpret_cast<h8_t*>(wb_at(p, j)) = dequant8(wr[st][p][j], d[p]);
        }
    };
    auto afrag = [&](int st, int p, int j, const Deq (&d)[NP]) -> h8_t {
        if constexpr (WB != 0) return *reinterpret_cast<const h8_t*>(wb_at(p, j));
        else return dequant8(wr[st][p][j], d[p]);
    };
    auto load_step0 = [&](int st) __attribute__((always_inline)) {
        make_d(st, dcur);
#pragma unroll
        for (int p = 0; p < NP; ++p) fa[0][p] = afrag(st, p, 0, dcur);
#pragma unroll
        for (int mt = 0; mt < MTT; ++mt) fb[0][mt] = bfrag(st, mt, 0);
    };
    // One k-group on stage / ring slot st, its step-0 fragments already in
    // fa[0], fb[0].  At its barrier at most `wgroups` k-groups of this wave's
    // loads stay in flight; `next`: a k-group follows in slot st+1.
    auto kgroup = [&](int st, int wgroups, bool next) __attribute__((always_inline)) {
        const int sn = (st + 1) % NST;
        Deq dn[NP];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int cu = j & 1, nx = cu ^ 1;
            if (j == 3 && next) make_d(sn, dn);
#pragma unroll
            for (int mt = 0; mt < MTT; ++mt) {
#pragma unroll
                for (int p = 0; p < NP; ++p) acc[p][mt] = mfma16(fa[cu][p], fb[cu][mt], acc[p][mt]);
                if (j < 3) fb[nx][mt] = bfrag(st, mt, j + 1);
                else if (next) fb[nx][mt] = bfrag(sn, mt, 0);
            }
            if (j < 3) {
#pragma unroll
                for (int p = 0; p < NP; ++p) fa[nx][p] = afrag(st, p, j + 1, dcur);
            } else if (next) {
#pragma unroll
                for (int p = 0; p < NP; ++p) fa[nx][p] = afrag(sn, p, 0, dn);
            }
            constexpr int VPER = (13 * NP + MTT - 1) / MTT;  // dequant VALU ops per block
#pragma unroll
            for (int mt = 0; mt < MTT; ++mt) {
                __builtin_amdgcn_sched_group_barrier(0x008, NP, 0);   // matrix
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // LDS read
                __builtin_amdgcn_sched_group_barrier(0x002, VPER, 0); // VALU
            }
            if (j == 2) {
                // After the barrier k-group st+1 has landed for every wave,
                // and every wave's reads of stage st (step 3, just issued)
                // have returned, so stage st may be refilled once the next
                // k-group starts.  The step-3 instructions below need those
                // fragments first anyway.
                wait_groups(wgroups);
                wait_lds();
                barrier();
                sched_fence();
            }
        }
        if (next) {
#pragma unroll
            for (int p = 0; p < NP; ++p) dcur[p] = dn[p];
        }
    };

    // acc = x[m0 .. m0+BM) [k-groups kb .. ke) . W[.., this wave's columns)
    auto run = [&](int kb, int ke) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int mt = 0; mt < MTT; ++mt) acc[p][mt] = f4_t{0.f, 0.f, 0.f, 0.f};
        // prologue: k-groups kb .. kb+NST-2 in flight, then wait for kb
#pragma unroll
        for (int i = 0; i < NST - 1; ++i)
            if (kb + i < ke) fetch(i, kb + i);
        wait_groups(min(NST - 2, ke - kb - 1));
        barrier();
        sched_fence();
        load_step0(0);

        // steady state: straight-line body (unconditional requests) so the
        // compiler's own wait analysis keeps the requested k-groups in flight;
        // k-group kg+i+NST-1 goes into the slot k-group kg+i-1 left
        int kg = kb;
        for (; kg + 2 * NST - 1 <= ke; kg += NST) {
#pragma unroll
            for (int i = 0; i < NST; ++i) {
                fetch((i + NST - 1) % NST, kg + i + NST - 1);
                kgroup(i, NST - 2, true);
            }
        }
        // tail
        for (; kg < ke; kg += NST) {
#pragma unroll
            for (int i = 0; i < NST; ++i) {
                const int k = kg + i;
                if (k < ke) {
                    if (k + NST - 1 < ke) fetch((i + NST - 1) % NST, k + NST - 1);
                    kgroup(i, min(NST - 2, ke - k - 2), k + 1 < ke);
                }
            }
        }
    };

    // (gated form: NP even and ntw even, so tiles p, p+1 are a gate tile
    // and its up tile)
    auto store_y = [&](const f4_t (&v)[NP][MTT]) __attribute__((always_inline)) {
        if constexpr (!EP) {
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                if (ntw + p >= NT) continue;
                const int n = (ntw + p) * 16 + 4 * g;
#pragma unroll
                for (int mt = 0; mt < MTT; ++mt) {
                    const int m = m0 + mt * 16 + c;
                    if (m < mend) store_h4(y + (size_t)m * N + n, v[p][mt]);
                }
            }
            return;
        }
        if (NP % 2 == 0 && epi.act) {
#pragma unroll
            for (int p = 0; p < NP; p += 2) {
                if (ntw + p >= NT) continue;
#pragma unroll
                for (int mt = 0; mt < MTT; ++mt) {
                    const int m = m0 + mt * 16 + c;
                    if (m < mend) store_gated(y, epi, m, N, (ntw + p) * 16 + 4 * g, v[p][mt], v[(p + 1) % NP][mt]);
                }
            }
            return;
        }
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            if (ntw + p >= NT) continue;
            const int n = (ntw + p) * 16 + 4 * g;
#pragma unroll
            for (int mt = 0; mt < MTT; ++mt) {
                const int m = m0 + mt * 16 + c;
                if (m < mend) store_out(y, epi, m, N, n, v[p][mt]);
            }
        }
    };

    if (n_splits > 0) {
        // ---- data-parallel / split-K: one (tile, K slice) per workgroup
        // (grouped: n_mtiles is the host's upper bound of the m-tiles; the
        // workgroups past the actual tile count exit)
        const int nblk = n_mtiles * n_ntiles * n_splits;
        const int per_xcd = gridDim.x >> 3;
        const int t = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
        if (t >= nblk) return;
        const int split = t / (n_mtiles * n_ntiles);
        const int tin = t - split * (n_mtiles * n_ntiles);
        if (tin >= n_mt * n_ntiles) return;
        set_tile(tin);
        const int kb = split * kg_per_split;
        run(kb, min(KG, kb + kg_per_split));
        if (n_splits == 1) {
            store_y(acc);
            return;
        }
        const int rows_out = GRP ? ga.routed : M;
        float* part = ws + kSkCounterBytes / sizeof(float) + (size_t)split * rows_out * N;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            if (ntw + p >= NT) continue;
            const int n = (ntw + p) * 16 + 4 * g;
#pragma unroll
            for (int mt = 0; mt < MTT; ++mt) {
                const int m = m0 + mt * 16 + c;
                if (m < mend) *reinterpret_cast<f4_t*>(part + (size_t)m * N + n) = acc[p][mt];
            }
        }
        return;
    }

    // ---- stream-K: whole rounds of tiles first, one tile per workgroup
    // (tiles wid, wid + G, ..), then the remaining tiles x k-groups units in
    // equal contiguous ranges: this workgroup owns units [u0, u1) of them.
    // The host launches 8 <= gridDim.x <= tiles * KG, a multiple of 8; the
    // stream-K part keeps at least gridDim.x units, so every range is
    // non-empty and a tile's contributors are consecutive.  Workgroups of
    // one XCD take consecutive ranges, so at any moment they work on a few
    // n-tiles at the same k offset (shared in L2); a stream-K partition of
    // every tile would start them at staggered k offsets instead.
    int64_t U = (int64_t)n_mt * n_ntiles * KG;
    int G = gridDim.x;
    int wid = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    int64_t u0, u1, ub = 0;
    if constexpr (GRP) {
        // the unit count is known only here: use the largest multiple of 8
        // workgroups not above it (the rest exit), or, with fewer than 8
        // units, one workgroup per whole tile
        const int ge = (int)(min<int64_t>(G, U) / 8 * 8);
        if (ge >= 8) {
            if ((int)(blockIdx.x >> 3) >= (ge >> 3)) return;
            G = ge;
            wid = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
        } else {
            if ((int64_t)blockIdx.x * KG >= U) return;
            G = 0;
        }
    }
    if (G == 0) {
        u0 = (int64_t)blockIdx.x * KG;
        u1 = u0 + KG;
    } else {
        const int T = n_mt * n_ntiles;
        int tdp = T / G * G;
        // the stream-K part takes 1/2 to 3/2 tiles per workgroup: smaller
        // pieces cost more in fix-ups than the idle compute units they save
        if (tdp > 0 && tdp < T && (2 * (T - tdp) < G || (int64_t)(T - tdp) * KG < G)) tdp -= G;
        for (int t = wid; t < tdp; t += G) {
            set_tile(t);
            run(0, KG);
            store_y(acc);
            __syncthreads();  // LDS stages are reused by the next tile
        }
        ub = (int64_t)tdp * KG;
        U -= ub;
        u0 = ub + (int64_t)wid * U / G;
        u1 = ub + (int64_t)(wid + 1) * U / G;
    }
    unsigned* counters = reinterpret_cast<unsigned*>(ws);
    // partial-tile slot: thread-major f4 at ((wave * NP + p) * MTT + mt) * 64 + lane
    constexpr uint32_t SLOT_BYTES = (uint32_t)WAVES * NP * MTT * 64 * 16;
    const rsrc_t rp = make_rsrc(ws + kSkCounterBytes / sizeof(float), (uint32_t)(2 * gridDim.x) * SLOT_BYTES);
    auto slot_off = [&](int p, int mt) -> uint32_t {
        return (uint32_t)((((wave * NP + p) * MTT + mt) * 64 + lane) * 16);
    };
    __shared__ int sk_last;
    for (int64_t u = u0; u < u1;) {
        const int tt = (int)(u / KG);
        const int kb = (int)(u - (int64_t)tt * KG);
        const int ke = (int)min<int64_t>(KG, kb + (u1 - u));
        set_tile(tt);
        run(kb, ke);
        if (kb == 0 && ke == KG) {
            store_y(acc);
        } else {
            const int64_t tb = (int64_t)tt * KG - ub;            // stream-K units before the tile
            const int w0 = (int)(((tb + 1) * G - 1) / U);        // owner of the tile's first unit
            const int w1 = (int)(((tb + KG) * G - 1) / U);       // ... and of its last
            // slot 2w: the piece that starts w's range; 2w+1: the piece that ends it
            const uint32_t mine = uniform((uint32_t)(2 * wid + (u == u0 ? 0 : 1)) * SLOT_BYTES);
#pragma unroll
            for (int p = 0; p < NP; ++p)
#pragma unroll
                for (int mt = 0; mt < MTT; ++mt)
                    __builtin_amdgcn_raw_buffer_store_b128(bits_as<u4_t>(acc[p][mt]), rp, slot_off(p, mt), mine,
                                                           kCoherentAux);
            wait_all();       // this wave's partial is written through
            __syncthreads();  // ... and every wave's
            if (threadIdx.x == 0)
                sk_last = __hip_atomic_fetch_add(&counters[w1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                          (unsigned)(w1 - w0);
            __syncthreads();
            if (sk_last) {
                // sum the pieces in k order: contributor w0, w0+1, .., w1
#pragma unroll
                for (int p = 0; p < NP; ++p) {
#pragma unroll
                    for (int mt = 0; mt < MTT; ++mt) {
                        f4_t sum = f4_t{0.f, 0.f, 0.f, 0.f};
                        for (int w = w0; w <= w1; ++w) {
                            f4_t v;
                            if (w == wid) {
                                v = acc[p][mt];
                            } else {
                                const int first = (int64_t)w * U / G >= tb ? 0 : 1;
                                v = bits_as<f4_t>(__builtin_amdgcn_raw_buffer_load_b128(
                                    rp, slot_off(p, mt), uniform((uint32_t)(2 * w + first) * SLOT_BYTES),
                                    kCoherentAux));
                            }
                            sum = w == w0 ? v : sum + v;
                        }
                        acc[p][mt] = sum;
                    }
                }
                store_y(acc);
                if (threadIdx.x == 0)
                    __hip_atomic_store(&counters[w1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        u += ke - kb;
        __syncthreads();  // LDS stages and sk_last are reused by the next piece
    }
}

// ---------------------------------------------------------------------------
// Sliced stream kernel (M <= 16, bandwidth-bound).
//
// The stream kernel gives a workgroup a few n-tiles and the whole K, so every
// workgroup reads all of x: at M = 16 that is 2 (two n-tiles per wave) to 4
// bytes of activations from L2 per byte of packed weights, and once 16 rows
// of K channels outgrow its LDS they come as global loads.  Here the 8 waves
// of a workgroup split the columns instead (wave w streams n-tiles
// 8*NPW*cg + NPW*w .. +NPW-1 of column group cg) and the workgroups split K
// into S slices of at most 16 k-groups.  A workgroup copies its slice of x
// (M rows x its k-groups) into LDS once with the 16-byte LDS-DMA load, and all
// 8 waves read their fragments from there, so activations cost 1/(2 NPW)
// byte per weight byte.  Inside a 256-byte piece of the slice (one row, one
// k-group) the 16-byte chunk with channels 8q .. 8q+7 sits at position
// q ^ (row % 16), so the 16 rows of a fragment read hit distinct banks.  Each
// wave then runs the stream kernel's single pass over its units: specialised
// on the unit count, a few units requested ahead, every unit multiplied as it
// lands; weights are loaded and dequantized straight into VGPRs as in the
// other kernels.
//
// With S > 1 each workgroup writes its fp32 partial columns with
// device-coherent stores and bumps its column group's arrival counter; the
// last of the S to arrive adds the partials in slice order (so the result
// does not depend on who is last), applies the epilogue, rounds once, stores
// y and re-arms the counter.  Workgroup ids map onto (slice, column group)
// slice-major with consecutive ids on one XCD, so the workgroups of an XCD
// share one activation slice in its L2.
// ---------------------------------------------------------------------------
constexpr int kKsWaves = 8;
constexpr int kKsMaxKg = kStreamSinglePass;   // k-groups per slice
[[maybe_unused]] constexpr size_t kKsLds = 64 * 1024;          // LDS bytes for the slice (16 rows x 16 k-groups)

template <int NPW>
__global__ void __launch_bounds__(64 * kKsWaves)
kstream_kernel(const uint16_t* __restrict__ x, const u4_t* __restrict__ pw,
               const uint16_t* __restrict__ ps, const uint32_t* __restrict__ pz,
               uint16_t* __restrict__ y, float* __restrict__ ws, int M, int N, int K,
               int kgps, int n_cg, int S, Epi epi)
{
    extern __shared__ __attribute__((aligned(1024))) uint8_t xs[];
    __shared__ int ks_last;
    const int KG = K >> 7;
    const int NT = N >> 4;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = lane & 15;
    const int g = lane >> 4;
    // gridDim.x is a multiple of 8; ids past the n_cg * S workgroups exit
    const int t = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    if (t >= n_cg * S) return;
    const int s = t / n_cg;
    const int cg = t - s * n_cg;
    const int kb = s * kgps;
    const int nk = min(KG, kb + kgps) - kb;   // 1 .. 16: the host leaves no slice empty
    const int ntw = cg * (kKsWaves * NPW) + wave * NPW;

    const rsrc_t rw = make_rsrc(pw, (uint32_t)((size_t)K * N / 2));
    const rsrc_t rs = make_rsrc(ps, (uint32_t)((size_t)K * N / 64));
    const rsrc_t rz = make_rsrc(pz, (uint32_t)((size_t)K * N / 256));
    const rsrc_t rx = make_rsrc(x, (uint32_t)((size_t)M * K * 2));
    // n-tiles past the end are clamped to the last one: computed on valid
    // data, never stored
    uint32_t ubase[NPW];
#pragma unroll
    for (int p = 0; p < NPW; ++p) ubase[p] = (uint32_t)min(ntw + p, NT - 1) * KG;
    const uint32_t vw = lane * 16;
    const uint32_t vs = c * 2;
    const uint32_t vz = (c >> 3) * 4;

    // Copy the slice: LDS chunk i (16 bytes) is row i / (16 nk), chunk
    // position q = i % (16 nk) of that row's slice, holding source chunk
    // (q & ~15) | ((q ^ row) & 15).  Instruction i0 / 64 moves chunks
    // i0 .. i0+63; lanes past the last chunk re-read it into the padding of
    // the allocation (whole KiB).
    const int chunks = M * nk * 16;
    for (int i0 = wave * 64; i0 < chunks; i0 += 64 * kKsWaves) {
        const int idx = min(i0 + lane, chunks - 1);
        const int row = idx / (nk * 16);
        const int q = idx - row * nk * 16;
        const int qs = (q & ~15) | ((q ^ row) & 15);
        dma16(rx, xs + (size_t)i0 * 16, (uint32_t)(row * K + kb * 128 + qs * 8) * 2, 0);
    }

    // fragment of step j: row c (rows past M read row M-1), channels
    // 32j + 8g .. +7 of the k-group
    const int row = min(c, M - 1);
    uint32_t xq[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) xq[j] = (uint32_t)(row * nk * 256) + ((((4 * j + g) ^ row) & 15) << 4);
    auto load_x = [&](u4_t (&xb)[4], int kl) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) xb[j] = *reinterpret_cast<const u4_t*>(xs + xq[j] + kl * 256);
    };
    auto load_w = [&](WStage<NPW>& st, int kg) __attribute__((always_inline)) {
#pragma unroll
        for (int p = 0; p < NPW; ++p) {
            const uint32_t u = uniform(ubase[p] + kg);
            st.w[p] = ld128(rw, vw, u * 1024u);
            st.s[p] = ld16(rs, vs, u * 32u);
            st.z[p] = ld32(rz, vz, u * 8u);
        }
    };
    f4_t acc[NPW];
#pragma unroll
    for (int p = 0; p < NPW; ++p) acc[p] = f4_t{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const WStage<NPW>& st, const u4_t (&xb)[4]) __attribute__((always_inline)) {
        Deq d[NPW];
#pragma unroll
        for (int p = 0; p < NPW; ++p) d[p] = make_deq(st.s[p], (st.z[p] >> (4 * (c & 7))) & 15u);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int p = 0; p < NPW; ++p) acc[p] = mfma16(dequant8(st.w[p][j], d[p]), bits_as<h8_t>(xb[j]), acc[p]);
    };

    u4_t xf[2][4];
    with_count<kKsMaxKg>(nk, [&](auto nkc) {
        constexpr int NKC = decltype(nkc)::value;
        constexpr int LA = NKC < kStreamLookahead ? NKC : kStreamLookahead;
        constexpr int R = LA + 1;
        WStage<NPW> sring[R];
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            load_w(sring[i], kb + i);
            sched_fence();
        }
        if constexpr (NKC > 0) {
            // this wave's copy instructions, issued before these 3 * NPW * LA
            // loads, have landed; after the barrier every wave's have (all
            // waves of the workgroup have the same unit count)
            wait_vm<3 * NPW * LA>();
            barrier();
            asm volatile("" ::: "memory");
            sched_fence();
            load_x(xf[0], 0);
#pragma unroll
            for (int i = 0; i < NKC; ++i) {
                if (i + 1 < NKC) load_x(xf[(i + 1) & 1], i + 1);
                compute(sring[i % R], xf[i & 1]);
                if (i + LA < NKC) load_w(sring[(i + LA) % R], kb + i + LA);
                sched_fence();
            }
        }
    });

    // row c, columns 16 * (ntw + p) + 4g .. +3 (gated form: NPW == 2 and ntw
    // even, so tile 0 is a gate tile and tile 1 its up tile)
    auto store = [&](const f4_t (&v)[NPW]) __attribute__((always_inline)) {
        if (c >= M) return;
        if (NPW == 2 && epi.act) {
            if (ntw < NT) store_gated(y, epi, c, N, ntw * 16 + 4 * g, v[0], v[NPW - 1]);
            return;
        }
#pragma unroll
        for (int p = 0; p < NPW; ++p)
            if (ntw + p < NT) store_out(y, epi, c, N, (ntw + p) * 16 + 4 * g, v[p]);
    };
    if (S == 1) {
        store(acc);
        return;
    }
    // partials: slot (cg, slice) holds the workgroup's 8 * NPW tiles, 1 KiB each
    constexpr uint32_t WG_BYTES = kKsWaves * NPW * 1024;
    unsigned* counters = reinterpret_cast<unsigned*>(ws);
    const rsrc_t rp = make_rsrc(ws + kSkCounterBytes / sizeof(float), (uint32_t)n_cg * S * WG_BYTES);
    auto slot = [&](int ss, int p) {
        return uniform((uint32_t)(cg * S + ss) * WG_BYTES + (uint32_t)(wave * NPW + p) * 1024u);
    };
#pragma unroll
    for (int p = 0; p < NPW; ++p)
        __builtin_amdgcn_raw_buffer_store_b128(bits_as<u4_t>(acc[p]), rp, lane * 16u, slot(s, p), kCoherentAux);
    wait_all();       // this wave's partials are written through
    __syncthreads();  // ... and every wave's
    if (threadIdx.x == 0)
        ks_last = __hip_atomic_fetch_add(&counters[cg], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                  (unsigned)(S - 1);
    __syncthreads();
    if (!ks_last) return;
    f4_t tot[NPW];
#pragma unroll
    for (int p = 0; p < NPW; ++p) {
        f4_t sum = f4_t{0.f, 0.f, 0.f, 0.f};
        for (int ss = 0; ss < S; ++ss) {
            const f4_t v = ss == s ? acc[p]
                                   : bits_as<f4_t>(__builtin_amdgcn_raw_buffer_load_b128(rp, lane * 16u, slot(ss, p),
                                                                                        kCoherentAux));
            sum = ss == 0 ? v : sum + v;
        }
        tot[p] = sum;
    }
    store(tot);
    if (threadIdx.x == 0) __hip_atomic_store(&counters[cg], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Tiled kernel on the 32x32x16 matrix instruction (large M).
//
// The tiles, schedules (data-parallel, split-K, stream-K with the
// last-arriver fix-up), XCD-aware tile order and the 4-stage activation ring
// in LDS are those of tiled_kernel.  What differs is the matrix step: each
// wave multiplies pairs of n-tiles (32 output columns) with
// v_mfma_f32_32x32x16_f16, one 32 x 16 weight operand against BM/32
// activation operands of 32 rows per 16-channel step, so a k-group takes
// half as many matrix instructions for the same fragment reads and the same
// dequantization.
//
// The QPK16 units serve this operand without repacking.  Lane l of the
// instruction holds output column l % 32 of the pair (n-tile t = (l/16) % 2,
// column c = l % 16) and channels 8h .. 8h+7 (h = l / 32) of the step.  It
// loads the 16 bytes of QPK16 lane 16h + c of n-tile t's unit, whose words
// hold channels 32j + 8h + e, and those of QPK16 lane 16(h+2) + c, channels
// 32j + 16 + 8h + e.  Step s = 2j (first load, word j) and s = 2j + 1
// (second load, word j) then covers channels 16s + 8h + e for every row, the
// k assignment the activation operand uses too: lane l reads row l % 32 of
// its block, channel chunk 2s + h of the stage.
//
// Output: lane l holds row l % 32 of a block and, in accumulator 4b + i, the
// column 8b + 4h + i of the pair, so every lane stores four 8-byte quads per
// block (b = 0, 1 in the first n-tile, b = 2, 3 in the second).
// ---------------------------------------------------------------------------
typedef float f16v_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ f16v_t mfma32(const h8_t& a, const h8_t& b, const f16v_t& c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

template <int BM, int WN, bool EP = false>
__global__ void __launch_bounds__(64 * kTiledWaves, 1)
tiled32_kernel(const uint16_t* __restrict__ x, const u4_t* __restrict__ pw,
               const uint16_t* __restrict__ ps, const uint32_t* __restrict__ pz,
               uint16_t* __restrict__ y, float* __restrict__ ws, int M, int N, int K,
               int kg_per_split, int n_mtiles, int n_ntiles, int n_splits, Epi epi)
{
    constexpr int WAVES = kTiledWaves;
    constexpr int NST = kTiledStages;
    constexpr int NPR = WN / 32;                  // n-tile pairs per wave
    constexpr int NP = 2 * NPR;                   // n-tiles per wave
    constexpr int MB = BM / 32;                   // 32-row blocks
    constexpr int ROWB = 256;                     // bytes per activation row of a stage
    constexpr int STAGE = BM * ROWB;
    constexpr int NDMA = STAGE / 1024;            // 1 KiB LDS-DMA instructions per stage
    constexpr int DMA_PER_WAVE = (NDMA + WAVES - 1) / WAVES;
    static_assert(WN % 32 == 0 && BM % 32 == 0, "pairs of n-tiles and 32-row blocks");
    static_assert(NDMA >= 1 && STAGE % 1024 == 0 && (NDMA % WAVES == 0 || NDMA < WAVES), "DMA split");
    static_assert(2 * (DMA_PER_WAVE + 4 * NPR) < 64, "vmcnt range");
    static_assert(NST == 4, "stage objects below");
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s0[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s1[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s2[STAGE];
    __shared__ __attribute__((aligned(1024))) uint8_t lds_s3[STAGE];
    auto stage_ptr = [&](int st) -> uint8_t* {
        return st == 0 ? lds_s0 : st == 1 ? lds_s1 : st == 2 ? lds_s2 : lds_s3;
    };

    const int KG = K >> 7;
    const int NT = N >> 4;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = lane & 15;          // column inside the n-tile
    const int tp = (lane >> 4) & 1;   // n-tile of the pair
    const int h = lane >> 5;          // channel half of a 16-channel step
    const int r32 = lane & 31;        // row inside a 32-row block

    const size_t wbytes = (size_t)K * N / 2;
    const rsrc_t rw = make_rsrc(pw, (uint32_t)wbytes);
    const rsrc_t rs = make_rsrc(ps, (uint32_t)(wbytes / 32));
    const rsrc_t rz = make_rsrc(pz, (uint32_t)(wbytes / 128));
    const rsrc_t rx = make_rsrc(x, (uint32_t)((size_t)M * K * 2));
    const int ndma = NDMA >= WAVES ? DMA_PER_WAVE : (wave < NDMA ? 1 : 0);

    int m0 = 0;     // first row of the tile
    int ntw = 0;    // first n-tile of this wave
    // per pair: this lane's byte offsets of its n-tile's first unit (packed
    // weights at its QPK16 lane 16h + c, scales, zeros); n-tiles past the
    // end are clamped to the last one (computed, never stored)
    uint32_t vw[NPR], vs[NPR], vz[NPR];
    uint32_t vx[DMA_PER_WAVE];
    auto set_tile = [&](int t) __attribute__((always_inline)) {
        m0 = (t % n_mtiles) * BM;
        const int ntile = (t / n_mtiles) % n_ntiles;
        ntw = ntile * (WAVES * NP) + wave * NP;
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) {
            const uint32_t u = (uint32_t)min(ntw + 2 * pr + tp, NT - 1) * (uint32_t)KG;
            vw[pr] = u * 1024u + (uint32_t)(16 * h + c) * 16u;
            vs[pr] = u * 32u + (uint32_t)c * 2u;
            vz[pr] = u * 8u + (uint32_t)(c >> 3) * 4u;
        }
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i) {
            const int rr = (wave + i * WAVES) * 4 + (lane >> 4);
            const int row = min(m0 + rr, M - 1);
            vx[i] = ((uint32_t)row * (uint32_t)K + 8 * ((lane & 15) ^ (rr & 15))) * 2;
        }
    };

    u4_t wa[NST][NPR], wb[NST][NPR];
    uint32_t sr[NST][NPR], zr[NST][NPR];
    auto fetch = [&](int st, int kg) __attribute__((always_inline)) {
        const uint32_t soff = uniform((uint32_t)kg * 256u);
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i)
            if (i < ndma) dma16(rx, stage_ptr(st) + (wave + i * WAVES) * 1024, vx[i], soff);
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) {
            wa[st][pr] = ld128(rw, vw[pr], uniform((uint32_t)kg * 1024u));
            wb[st][pr] = ld128(rw, vw[pr] + 512u, uniform((uint32_t)kg * 1024u));
            sr[st][pr] = ld16(rs, vs[pr], uniform((uint32_t)kg * 32u));
            zr[st][pr] = ld32(rz, vz[pr], uniform((uint32_t)kg * 8u));
        }
    };
    auto wait_vmc = [](auto n) { __builtin_amdgcn_s_waitcnt(0x0F70 | (n & 15) | ((n >> 4) << 14)); };
    constexpr int GL_FULL = DMA_PER_WAVE + 4 * NPR;
    constexpr int GL_NODMA = 4 * NPR;
    auto wait_groups = [&](int groups) {
        if (ndma == DMA_PER_WAVE) {
            if (groups >= 2) wait_vmc(std::integral_constant<int, 2 * GL_FULL>{});
            else if (groups == 1) wait_vmc(std::integral_constant<int, GL_FULL>{});
            else wait_vmc(std::integral_constant<int, 0>{});
        } else {
            if (groups >= 2) wait_vmc(std::integral_constant<int, 2 * GL_NODMA>{});
            else if (groups == 1) wait_vmc(std::integral_constant<int, GL_NODMA>{});
            else wait_vmc(std::integral_constant<int, 0>{});
        }
    };

    f16v_t acc[NPR][MB];
    // activation operand of step s: row mb*32 + r32, channel chunk 2s + h
    // (stored at position (2s + h) ^ (row % 16), row % 16 == c)
    auto bfrag = [&](int st, int mb, int s) -> h8_t {
        const uint8_t* src = stage_ptr(st) + (mb * 32 + r32) * ROWB + (((2 * s + h) ^ c) << 4);
        return bits_as<h8_t>(*reinterpret_cast<const u4_t*>(src));
    };
    Deq dcur[NPR];
    auto make_d = [&](int st, Deq (&d)[NPR]) __attribute__((always_inline)) {
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) d[pr] = make_deq(sr[st][pr], (zr[st][pr] >> (4 * (c & 7))) & 15u);
    };
    auto afrag = [&](int st, int pr, int s, const Deq (&d)[NPR]) -> h8_t {
        return dequant8((s & 1) ? wb[st][pr][s >> 1] : wa[st][pr][s >> 1], d[pr]);
    };
    h8_t fa[2][NPR];
    h8_t fb[2][MB];
    auto load_step0 = [&](int st) __attribute__((always_inline)) {
        make_d(st, dcur);
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) fa[0][pr] = afrag(st, pr, 0, dcur);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) fb[0][mb] = bfrag(st, mb, 0);
    };
    // One k-group (8 steps of 16 channels) on stage / ring slot st, its
    // step-0 operands already in fa[0], fb[0]; the operands of step s+1 are
    // read and dequantized under the matrix instructions of step s, the
    // last step's under those of the next k-group's first.
    auto kgroup = [&](int st, int wgroups, bool next) __attribute__((always_inline)) {
        const int sn = (st + 1) % NST;
        Deq dn[NPR];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const int cu = s & 1, nx = cu ^ 1;
            if (s == 7 && next) make_d(sn, dn);
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
                for (int pr = 0; pr < NPR; ++pr) acc[pr][mb] = mfma32(fa[cu][pr], fb[cu][mb], acc[pr][mb]);
                if (s < 7) fb[nx][mb] = bfrag(st, mb, s + 1);
                else if (next) fb[nx][mb] = bfrag(sn, mb, 0);
            }
            if (s < 7) {
#pragma unroll
                for (int pr = 0; pr < NPR; ++pr) fa[nx][pr] = afrag(st, pr, s + 1, dcur);
            } else if (next) {
#pragma unroll
                for (int pr = 0; pr < NPR; ++pr) fa[nx][pr] = afrag(sn, pr, 0, dn);
            }
            constexpr int VPER = (13 * NPR + MB - 1) / MB;  // dequant VALU ops per block
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                __builtin_amdgcn_sched_group_barrier(0x008, NPR, 0);   // matrix
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);     // LDS read
                __builtin_amdgcn_sched_group_barrier(0x002, VPER, 0);  // VALU
            }
            if (s == 6) {
                // k-group st+1 has landed for every wave, and every wave's
                // reads of stage st have returned (see tiled_kernel)
                wait_groups(wgroups);
                wait_lds();
                barrier();
                sched_fence();
            }
        }
        if (next) {
#pragma unroll
            for (int pr = 0; pr < NPR; ++pr) dcur[pr] = dn[pr];
        }
    };

    auto run = [&](int kb, int ke) __attribute__((always_inline)) {
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[pr][mb][v] = 0.f;
#pragma unroll
        for (int i = 0; i < NST - 1; ++i)
            if (kb + i < ke) fetch(i, kb + i);
        wait_groups(min(NST - 2, ke - kb - 1));
        barrier();
        sched_fence();
        load_step0(0);
        int kg = kb;
        for (; kg + 2 * NST - 1 <= ke; kg += NST) {
#pragma unroll
            for (int i = 0; i < NST; ++i) {
                fetch((i + NST - 1) % NST, kg + i + NST - 1);
                kgroup(i, NST - 2, true);
            }
        }
        for (; kg < ke; kg += NST) {
#pragma unroll
            for (int i = 0; i < NST; ++i) {
                const int k = kg + i;
                if (k < ke) {
                    if (k + NST - 1 < ke) fetch((i + NST - 1) % NST, k + NST - 1);
                    kgroup(i, min(NST - 2, ke - k - 2), k + 1 < ke);
                }
            }
        }
    };

    // quad b (0..3) of block mb of pair pr: columns 16(ntw+2pr) + 8b + 4h .. +3
    auto quad = [&](const f16v_t& v, int b) -> f4_t { return f4_t{v[4 * b], v[4 * b + 1], v[4 * b + 2], v[4 * b + 3]}; };
    auto store_y = [&](const f16v_t (&v)[NPR][MB]) __attribute__((always_inline)) {
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) {
            const int nb = (ntw + 2 * pr) * 16 + 4 * h;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int m = m0 + mb * 32 + r32;
                if (m >= M) continue;
                if (EP && epi.act) {
                    // gate quads b = 0, 1 with their up quads b + 2 (16 columns on)
                    if (ntw + 2 * pr < NT) {
                        store_gated(y, epi, m, N, nb, quad(v[pr][mb], 0), quad(v[pr][mb], 2));
                        store_gated(y, epi, m, N, nb + 8, quad(v[pr][mb], 1), quad(v[pr][mb], 3));
                    }
                    continue;
                }
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    if (ntw + 2 * pr + (b >> 1) >= NT) continue;
                    if constexpr (EP) store_out(y, epi, m, N, nb + 8 * b, quad(v[pr][mb], b));
                    else store_h4(y + (size_t)m * N + nb + 8 * b, quad(v[pr][mb], b));
                }
            }
        }
    };

    if (n_splits > 0) {
        // data-parallel / split-K: one (tile, K slice) per workgroup
        const int nblk = n_mtiles * n_ntiles * n_splits;
        const int per_xcd = gridDim.x >> 3;
        const int t = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
        if (t >= nblk) return;
        const int split = t / (n_mtiles * n_ntiles);
        const int tin = t - split * (n_mtiles * n_ntiles);
        set_tile(tin);
        const int kb = split * kg_per_split;
        run(kb, min(KG, kb + kg_per_split));
        if (n_splits == 1) {
            store_y(acc);
            return;
        }
        float* part = ws + kSkCounterBytes / sizeof(float) + (size_t)split * M * N;
#pragma unroll
        for (int pr = 0; pr < NPR; ++pr) {
            const int nb = (ntw + 2 * pr) * 16 + 4 * h;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
                const int m = m0 + mb * 32 + r32;
                if (m >= M) continue;
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    if (ntw + 2 * pr + (b >> 1) < NT)
                        *reinterpret_cast<f4_t*>(part + (size_t)m * N + nb + 8 * b) = quad(acc[pr][mb], b);
            }
        }
        return;
    }

    // ---- stream-K (see tiled_kernel): whole rounds of tiles first, then
    // equal contiguous ranges of the remaining tiles x k-groups units,
    // last-arriver fix-up in k order
    const int T = n_mtiles * n_ntiles;
    const int G = gridDim.x;
    const int wid = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    int tdp = T / G * G;
    if (tdp > 0 && tdp < T && (2 * (T - tdp) < G || (int64_t)(T - tdp) * KG < G)) tdp -= G;
    for (int t = wid; t < tdp; t += G) {
        set_tile(t);
        run(0, KG);
        store_y(acc);
        __syncthreads();  // LDS stages are reused by the next tile
    }
    const int64_t ub = (int64_t)tdp * KG;
    const int64_t U = (int64_t)T * KG - ub;
    const int64_t u0 = ub + (int64_t)wid * U / G;
    const int64_t u1 = ub + (int64_t)(wid + 1) * U / G;
    unsigned* counters = reinterpret_cast<unsigned*>(ws);
    // partial-tile slot: thread-major f4 at (((wave * NPR + pr) * MB + mb) * 4 + b) * 64 + lane
    constexpr uint32_t SLOT_BYTES = (uint32_t)WAVES * NPR * MB * 4 * 64 * 16;
    const rsrc_t rp = make_rsrc(ws + kSkCounterBytes / sizeof(float), (uint32_t)(2 * gridDim.x) * SLOT_BYTES);
    auto slot_off = [&](int pr, int mb, int b) -> uint32_t {
        return (uint32_t)(((((wave * NPR + pr) * MB + mb) * 4 + b) * 64 + lane) * 16);
    };
    __shared__ int sk_last;
    for (int64_t u = u0; u < u1;) {
        const int tt = (int)(u / KG);
        const int kb = (int)(u - (int64_t)tt * KG);
        const int ke = (int)min<int64_t>(KG, kb + (u1 - u));
        set_tile(tt);
        run(kb, ke);
        if (kb == 0 && ke == KG) {
            store_y(acc);
        } else {
            const int64_t tb = (int64_t)tt * KG - ub;
            const int w0 = (int)(((tb + 1) * G - 1) / U);
            const int w1 = (int)(((tb + KG) * G - 1) / U);
            const uint32_t mine = uniform((uint32_t)(2 * wid + (u == u0 ? 0 : 1)) * SLOT_BYTES);
#pragma unroll
            for (int pr = 0; pr < NPR; ++pr)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
#pragma unroll
                    for (int b = 0; b < 4; ++b)
                        __builtin_amdgcn_raw_buffer_store_b128(bits_as<u4_t>(quad(acc[pr][mb], b)), rp,
                                                               slot_off(pr, mb, b), mine, kCoherentAux);
            wait_all();
            __syncthreads();
            if (threadIdx.x == 0)
                sk_last = __hip_atomic_fetch_add(&counters[w1], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                          (unsigned)(w1 - w0);
            __syncthreads();
            if (sk_last) {
#pragma unroll
                for (int pr = 0; pr < NPR; ++pr) {
#pragma unroll
                    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
                        for (int b = 0; b < 4; ++b) {
                            f4_t sum = f4_t{0.f, 0.f, 0.f, 0.f};
                            for (int w = w0; w <= w1; ++w) {
                                f4_t v;
                                if (w == wid) {
                                    v = quad(acc[pr][mb], b);
                                } else {
                                    const int first = (int64_t)w * U / G >= tb ? 0 : 1;
                                    v = bits_as<f4_t>(__builtin_amdgcn_raw_buffer_load_b128(
                                        rp, slot_off(pr, mb, b), uniform((uint32_t)(2 * w + first) * SLOT_BYTES),
                                        kCoherentAux));
                                }
                                sum = w == w0 ? v : sum + v;
                            }
                            acc[pr][mb][4 * b] = sum[0];
                            acc[pr][mb][4 * b + 1] = sum[1];
                            acc[pr][mb][4 * b + 2] = sum[2];
                            acc[pr][mb][4 * b + 3] = sum[3];
                        }
                    }
                }
                store_y(acc);
                if (threadIdx.x == 0)
                    __hip_atomic_store(&counters[w1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        u += ke - kb;
        __syncthreads();  // LDS stages and sk_last are reused by the next piece
    }
}

// Sum of S fp32 partial outputs [S][rows][N] in split order, then the
// epilogue and one rounding to f16.  One thread per 4 output columns.
__global__ void __launch_bounds__(256)
splitk_reduce_kernel(const float* __restrict__ ws, uint16_t* __restrict__ y, int64_t rows, int N, int S, Epi epi)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int quads = (epi.act ? N / 2 : N) / 4;   // output quads per row
    if (i >= rows * quads) return;
    const int64_t m = i / quads;
    const int q = (int)(i - m * quads);
    const int64_t plane = rows * N / 4;             // quads per split
    auto sum_at = [&](int n) {
        const f4_t* p = reinterpret_cast<const f4_t*>(ws) + (m * N + n) / 4;
        f4_t sum = p[0];
        for (int s = 1; s < S; ++s) sum += p[(size_t)s * plane];
        return sum;
    };
    if (epi.act) {
        const int n = (q >> 2) * 32 + (q & 3) * 4;   // gate quad; its up quad is 16 columns on
        store_gated(y, epi, m, N, n, sum_at(n), sum_at(n + 16));
    } else {
        store_out(y, epi, m, N, q * 4, sum_at(q * 4));
    }
}

// ---------------------------------------------------------------------------
// Host side: validation, configuration, workspace, launch.
// ---------------------------------------------------------------------------
constexpr int kVariantStream = 1;
// LDS bytes the stream kernel may give to activations: gfx950's 160 KiB
// less the 16 KiB its waves' partial sums take at most (a workgroup above
// 80 KiB then has its compute unit to itself)
[[maybe_unused]] constexpr size_t kStreamLdsX = 144 * 1024;
[[maybe_unused]] constexpr size_t kDefaultLds = 64 * 1024;   // dynamic LDS without a raised limit
constexpr int kVariantTiled = 2;
constexpr int kVariantStreamK = 3;  // tiled kernel, stream-K schedule
// (variant 4, a balanced stream kernel, was withdrawn: it never won on a
// measured shape; the number stays reserved and is rejected)
constexpr int kVariantKStream = 5;  // sliced stream kernel
constexpr int kVariantTiled32 = 6;   // tiled kernel on the 32x32x16 instruction
constexpr int kVariantStreamK32 = 7; // the same, stream-K schedule

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// Column groups (8 waves x npw n-tiles) of the sliced stream kernel, and the
// fewest K slices that keep each slice within its 16 k-groups.
int ks_groups(int64_t N, int npw) { return ceil_div(N / 16, kKsWaves * npw); }
int ks_min_slices(int64_t K) { return ceil_div(K / 128, kKsMaxKg); }

bool is_tiled(int variant)
{
    return variant == kVariantTiled || variant == kVariantStreamK || variant == kVariantTiled32 ||
           variant == kVariantStreamK32;
}
bool is_streamk(int variant) { return variant == kVariantStreamK || variant == kVariantStreamK32; }
bool is_t32(int variant) { return variant == kVariantTiled32 || variant == kVariantStreamK32; }

// Bytes of one stream-K partial-tile slot.
size_t sk_slot_bytes(int bm, int wn) { return (size_t)bm * kTiledWaves * wn * sizeof(float); }

}  // namespace

#if QUICK_TILED
namespace quick {

template <class F>
int resident_per_cu(F* kernel)
{
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(kernel), 64 * kTiledWaves,
                                                     0) != hipSuccess ||
        n < 1)
        n = 1;
    return n;
}

// Workgroups of the tiled kernel that are resident at once on the current
// device (compute units x workgroups per compute unit); 256 when no device
// can be queried.
int tiled_resident(int bm, int wn, bool mfma32)
{
    static std::mutex mu;
    static std::map<std::pair<int, int>, int> cache;  // (device, tile id) -> workgroups
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
        (void)hipGetLastError();
        return 256;
    }
    const int id = bm * 1000 + wn + (mfma32 ? 1000000 : 0);
    std::lock_guard<std::mutex> lk(mu);
    auto it = cache.find({dev, id});
    if (it != cache.end()) return it->second;
    int per = 1;
    if (mfma32) {
        if (bm == 32 && wn == 32) per = resident_per_cu(&tiled32_kernel<32, 32>);
        else if (bm == 64 && wn == 32) per = resident_per_cu(&tiled32_kernel<64, 32>);
        else if (bm == 128 && wn == 32) per = resident_per_cu(&tiled32_kernel<128, 32>);
    } else if (bm == 16 && wn == 16) per = resident_per_cu(&tiled_kernel<16, 16>);
    else if (bm == 16 && wn == 32) per = resident_per_cu(&tiled_kernel<16, 32>);
    else if (bm == 32 && wn == 16) per = resident_per_cu(&tiled_kernel<32, 16>);
    else if (bm == 32 && wn == 32) per = resident_per_cu(&tiled_kernel<32, 32>);
    else if (bm == 64 && wn == 16) per = resident_per_cu(&tiled_kernel<64, 16>);
    else if (bm == 64 && wn == 32) per = resident_per_cu(&tiled_kernel<64, 32>);
    else if (bm == 128 && wn == 16) per = resident_per_cu(&tiled_kernel<128, 16>);
    else if (bm == 128 && wn == 32) per = resident_per_cu(&tiled_kernel<128, 32>);
    (void)hipGetLastError();
    const int g = std::min(cus * per, kSkMaxWorkgroups);
    cache[{dev, id}] = g;
    return g;
}

}  // namespace quick
#endif

namespace {

using quick::tiled_resident;

// The stream kernel's automatic shape: 2 n-tiles per wave for wide N, and
// waves per workgroup doubled while there are fewer than 2048 waves and
// each keeps >= 2 k-groups.
void stream_defaults(int64_t N, int64_t K, Plan* pl)
{
    const int64_t KG = K / 128;
    const int64_t NT = N / 16;
    pl->variant = kVariantStream;
    pl->wn = NT / 2 >= 512 ? 2 : 1;
    const int64_t wgs = (NT + pl->wn - 1) / pl->wn;
    int w = 1;
    while (w < 8 && wgs * w < 2048 && KG / (2 * w) >= 2) w *= 2;
    pl->split = w;
    pl->bm = 0;
    pl->kgps = 0;
}

int auto_plan(int64_t M, int64_t N, int64_t K, Plan* pl)
{
    const int64_t KG = K / 128;
    auto stream_plan = [&]() { stream_defaults(N, K, pl); };
    if (M <= 8) {
        // weights dominate; each wave streams its own k-range (no LDS tile)
        stream_plan();
        return QUICK_OK;
    }
    if (M <= 16 && K * N / 2 < ((int64_t)128 << 20) &&
        (int64_t)ks_groups(N, 1) * ks_min_slices(K) >= 128 && ks_groups(N, 1) <= kSkMaxWorkgroups) {
        // sliced stream kernel, one n-tile per wave, the fewest K slices (at
        // least 128 workgroups); the largest weight matrices stay on the
        // 16-row tiles, which stream them as fast
        pl->variant = kVariantKStream;
        pl->split = 0;
        pl->bm = 0;
        pl->wn = 1;
        pl->kgps = 0;
        return QUICK_OK;
    }
    // Tiled kernel: an 8-wave workgroup computes BM x (8*WN), sharing one
    // activation tile in LDS.  Small BM tiles fit several workgroups per CU,
    // so they split K until ~384 workgroups exist; the 64/128-row tiles run
    // one workgroup per CU and split only when fewer than 160 tiles exist.
    pl->variant = kVariantTiled;
    if (M <= 16) {
        pl->bm = 16;
        pl->wn = 16;
    } else if (M <= 32) {
        pl->bm = 32;
        pl->wn = 16;
    } else if (M <= 64) {
        // 64-row tiles of 16-column waves when they alone fill the chip,
        // else 32-row ones (split below)
        const bool wide = (int64_t)ceil_div(M, 64) * ceil_div(N, 128) >= 160;
        pl->bm = wide ? 64 : 32;
        pl->wn = 16;
    } else {
        // Mid M with a short or medium K, when the 128 x 256 tiles are too
        // few to fill the chip: 16-column waves on 128- or 64-row tiles
        // (twice the workgroups of 32-column waves, each weight dequantized
        // ceil(M / BM) times) when they fill it without splitting K.
        bool mid = false;
        if ((int64_t)ceil_div(M, 128) * ceil_div(N, 256) < 160 && KG < 128)
            for (int bm : {128, 64})
                if (!mid && (int64_t)ceil_div(M, bm) * ceil_div(N, 128) >= 160) {
                    pl->bm = bm;
                    pl->wn = 16;
                    mid = true;
                }
        // Otherwise the largest tile whose K slices stay long: a split that
        // leaves few k-groups per workgroup pays the pipeline fill and the
        // partial-sum pass for little work, and a smaller tile that needs
        // less splitting wins (narrow N or short K).
        if (mid) {
            pl->split = 1;
            pl->kgps = 0;
            return QUICK_OK;
        }
        static const int cand[3][2] = {{128, 32}, {64, 32}, {32, 16}};
        for (int c = M <= 96 ? 1 : 0; c < 3; ++c) {
            pl->bm = cand[c][0];
            pl->wn = cand[c][1];
            const int64_t t = (int64_t)ceil_div(M, pl->bm) * ceil_div(N, kTiledWaves * pl->wn);
            const int64_t tgt = pl->wn == 16 ? 256 : 160;
            int s = 1;
            while (t * s < tgt && KG / (2 * s) >= 4 && s < 8) s *= 2;
            if (ceil_div(KG, s) >= 12) break;
        }
    }
    const int64_t tiles = (int64_t)ceil_div(M, pl->bm) * ceil_div(N, kTiledWaves * pl->wn);
    if (pl->bm == 16 && tiles < 48) {
        // too few column tiles to feed the chip without heavy split-K
        stream_plan();
        return QUICK_OK;
    }
    pl->kgps = 0;
    // More tiles than resident workgroups with the last round of tiles
    // less than 75 % full, and a long K: stream-K runs the whole rounds as
    // tiles and spreads the rest of the tiles x k-groups work evenly, each
    // split tile having only a few pieces to add.  A nearly full last round,
    // or a single partial round, runs faster as whole tiles (the chip is
    // power-limited under this load, so idle compute units cost less than
    // the pieces' fix-ups).  Short K (each piece's pipeline fill and
    // partial-tile traffic weigh more) or fewer tiles: split-K, whose
    // separate reduction pass spreads the adding over the whole chip.
    const int64_t resident = tiled_resident(pl->bm, pl->wn);
    const int64_t slots = (tiles + resident - 1) / resident * resident;
    if (pl->bm >= 64 && KG >= 48 && tiles > resident && (slots - tiles) * 4 > slots) {
        pl->variant = kVariantStreamK;
        pl->split = 0;
        return QUICK_OK;
    }
    const int64_t target = pl->wn == 16 ? (M > 64 ? 256 : M > 32 ? 160 : 384) : 160;
    int s = 1;
    while (tiles * s < target && KG / (2 * s) >= 4 && s < 8) s *= 2;
    pl->split = s;
    return QUICK_OK;
}

// ---- tune table: shape -> configuration measured fastest by quick_tune
struct ShapeKey {
    int64_t M, N, K;
    bool operator<(const ShapeKey& o) const
    {
        return M != o.M ? M < o.M : N != o.N ? N < o.N : K < o.K;
    }
};
std::mutex g_tune_mu;
std::map<ShapeKey, quick_config_t> g_tune;

bool tuned_config(int64_t M, int64_t N, int64_t K, quick_config_t* out)
{
    std::lock_guard<std::mutex> lk(g_tune_mu);
    auto it = g_tune.find(ShapeKey{M, N, K});
    if (it == g_tune.end()) return false;
    *out = it->second;
    return true;
}

bool tiled32_supported(int bm, int wn)
{
    // (64 x 64 wave tiles spill registers)
    return (bm == 32 || bm == 64 || bm == 128) && wn == 32;
}

bool tiled_supported(int bm, int wn)
{
    return (bm == 16 || bm == 32 || bm == 64 || bm == 128) && (wn == 16 || wn == 32);
}

int make_plan(int64_t M, int64_t N, int64_t K, const quick_config_t* cfg, Plan* pl)
{
    auto_plan(M, N, K, pl);
    quick_config_t tuned;
    if (!cfg && tuned_config(M, N, K, &tuned)) cfg = &tuned;
    if (!cfg) return QUICK_OK;
    const int64_t KG = K / 128;
    if (cfg->variant < 0 || cfg->variant > 7 || cfg->variant == 4 || cfg->split_k < 0) return QUICK_ERR_INVALID_ARG;
    if (cfg->variant == kVariantKStream) {
        // split_k: K slices (0 = auto; raised to the minimum); tile_n:
        // n-tiles per wave (0 = 2); the arrival counters cover every column
        // group
        if (M > 16 || cfg->tile_m || (cfg->tile_n != 0 && cfg->tile_n != 1 && cfg->tile_n != 2) ||
            cfg->split_k > KG || ks_groups(N, 1) > kSkMaxWorkgroups)
            return QUICK_ERR_INVALID_ARG;
        pl->variant = kVariantKStream;
        pl->split = cfg->split_k;
        pl->bm = 0;
        pl->wn = cfg->tile_n ? cfg->tile_n : 2;
        pl->kgps = 0;
        return QUICK_OK;
    }
    if (cfg->variant == kVariantStream) {
        if (M > 64) return QUICK_ERR_INVALID_ARG;
        if (pl->variant != kVariantStream) stream_defaults(N, K, pl);
        if (cfg->split_k) {
            if (cfg->split_k != 1 && cfg->split_k != 2 && cfg->split_k != 4 && cfg->split_k != 8)
                return QUICK_ERR_INVALID_ARG;
            pl->split = cfg->split_k;
        }
        if (cfg->tile_n) {
            if (cfg->tile_n != 1 && cfg->tile_n != 2) return QUICK_ERR_INVALID_ARG;
            pl->wn = cfg->tile_n;
        }
    } else if (is_tiled(cfg->variant)) {
        if (!is_tiled(pl->variant)) {
            pl->bm = 64;
            pl->wn = 32;
            pl->split = 1;
        }
        if (is_streamk(pl->variant) != is_streamk(cfg->variant)) pl->split = is_streamk(cfg->variant) ? 0 : 1;
        if (is_t32(cfg->variant)) {
            // pairs of n-tiles, 32-row blocks
            pl->wn = std::max(pl->wn, 32);
            pl->bm = std::max(pl->bm, 32);
        }
        pl->variant = cfg->variant;
    }
    if (is_streamk(pl->variant)) {
        // split_k: persistent workgroups, a multiple of 8 (0 = all resident)
        if (cfg->split_k && (cfg->split_k % 8 != 0 || cfg->split_k > kSkMaxWorkgroups))
            return QUICK_ERR_INVALID_ARG;
        pl->split = cfg->split_k;
    }
    if (is_tiled(pl->variant)) {
        if (cfg->tile_m) {
            if (cfg->tile_m != 16 && cfg->tile_m != 32 && cfg->tile_m != 64 && cfg->tile_m != 128)
                return QUICK_ERR_INVALID_ARG;
            pl->bm = cfg->tile_m;
        }
        if (cfg->tile_n) {
            if (cfg->tile_n != 16 && cfg->tile_n != 32) return QUICK_ERR_INVALID_ARG;
            pl->wn = cfg->tile_n;
        }
        if (cfg->split_k && !is_streamk(pl->variant)) {
            if (cfg->split_k > KG) return QUICK_ERR_INVALID_ARG;
            pl->split = cfg->split_k;
        }
        if (is_t32(pl->variant) ? !tiled32_supported(pl->bm, pl->wn) : !tiled_supported(pl->bm, pl->wn))
            return QUICK_ERR_INVALID_ARG;
    }
    return QUICK_OK;
}

void finish_plan(int64_t M, int64_t N, int64_t K, Plan* pl)
{
    (void)M;
    if (pl->variant == kVariantKStream) {
        // automatic: the fewest slices (the best or within 6 % of the best
        // slice count on the bench shapes at M = 16)
        const int64_t KG = K / 128;
        const int smin = ks_min_slices(K);
        const int s = (int)std::min<int64_t>(std::max(pl->split, smin), KG);
        pl->kgps = ceil_div(KG, s);
        pl->split = ceil_div(KG, pl->kgps);  // no empty slices
        return;
    }
    if (is_streamk(pl->variant)) {
        // 8 <= workgroups <= tiles x k-groups, a multiple of 8: every
        // workgroup gets a non-empty range and the XCD mapping is exact
        const int64_t units = (int64_t)ceil_div(M, pl->bm) * ceil_div(N, kTiledWaves * pl->wn) * (K / 128);
        int64_t g = pl->split ? pl->split : tiled_resident(pl->bm, pl->wn, is_t32(pl->variant));
        g = std::min<int64_t>(g, units) / 8 * 8;
        if (g >= 8) {
            pl->split = (int)g;
            pl->kgps = 0;
            return;
        }
        // too little work: one workgroup per tile
        pl->variant = is_t32(pl->variant) ? kVariantTiled32 : kVariantTiled;
        pl->split = 1;
    }
    if (pl->variant == kVariantTiled || pl->variant == kVariantTiled32) {
        const int64_t KG = K / 128;
        if (pl->split > KG) pl->split = (int)KG;
        if (pl->split < 1) pl->split = 1;
        pl->kgps = ceil_div(KG, pl->split);
        pl->split = ceil_div(KG, pl->kgps);  // no empty splits
    }
}

// Workspace layout: kSkCounterBytes of stream-K arrival counters (zero
// between calls), then split-K partial outputs or stream-K partial tiles.
size_t plan_workspace(int64_t M, int64_t N, const Plan& pl)
{
    if (pl.variant == kVariantKStream && pl.split > 1)
        return kSkCounterBytes + (size_t)ks_groups(N, pl.wn) * pl.split * kKsWaves * pl.wn * 1024;
    if ((pl.variant == kVariantTiled || pl.variant == kVariantTiled32) && pl.split > 1)
        return kSkCounterBytes + (size_t)pl.split * M * N * sizeof(float);
    if (is_streamk(pl.variant)) return kSkCounterBytes + 2 * (size_t)pl.split * sk_slot_bytes(pl.bm, pl.wn);
    return 0;
}

// Library-owned workspace, one per (device, stream).  A buffer that a larger
// plan outgrows is retired but never freed: a graph captured while it was
// current keeps launching with its address.
struct WsKey {
    int dev;
    void* stream;
    bool operator<(const WsKey& o) const { return dev != o.dev ? dev < o.dev : stream < o.stream; }
};
struct WsBuf {
    void* ptr = nullptr;
    size_t bytes = 0;
};
std::mutex g_ws_mu;
std::map<WsKey, WsBuf> g_ws;
std::vector<void*> g_ws_retired;

int get_workspace(size_t need, hipStream_t stream, void** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return QUICK_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    WsBuf& b = g_ws[WsKey{dev, (void*)stream}];
    if (b.bytes < need) {
        // Allocating and clearing are not allowed on a capturing stream:
        // the caller gets a status and nothing is enqueued.
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
            (void)hipGetLastError();
            return QUICK_ERR_HIP;
        }
        if (cs != hipStreamCaptureStatusNone) return QUICK_ERR_CAPTURE;
        const size_t sz = std::max<size_t>(need, (size_t)1 << 20);
        void* p = nullptr;
        if (hipMalloc(&p, sz) != hipSuccess) {
            (void)hipGetLastError();
            return QUICK_ERR_HIP;
        }
        // arrival counters start at zero (every call leaves them zero)
        if (hipMemsetAsync(p, 0, kSkCounterBytes, stream) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipFree(p);
            return QUICK_ERR_HIP;
        }
        // work already enqueued (or captured) with the old buffer keeps it
        if (b.ptr) g_ws_retired.push_back(b.ptr);
        b.ptr = p;
        b.bytes = sz;
    }
    *out = b.ptr;
    return QUICK_OK;
}

}  // namespace

namespace quick {

#if QUICK_STREAM
// Raise a kernel's dynamic-LDS limit to `bytes`, once per (device, kernel):
// the attribute belongs to the device that is current when it is set.
bool lds_limit_set(const void* fn, size_t bytes)
{
    static std::mutex mu;
    static std::set<std::pair<int, const void*>> done;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    std::lock_guard<std::mutex> lk(mu);
    if (done.count({dev, fn})) return true;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) != hipSuccess) return false;
    done.insert({dev, fn});
    return true;
}

template <int MT, int NPW, int WAVES>
void launch_stream_t(const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz,
                     uint16_t* y, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    const int NT = N / 16;
    dim3 grid((NT + NPW - 1) / NPW);
    // activations staged in LDS when all of x fits (one padded slice per wave)
    const size_t xbytes = (size_t)WAVES * stream_slice_bytes(M, K / 128, WAVES);
    // (only single-block tiles stage x: no staged instantiation for MT > 1)
    if constexpr (MT == 1) {
        constexpr int D = NPW == 1 ? 8 : 4;
        auto* kern = &stream_kernel<MT, NPW, WAVES, D, true>;
        // more than the default dynamic LDS needs the kernel's limit raised
        if (xbytes <= kDefaultLds ||
            (xbytes <= kStreamLdsX && lds_limit_set(reinterpret_cast<const void*>(kern), kStreamLdsX))) {
            hipLaunchKernelGGL(kern, grid, dim3(64 * WAVES), xbytes, st, x, pw, ps, pz, y, M, N, K, epi);
            return;
        }
    }
    constexpr int D = MT == 1 ? (NPW == 1 ? 8 : 4) : 2;
    hipLaunchKernelGGL((stream_kernel<MT, NPW, WAVES, D, false>), grid, dim3(64 * WAVES), 0, st, x, pw, ps,
                       pz, y, M, N, K, epi);
}

template <int MT, int NPW>
int launch_stream_w(int waves, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                    const uint32_t* pz, uint16_t* y, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    switch (waves) {
    case 1: launch_stream_t<MT, NPW, 1>(x, pw, ps, pz, y, M, N, K, st, epi); break;
    case 2: launch_stream_t<MT, NPW, 2>(x, pw, ps, pz, y, M, N, K, st, epi); break;
    case 4: launch_stream_t<MT, NPW, 4>(x, pw, ps, pz, y, M, N, K, st, epi); break;
    case 8: launch_stream_t<MT, NPW, 8>(x, pw, ps, pz, y, M, N, K, st, epi); break;
    default: return QUICK_ERR_INVALID_ARG;
    }
    return QUICK_OK;
}

template <int MT>
int launch_stream_n(int npw, int waves, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                    const uint32_t* pz, uint16_t* y, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    if (npw == 1) return launch_stream_w<MT, 1>(waves, x, pw, ps, pz, y, M, N, K, st, epi);
    if (npw == 2) return launch_stream_w<MT, 2>(waves, x, pw, ps, pz, y, M, N, K, st, epi);
    return QUICK_ERR_INVALID_ARG;
}

int launch_stream(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                  const uint32_t* pz, uint16_t* y, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    const int mt = (M + 15) / 16;
    switch (mt) {
    case 1: return launch_stream_n<1>(pl.wn, pl.split, x, pw, ps, pz, y, M, N, K, st, epi);
    case 2: return launch_stream_n<2>(pl.wn, pl.split, x, pw, ps, pz, y, M, N, K, st, epi);
    case 3: return launch_stream_n<3>(pl.wn, pl.split, x, pw, ps, pz, y, M, N, K, st, epi);
    case 4: return launch_stream_n<4>(pl.wn, pl.split, x, pw, ps, pz, y, M, N, K, st, epi);
    default: return QUICK_ERR_INVALID_ARG;
    }
}

int launch_kstream(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz,
                   uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    const int ncg = ks_groups(N, pl.wn);
    const int64_t G = (int64_t)ncg * pl.split;
    // partial slots addressed with 32-bit offsets
    if (pl.split > 1 && (size_t)G * kKsWaves * pl.wn * 1024 >= ((size_t)1 << 32)) return QUICK_ERR_SHAPE;
    // the slice: M rows x kgps k-groups of 256 bytes, whole KiB (<= 64 KiB)
    const size_t lds = (size_t)ceil_div((int64_t)M * pl.kgps, 4) * 1024;
    if (lds > kKsLds) return QUICK_ERR_INVALID_ARG;
    if (!lds_limit_set(pl.wn == 1 ? reinterpret_cast<const void*>(&kstream_kernel<1>)
                                  : reinterpret_cast<const void*>(&kstream_kernel<2>),
                       kKsLds))
        return QUICK_ERR_HIP;
    const dim3 grid((unsigned)((G + 7) / 8 * 8));
    if (pl.wn == 1)
        hipLaunchKernelGGL((kstream_kernel<1>), grid, dim3(64 * kKsWaves), lds, st, x, pw, ps, pz, y, ws, M, N, K,
                           pl.kgps, ncg, pl.split, epi);
    else
        hipLaunchKernelGGL((kstream_kernel<2>), grid, dim3(64 * kKsWaves), lds, st, x, pw, ps, pz, y, ws, M, N, K,
                           pl.kgps, ncg, pl.split, epi);
    return QUICK_OK;
}
#endif  // QUICK_STREAM

#if QUICK_TILED
// nm: m-tiles of the tile space (grouped: the host's upper bound, the
// kernel derives the actual count from the expert offsets)
template <int BM, int WN, bool GRP, bool EP>
void launch_tiled_e(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                    const uint32_t* pz, uint16_t* y, float* ws, int M, int N, int K, hipStream_t st,
                    const GroupArgs& ga, const Epi& epi)
{
    const int nm = GRP ? (int)(((int64_t)ga.routed + (int64_t)ga.experts * (BM - 1)) / BM) : ceil_div(M, BM);
    const int nn = ceil_div(N, kTiledWaves * WN);
    if (pl.variant == kVariantStreamK) {
        hipLaunchKernelGGL((tiled_kernel<BM, WN, 0, GRP, EP>), dim3(pl.split), dim3(64 * kTiledWaves), 0, st, x,
                           pw, ps, pz, y, ws, M, N, K, 0, nm, nn, 0, ga, epi);
        return;
    }
    const int nblk = nm * nn * pl.split;
    const int grid = ceil_div(nblk, 8) * 8;
    hipLaunchKernelGGL((tiled_kernel<BM, WN, 0, GRP, EP>), dim3(grid), dim3(64 * kTiledWaves), 0, st, x, pw, ps,
                       pz, y, ws, M, N, K, pl.kgps, nm, nn, pl.split, ga, epi);
}

// A split-K launch writes raw partial sums and its reduction pass applies
// the epilogue, so only unsplit launches need the epilogue build.
template <int BM, int WN, bool GRP>
void launch_tiled_t(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                    const uint32_t* pz, uint16_t* y, float* ws, int M, int N, int K, hipStream_t st,
                    const GroupArgs& ga, const Epi& epi)
{
    const bool split = pl.variant == kVariantTiled && pl.split > 1;
    if ((epi.bias || epi.act) && !split)
        launch_tiled_e<BM, WN, GRP, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, ga, epi);
    else
        launch_tiled_e<BM, WN, GRP, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, ga, epi);
}

// Tile shapes of the grouped form.
// ga == nullptr: the plain GEMM; otherwise the grouped form (M = token rows).
int launch_tiled(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps,
                 const uint32_t* pz, uint16_t* y, float* ws, int M, int N, int K, hipStream_t st,
                 const Epi& epi, const GroupArgs* ga)
{
    if (ga) {
        if (pl.bm == 16 && pl.wn == 16) launch_tiled_t<16, 16, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else if (pl.bm == 16 && pl.wn == 32) launch_tiled_t<16, 32, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else if (pl.bm == 32 && pl.wn == 32) launch_tiled_t<32, 32, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else if (pl.bm == 32 && pl.wn == 16) launch_tiled_t<32, 16, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else if (pl.bm == 64 && pl.wn == 32) launch_tiled_t<64, 32, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else if (pl.bm == 128 && pl.wn == 32)
            launch_tiled_t<128, 32, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, *ga, epi);
        else return QUICK_ERR_INVALID_ARG;
    } else {
        const GroupArgs none{nullptr, nullptr, 0, 0};
        if (pl.bm == 16 && pl.wn == 32) launch_tiled_t<16, 32, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 32 && pl.wn == 32) launch_tiled_t<32, 32, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 16 && pl.wn == 16) launch_tiled_t<16, 16, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 32 && pl.wn == 16) launch_tiled_t<32, 16, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 64 && pl.wn == 32) launch_tiled_t<64, 32, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 64 && pl.wn == 16) launch_tiled_t<64, 16, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 128 && pl.wn == 16)
            launch_tiled_t<128, 16, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else if (pl.bm == 128 && pl.wn == 32)
            launch_tiled_t<128, 32, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, none, epi);
        else return QUICK_ERR_INVALID_ARG;
    }
    if (pl.variant == kVariantTiled && pl.split > 1) {
        const int64_t rows = ga ? ga->routed : M;
        const int64_t quads = rows * (epi.act ? N / 2 : N) / 4;
        hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, st,
                           ws + kSkCounterBytes / sizeof(float), y, rows, N, pl.split, epi);
    }
    return QUICK_OK;
}

template <int BM, int WN, bool EP>
void launch_tiled32_e(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz,
                      uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    const int nm = ceil_div(M, BM);
    const int nn = ceil_div(N, kTiledWaves * WN);
    if (pl.variant == kVariantStreamK32) {
        hipLaunchKernelGGL((tiled32_kernel<BM, WN, EP>), dim3(pl.split), dim3(64 * kTiledWaves), 0, st, x, pw, ps,
                           pz, y, ws, M, N, K, 0, nm, nn, 0, epi);
        return;
    }
    const int grid = ceil_div((int64_t)nm * nn * pl.split, 8) * 8;
    hipLaunchKernelGGL((tiled32_kernel<BM, WN, EP>), dim3(grid), dim3(64 * kTiledWaves), 0, st, x, pw, ps, pz, y,
                       ws, M, N, K, pl.kgps, nm, nn, pl.split, epi);
}

template <int BM, int WN>
void launch_tiled32_t(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz,
                      uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    const bool split = pl.variant == kVariantTiled32 && pl.split > 1;
    if ((epi.bias || epi.act) && !split) launch_tiled32_e<BM, WN, true>(pl, x, pw, ps, pz, y, ws, M, N, K, st, epi);
    else launch_tiled32_e<BM, WN, false>(pl, x, pw, ps, pz, y, ws, M, N, K, st, epi);
}

int launch_tiled32(const Plan& pl, const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz,
                   uint16_t* y, float* ws, int M, int N, int K, hipStream_t st, const Epi& epi)
{
    if (pl.bm == 32 && pl.wn == 32) launch_tiled32_t<32, 32>(pl, x, pw, ps, pz, y, ws, M, N, K, st, epi);
    else if (pl.bm == 64 && pl.wn == 32) launch_tiled32_t<64, 32>(pl, x, pw, ps, pz, y, ws, M, N, K, st, epi);
    else if (pl.bm == 128 && pl.wn == 32) launch_tiled32_t<128, 32>(pl, x, pw, ps, pz, y, ws, M, N, K, st, epi);
    else return QUICK_ERR_INVALID_ARG;
    if (pl.variant == kVariantTiled32 && pl.split > 1) {
        const int64_t quads = (int64_t)M * (epi.act ? N / 2 : N) / 4;
        hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((quads + 255) / 256)), dim3(256), 0, st,
                           ws + kSkCounterBytes / sizeof(float), y, (int64_t)M, N, pl.split, epi);
    }
    return QUICK_OK;
}

int launch_ablation(const uint16_t* x, const u4_t* pw, const uint16_t* ps, const uint32_t* pz, uint16_t* y,
                    int M, int N, int K, int mode, hipStream_t st)
{
    const int nm = ceil_div(M, 64), nn = ceil_div(N, kTiledWaves * 32);
    const int grid = ceil_div((int64_t)nm * nn, 8) * 8;
    const int KG = K / 128;
    auto args = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * kTiledWaves), 0, st, x, pw, ps, pz, y, (float*)nullptr,
                           M, N, K, KG, nm, nn, 1, GroupArgs{nullptr, nullptr, 0, 0}, Epi{nullptr, 0});
    };
    if (mode == 0) args(tiled_kernel<64, 32, 0>);
    else if (mode == 1) args(tiled_kernel<64, 32, 1>);
    else if (mode == 2) args(tiled_kernel<64, 32, 2>);
    else return QUICK_ERR_INVALID_ARG;
    return QUICK_OK;
}

#endif  // QUICK_TILED

}  // namespace quick

#if QUICK_HOST
namespace {

using quick::launch_ablation;
using quick::launch_kstream;
using quick::launch_stream;
using quick::launch_tiled;
using quick::launch_tiled32;

bool grouped_tile_supported(int bm, int wn)
{
    return ((bm == 16 || bm == 32) && (wn == 16 || wn == 32)) || (bm == 64 && wn == 32) || (bm == 128 && wn == 32);
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

int validate(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
             int64_t M, int64_t N, int64_t K, int64_t group)
{
    if (group != quick::kGroup) return QUICK_ERR_UNSUPPORTED;
    if (M < 0 || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return QUICK_ERR_SHAPE;
    // 32-bit buffer offsets and index arithmetic inside the kernels: packed
    // weights (K*N/2 bytes) and activations (2*M*K bytes) below 4 GiB, the
    // output below 2^31 elements.
    if (K * N / 2 >= ((int64_t)1 << 32) || M * K >= ((int64_t)1 << 31) || M * N >= ((int64_t)1 << 31) ||
        M > (1 << 24))
        return QUICK_ERR_SHAPE;
    if (M == 0) return QUICK_OK;
    if (!x || !packed || !scales || !zeros || !y) return QUICK_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(packed, 16) || !aligned(scales, 2) || !aligned(zeros, 4) ||
        !aligned(y, 8))
        return QUICK_ERR_ALIGNMENT;
    return QUICK_OK;
}

// The epilogue's constraints on a plan.  The gated form needs each gate
// tile and its up tile in one wave (stream kernel: 2 n-tiles per wave;
// tiled kernel: an even number of 16-column tiles per wave) unless a split-K
// reduction pass applies it.  Choices left automatic are adjusted; an
// explicit one that conflicts (a tile_n the caller set) is an error.
int epilogue_plan(const Epi& epi, const quick_config_t* cfg, Plan* pl)
{
    if (!epi.act) return QUICK_OK;
    const bool fixed_n = cfg && cfg->tile_n;
    if ((pl->variant == kVariantStream || pl->variant == kVariantKStream) && pl->wn != 2) {
        if (fixed_n) return QUICK_ERR_INVALID_ARG;
        pl->wn = 2;
    }
    if (is_tiled(pl->variant) && pl->wn == 16 && !(pl->variant == kVariantTiled && pl->split > 1)) {
        if (fixed_n || pl->bm > 32) return QUICK_ERR_INVALID_ARG;
        pl->wn = 32;
    }
    return QUICK_OK;
}

int gemm_impl(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
              int64_t M, int64_t N, int64_t K, int64_t group, void* stream, const quick_config_t* cfg,
              void* workspace, size_t workspace_bytes, const Epi& epi = Epi{nullptr, 0})
{
    int st = validate(x, packed, scales, zeros, y, M, N, K, group);
    if (st) return st;
    if (epi.act < 0 || epi.act > 1) return QUICK_ERR_INVALID_ARG;
    if (epi.act && N % 32 != 0) return QUICK_ERR_SHAPE;
    if (M && epi.bias && !aligned(epi.bias, 8)) return QUICK_ERR_ALIGNMENT;
    Plan pl;
    st = make_plan(M, N, K, cfg, &pl);
    if (st) return st;
    st = epilogue_plan(epi, cfg, &pl);
    if (st) return st;
    if (M == 0) return QUICK_OK;
    finish_plan(M, N, K, &pl);
    hipStream_t hs = (hipStream_t)stream;
    const size_t need = plan_workspace(M, N, pl);
    void* ws = nullptr;
    if (need) {
        if (workspace) {
            if (workspace_bytes < need) return QUICK_ERR_WORKSPACE;
            if (!aligned(workspace, 16)) return QUICK_ERR_ALIGNMENT;
            ws = workspace;
        } else {
            st = get_workspace(need, hs, &ws);
            if (st) return st;
        }
    }
    const uint16_t* xx = static_cast<const uint16_t*>(x);
    const u4_t* pw = static_cast<const u4_t*>(packed);
    const uint16_t* ps = static_cast<const uint16_t*>(scales);
    const uint32_t* pz = static_cast<const uint32_t*>(zeros);
    uint16_t* yy = static_cast<uint16_t*>(y);
    (void)hipGetLastError();  // clear a stale error so the check below is ours
    if (pl.variant == kVariantStream)
        st = launch_stream(pl, xx, pw, ps, pz, yy, (int)M, (int)N, (int)K, hs, epi);
    else if (pl.variant == kVariantKStream)
        st = launch_kstream(pl, xx, pw, ps, pz, yy, static_cast<float*>(ws), (int)M, (int)N, (int)K, hs, epi);
    else if (is_t32(pl.variant))
        st = launch_tiled32(pl, xx, pw, ps, pz, yy, static_cast<float*>(ws), (int)M, (int)N, (int)K, hs, epi);
    else
        st = launch_tiled(pl, xx, pw, ps, pz, yy, static_cast<float*>(ws), (int)M, (int)N, (int)K, hs, epi);
    if (st) return st;
    if (hipGetLastError() != hipSuccess) return QUICK_ERR_HIP;
    return QUICK_OK;
}

}  // namespace

extern "C" int quick_w4a16_gemm(const void* x, const void* packed, const void* scales,
                                const void* zeros, void* y, int64_t M, int64_t N, int64_t K,
                                int64_t group, void* stream)
{
    return gemm_impl(x, packed, scales, zeros, y, M, N, K, group, stream, nullptr, nullptr, 0);
}

extern "C" int quick_w4a16_gemm_ex(const void* x, const void* packed, const void* scales,
                                   const void* zeros, void* y, int64_t M, int64_t N, int64_t K,
                                   int64_t group, void* stream, const quick_config_t* cfg,
                                   void* workspace, size_t workspace_bytes)
{
    return gemm_impl(x, packed, scales, zeros, y, M, N, K, group, stream, cfg, workspace,
                     workspace_bytes);
}

// ---------------------------------------------------------------------------
// Allocation-free entry point (declared in quick.h): the workspace is this
// file-scope device array, QUICK_SCRATCH_BYTES on every GPU the library runs
// on, held until the process ends.  In host code its name only stands in
// for the symbol: its device address comes from hipGetSymbolAddress, once per
// device, with that device current.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[QUICK_SCRATCH_BYTES];

namespace {

__global__ void __launch_bounds__(256) scratch_clear_kernel(uint32_t* p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch;  // device -> address of its copy of `scratch`

// This device's scratch address; the first call on a device looks it up and
// clears the arrival counters at its start with a kernel on `stream` (a
// kernel rather than a memset node, so a capturing caller may take it into
// its graph).  Every GEMM leaves the counters zero again.
int scratch_address(hipStream_t stream, void** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return QUICK_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    const auto it = g_scratch.find(dev);
    if (it != g_scratch.end()) {
        *out = it->second;
        return QUICK_OK;
    }
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
        (void)hipGetLastError();
        return QUICK_ERR_HIP;
    }
    const int n = (int)(kSkCounterBytes / sizeof(uint32_t));
    (void)hipGetLastError();
    hipLaunchKernelGGL(scratch_clear_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, static_cast<uint32_t*>(p),
                       n);
    if (hipGetLastError() != hipSuccess) return QUICK_ERR_HIP;
    g_scratch[dev] = p;
    *out = p;
    return QUICK_OK;
}

}  // namespace

extern "C" int quick_w4a16_gemm_noalloc(const void* x, const void* packed, const void* scales, const void* zeros,
                                        void* y, int64_t M, int64_t N, int64_t K, int64_t group, void* stream)
{
    // argument errors are reported before any set-up
    int st = validate(x, packed, scales, zeros, y, M, N, K, group);
    if (st || M == 0) return st;
    Plan pl;
    st = make_plan(M, N, K, nullptr, &pl);
    if (st) return st;
    finish_plan(M, N, K, &pl);
    if (plan_workspace(M, N, pl) > (size_t)QUICK_SCRATCH_BYTES) return QUICK_ERR_WORKSPACE;
    void* ws = nullptr;
    st = scratch_address((hipStream_t)stream, &ws);
    if (st) return st;
    return gemm_impl(x, packed, scales, zeros, y, M, N, K, group, stream, nullptr, ws, (size_t)QUICK_SCRATCH_BYTES);
}

extern "C" size_t quick_workspace_bytes(int64_t M, int64_t N, int64_t K, const quick_config_t* cfg)
{
    if (M <= 0 || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return 0;
    Plan pl;
    if (make_plan(M, N, K, cfg, &pl)) return 0;
    finish_plan(M, N, K, &pl);
    return plan_workspace(M, N, pl);
}

extern "C" int quick_select_config(int64_t M, int64_t N, int64_t K, quick_config_t* cfg)
{
    if (!cfg) return QUICK_ERR_INVALID_ARG;
    if (M < 0 || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return QUICK_ERR_SHAPE;
    Plan pl;
    if (make_plan(M, N, K, nullptr, &pl) != QUICK_OK) auto_plan(M, N, K, &pl);
    finish_plan(M, N, K, &pl);
    cfg->variant = pl.variant;
    cfg->split_k = pl.split;
    cfg->tile_m = is_tiled(pl.variant) ? pl.bm : 0;
    cfg->tile_n = pl.wn;
    return QUICK_OK;
}

namespace {

// Configurations worth timing for a shape: the stream kernel (small M), the
// sliced stream kernel (M <= 16), the tiled tiles no taller than the next
// power of two >= M (at least 16) with splits 1, 2, 4, 8 (each slice keeping
// >= 2 k-groups), and stream-K.
std::vector<quick_config_t> tune_candidates(int64_t M, int64_t N, int64_t K)
{
    std::vector<quick_config_t> c;
    const int64_t KG = K / 128;
    if (M <= 64)
        for (int w : {1, 2, 4, 8})
            for (int p : {1, 2}) c.push_back(quick_config_t{kVariantStream, w, 0, p});
    if (M <= 16) {
        // sliced stream kernel: 1, 2, 4, 8 times the fewest K slices, and
        // the slice counts that give about 1, 2, 3, 4 workgroups per compute
        // unit (256 CUs)
        const int smin = ks_min_slices(K);
        for (int p : {1, 2}) {
            std::vector<int> ss;
            for (int m = 1; m <= 8; m *= 2) ss.push_back(smin * m);
            for (int r = 1; r <= 4; ++r) ss.push_back(ceil_div(256 * r, ks_groups(N, p)));
            std::sort(ss.begin(), ss.end());
            int last = 0;
            for (int s : ss) {
                if (s < smin || s > KG || s == last || (s > smin && KG / s < 2)) continue;
                // distinct slice lengths only
                if (last && ceil_div(KG, ceil_div(KG, s)) == ceil_div(KG, ceil_div(KG, last))) continue;
                c.push_back(quick_config_t{kVariantKStream, s, 0, p});
                last = s;
            }
        }
    }
    int64_t mcap = 16;
    while (mcap < M && mcap < 128) mcap *= 2;
    static const int tiles[][2] = {{16, 16}, {16, 32}, {32, 16}, {32, 32}, {64, 16}, {64, 32}, {128, 16},
                                   {128, 32}};
    for (const auto& t : tiles) {
        if (t[0] > mcap) continue;
        for (int s : {1, 2, 4, 8})
            if (s == 1 || KG / s >= 2) c.push_back(quick_config_t{kVariantTiled, s, t[0], t[1]});
        c.push_back(quick_config_t{kVariantStreamK, 0, t[0], t[1]});
        if (!tiled32_supported(t[0], t[1])) continue;
        for (int s : {1, 2, 4, 8})
            if (s == 1 || KG / s >= 2) c.push_back(quick_config_t{kVariantTiled32, s, t[0], t[1]});
        c.push_back(quick_config_t{kVariantStreamK32, 0, t[0], t[1]});
    }
    return c;
}

}  // namespace

// Timed launches of quick_tune rotate through device copies of the weights
// spanning at least this many bytes (twice the 256 MB Infinity Cache), so
// that each launch streams its weights from HBM as in a forward pass.
constexpr size_t kTuneSpan = (size_t)512 << 20;
constexpr int kTuneMaxCopies = 64;

namespace {

// Time of `reps` launches of configuration c, each on the next weight copy,
// as the best of kTrials replays of one HIP graph holding them (captured on
// the private stream ts): the host's per-launch cost stays out of the timing
// of kernels shorter than it.  QUICK_ERR_INVALID_ARG when c does not apply to
// the shape.
int tune_time(const void* x, const std::vector<const void*>& cw, const std::vector<const void*>& cs,
              const std::vector<const void*>& cz, void* y, int64_t M, int64_t N, int64_t K, int64_t group,
              hipStream_t ts, const quick_config_t& c, int reps, hipEvent_t e0, hipEvent_t e1, float* ms)
{
    constexpr int kTrials = 3;
    const int ncopy = (int)cw.size();
    // warm-up on ts: plans the launch and sizes ts's workspace outside the capture
    int st = gemm_impl(x, cw[0], cs[0], cz[0], y, M, N, K, group, ts, &c, nullptr, 0);
    if (st) return st;
    hipGraph_t g = nullptr;
    hipGraphExec_t ge = nullptr;
    if (hipStreamBeginCapture(ts, hipStreamCaptureModeThreadLocal) != hipSuccess) return QUICK_ERR_HIP;
    for (int r = 0; r < reps && !st; ++r) {
        const int i = r % ncopy;
        st = gemm_impl(x, cw[i], cs[i], cz[i], y, M, N, K, group, ts, &c, nullptr, 0);
    }
    const bool ended = hipStreamEndCapture(ts, &g) == hipSuccess;
    if (!st && (!ended || hipGraphInstantiate(&ge, g, nullptr, nullptr, 0) != hipSuccess)) st = QUICK_ERR_HIP;
    for (int t = 0; t <= kTrials && !st; ++t) {   // t == 0: a replay that is not timed
        float tm = 0.f;
        if (hipEventRecord(e0, ts) != hipSuccess || hipGraphLaunch(ge, ts) != hipSuccess ||
            hipEventRecord(e1, ts) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&tm, e0, e1) != hipSuccess) {
            st = QUICK_ERR_HIP;
            break;
        }
        if (t == 1 || (t > 1 && tm < *ms)) *ms = tm;
    }
    if (ge) (void)hipGraphExecDestroy(ge);
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();
    return st;
}

}  // namespace

extern "C" int quick_tune(const void* x, const void* packed, const void* scales, const void* zeros, void* y,
                          int64_t M, int64_t N, int64_t K, int64_t group, void* stream, quick_config_t* best)
{
    int st = validate(x, packed, scales, zeros, y, M, N, K, group);
    if (st) return st;
    if (M == 0) return QUICK_OK;
    hipStream_t hs = (hipStream_t)stream;
    hipStreamCaptureStatus cs0 = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(hs, &cs0) != hipSuccess) return QUICK_ERR_HIP;
    if (cs0 != hipStreamCaptureStatusNone) return QUICK_ERR_CAPTURE;
    // the timings run on a private stream that first waits for the caller's
    // (whose work may be producing the inputs)
    hipStream_t ts = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipStreamCreateWithFlags(&ts, hipStreamNonBlocking) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
        hipEventCreate(&e1) != hipSuccess || hipEventRecord(e0, hs) != hipSuccess ||
        hipStreamWaitEvent(ts, e0, 0) != hipSuccess) {
        (void)hipGetLastError();
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
        if (ts) (void)hipStreamDestroy(ts);
        return QUICK_ERR_HIP;
    }
    // weight copies: copy 0 is the caller's; the others live in one
    // temporary allocation (none when it cannot be had: then the timings
    // repeat the caller's buffers)
    const size_t wb = (size_t)K * N / 2, sb = wb / 32, zb = wb / 128;
    // 2 MiB-aligned like the caller's allocations, so that every copy maps
    // onto the memory channels as the original does
    auto al = [](size_t b) { return (b + ((size_t)2 << 20) - 1) / ((size_t)2 << 20) * ((size_t)2 << 20); };
    const size_t per = al(wb) + al(sb) + al(zb);
    int ncopy = (int)std::min<size_t>(kTuneMaxCopies, std::max<size_t>(1, (kTuneSpan + per - 1) / per));
    uint8_t* extra = nullptr;
    if (ncopy > 1 && hipMalloc(&extra, (size_t)(ncopy - 1) * per) != hipSuccess) {
        (void)hipGetLastError();
        extra = nullptr;
        ncopy = 1;
    }
    std::vector<const void*> cw(ncopy, packed), cs(ncopy, scales), cz(ncopy, zeros);
    for (int i = 1; i < ncopy && !st; ++i) {
        uint8_t* b = extra + (size_t)(i - 1) * per;
        cw[i] = b;
        cs[i] = b + al(wb);
        cz[i] = b + al(wb) + al(sb);
        if (hipMemcpyAsync((void*)cw[i], packed, wb, hipMemcpyDeviceToDevice, ts) != hipSuccess ||
            hipMemcpyAsync((void*)cs[i], scales, sb, hipMemcpyDeviceToDevice, ts) != hipSuccess ||
            hipMemcpyAsync((void*)cz[i], zeros, zb, hipMemcpyDeviceToDevice, ts) != hipSuccess)
            st = QUICK_ERR_HIP;
    }
    const int reps = std::max(20, ncopy);
    float best_ms = 0.f;
    quick_config_t bestc{};
    bool found = false;
    for (const quick_config_t& c : tune_candidates(M, N, K)) {
        if (st) break;
        float ms = 0.f;
        st = tune_time(x, cw, cs, cz, y, M, N, K, group, ts, c, reps, e0, e1, &ms);
        if (st == QUICK_ERR_INVALID_ARG) {  // not supported for this shape
            st = QUICK_OK;
            continue;
        }
        if (st) break;
        if (!found || ms < best_ms) {
            best_ms = ms;
            bestc = c;
            found = true;
        }
    }
    // the copies and ts's launches are done before anything is freed or y
    // is written on the caller's stream
    if (hipStreamSynchronize(ts) != hipSuccess && !st) st = QUICK_ERR_HIP;
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    (void)hipStreamDestroy(ts);
    if (extra) (void)hipFree(extra);
    (void)hipGetLastError();
    if (st) return st;
    if (!found) return QUICK_ERR_INVALID_ARG;
    {
        std::lock_guard<std::mutex> lk(g_tune_mu);
        g_tune[ShapeKey{M, N, K}] = bestc;
    }
    // leave y holding the chosen configuration's result
    st = gemm_impl(x, packed, scales, zeros, y, M, N, K, group, stream, &bestc, nullptr, 0);
    if (st) return st;
    if (best) *best = bestc;
    return QUICK_OK;
}

extern "C" int quick_tune_table_save(const char* path)
{
    if (!path) return QUICK_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(g_tune_mu);
    FILE* f = std::fopen(path, "w");
    if (!f) return QUICK_ERR_IO;
    bool ok = std::fprintf(f, "quick-tune 1\n") > 0;
    for (const auto& e : g_tune)
        ok = ok && std::fprintf(f, "%lld %lld %lld %d %d %d %d\n", (long long)e.first.M, (long long)e.first.N,
                                (long long)e.first.K, e.second.variant, e.second.split_k, e.second.tile_m,
                                e.second.tile_n) > 0;
    ok = (std::fclose(f) == 0) && ok;
    return ok ? QUICK_OK : QUICK_ERR_IO;
}

extern "C" int quick_tune_table_load(const char* path)
{
    if (!path) return QUICK_ERR_INVALID_ARG;
    FILE* f = std::fopen(path, "r");
    if (!f) return QUICK_ERR_IO;
    char line[256];
    bool ok = std::fgets(line, sizeof line, f) && std::strncmp(line, "quick-tune 1", 12) == 0;
    std::vector<std::pair<ShapeKey, quick_config_t>> rows;
    while (ok && std::fgets(line, sizeof line, f)) {
        long long m, n, k;
        quick_config_t c{};
        char extra;
        const int got = std::sscanf(line, "%lld %lld %lld %d %d %d %d %c", &m, &n, &k, &c.variant, &c.split_k,
                                    &c.tile_m, &c.tile_n, &extra);
        if (got != 7 || m <= 0 || n <= 0 || k <= 0 || k % 128 != 0 || n % 16 != 0) {
            ok = false;
            break;
        }
        Plan pl;
        if (make_plan(m, n, k, &c, &pl) != QUICK_OK) {
            ok = false;
            break;
        }
        rows.push_back({ShapeKey{m, n, k}, c});
    }
    std::fclose(f);
    if (!ok) return QUICK_ERR_IO;
    std::lock_guard<std::mutex> lk(g_tune_mu);
    for (const auto& r : rows) g_tune[r.first] = r.second;
    return QUICK_OK;
}

extern "C" int quick_tune_table_size(void)
{
    std::lock_guard<std::mutex> lk(g_tune_mu);
    return (int)g_tune.size();
}

extern "C" void quick_tune_table_clear(void)
{
    std::lock_guard<std::mutex> lk(g_tune_mu);
    g_tune.clear();
}

// Ablation of the method's central choice (declared in quick_ablation.h): the
// 64 x 256 data-parallel tiled kernel with the dequantized weights going
// straight to the matrix-instruction registers (mode 0, the method) or
// through an LDS tile and back (mode 1 padded rows, mode 2 unpadded rows).
extern "C" int quick_ablation_gemm(const void* x, const void* packed, const void* scales, const void* zeros,
                                   void* y, int64_t M, int64_t N, int64_t K, int mode, void* stream)
{
    int st = validate(x, packed, scales, zeros, y, M, N, K, 128);
    if (st) return st;
    if (mode < 0 || mode > 2) return QUICK_ERR_INVALID_ARG;
    if (M == 0) return QUICK_OK;
    (void)hipGetLastError();
    st = launch_ablation(static_cast<const uint16_t*>(x), static_cast<const u4_t*>(packed),
                         static_cast<const uint16_t*>(scales), static_cast<const uint32_t*>(zeros),
                         static_cast<uint16_t*>(y), (int)M, (int)N, (int)K, mode, (hipStream_t)stream);
    if (st) return st;
    return hipGetLastError() == hipSuccess ? QUICK_OK : QUICK_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Grouped (mixture-of-experts) GEMM: declared in quick_grouped.h.
// ---------------------------------------------------------------------------
namespace {

int validate_grouped(const void* x, const int32_t* rows, const int32_t* offsets, const void* packed,
                     const void* scales, const void* zeros, void* y, int64_t T, int64_t R, int64_t E, int64_t N,
                     int64_t K, int64_t group)
{
    if (group != quick::kGroup) return QUICK_ERR_UNSUPPORTED;
    if (T < 0 || R < 0 || E < 1 || E > kMaxExperts || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0)
        return QUICK_ERR_SHAPE;
    // 32-bit offsets inside the kernel, as for the plain GEMM (per expert)
    if (K * N / 2 >= ((int64_t)1 << 32) || T * K >= ((int64_t)1 << 31) || R * N >= ((int64_t)1 << 31) ||
        R > (1 << 24) || T > (1 << 24))
        return QUICK_ERR_SHAPE;
    if (R == 0) return QUICK_OK;
    if (T == 0 || (!rows && T < R)) return QUICK_ERR_SHAPE;
    if (!x || !offsets || !packed || !scales || !zeros || !y) return QUICK_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(packed, 16) || !aligned(scales, 2) || !aligned(zeros, 4) || !aligned(y, 8) ||
        !aligned(offsets, 4) || (rows && !aligned(rows, 4)))
        return QUICK_ERR_ALIGNMENT;
    return QUICK_OK;
}

// Tile and schedule for R routed rows over E experts.  Rows per expert are
// known only on the device, so the tile is chosen for the mean (R / E) and
// the default schedule is stream-K, which spreads whatever tile count the
// kernel finds evenly over the resident workgroups.
int grouped_plan(int64_t R, int64_t E, int64_t N, int64_t K, const quick_config_t* cfg, Plan* pl)
{
    (void)N;
    const int64_t KG = K / 128;
    const int64_t avg = std::max<int64_t>(1, (R + E - 1) / E);
    pl->variant = kVariantStreamK;
    pl->split = 0;
    pl->kgps = 0;
    if (avg <= 16) {
        pl->bm = 16;
        pl->wn = 16;
    } else if (avg <= 32) {
        pl->bm = 32;
        pl->wn = 16;
    } else if (avg <= 96) {
        pl->bm = 64;
        pl->wn = 32;
    } else {
        pl->bm = 128;
        pl->wn = 32;
    }
    if (cfg) {
        if (cfg->variant < 0 || cfg->variant == kVariantStream || cfg->variant > 3 || cfg->split_k < 0)
            return QUICK_ERR_INVALID_ARG;
        if (cfg->variant == kVariantTiled) {
            if (cfg->split_k > KG) return QUICK_ERR_INVALID_ARG;
            pl->variant = kVariantTiled;
            pl->split = cfg->split_k ? cfg->split_k : 1;
        } else if (cfg->split_k) {
            if (cfg->split_k % 8 != 0 || cfg->split_k > kSkMaxWorkgroups) return QUICK_ERR_INVALID_ARG;
            pl->split = cfg->split_k;
        }
        if (cfg->tile_m) pl->bm = cfg->tile_m;
        if (cfg->tile_n) pl->wn = cfg->tile_n;
        if (!grouped_tile_supported(pl->bm, pl->wn)) return QUICK_ERR_INVALID_ARG;
    }
    if (pl->variant == kVariantStreamK) {
        const int g = pl->split ? pl->split : tiled_resident(pl->bm, pl->wn);
        pl->split = std::max(8, std::min(g, kSkMaxWorkgroups) / 8 * 8);
    } else {
        pl->kgps = ceil_div(KG, pl->split);
        pl->split = ceil_div(KG, pl->kgps);  // no empty splits
    }
    return QUICK_OK;
}

size_t grouped_workspace(int64_t R, int64_t N, const Plan& pl)
{
    if (pl.variant == kVariantTiled && pl.split > 1)
        return kSkCounterBytes + (size_t)pl.split * R * N * sizeof(float);
    if (pl.variant == kVariantStreamK) return kSkCounterBytes + 2 * (size_t)pl.split * sk_slot_bytes(pl.bm, pl.wn);
    return 0;
}

// The automatic grouped plan with full-height (128-row) tiles runs in two
// launches: the experts' whole tiles (and remainders of at least 64 rows)
// with the 128-row tiles, then the short remainders with 32-row tiles, so a
// remainder of a few rows does not cost a full-height tile's matrix work.
// Returns whether `pl` is split that way, and the second launch's plan.
constexpr int kGroupTileUnit = 128;
constexpr int kGroupTailKeep = 64;
bool grouped_tail_plan(int64_t R, int64_t E, int64_t N, int64_t K, const quick_config_t* cfg, const Plan& pl,
                       Plan* tp)
{
    const bool automatic = !cfg || (cfg->variant == 0 && cfg->split_k == 0 && cfg->tile_m == 0 && cfg->tile_n == 0);
    if (!automatic || pl.bm != kGroupTileUnit) return false;
    const quick_config_t tc{kVariantStreamK, 0, 32, 32};
    return grouped_plan(R, E, N, K, &tc, tp) == QUICK_OK;
}

// The epilogue's constraints on a grouped plan (see epilogue_plan).
int grouped_epilogue_plan(const Epi& epi, const quick_config_t* cfg, Plan* pl)
{
    // a per-expert bias is added in the tile epilogue; the split-K reduction
    // pass does not know a row's expert
    if (epi.bias && pl->variant == kVariantTiled && pl->split > 1) return QUICK_ERR_INVALID_ARG;
    if (epi.act && pl->wn == 16 && !(pl->variant == kVariantTiled && pl->split > 1)) {
        // 16-column waves cannot pair a gate tile with its up tile
        if (cfg && cfg->tile_n) return QUICK_ERR_INVALID_ARG;
        pl->wn = 32;
    }
    return QUICK_OK;
}

int grouped_impl(const void* x, const int32_t* rows, const int32_t* offsets, const void* packed,
                 const void* scales, const void* zeros, void* y, int64_t T, int64_t R, int64_t E, int64_t N,
                 int64_t K, int64_t group, void* stream, const quick_config_t* cfg, void* workspace,
                 size_t workspace_bytes, const Epi& epi = Epi{nullptr, 0})
{
    int st = validate_grouped(x, rows, offsets, packed, scales, zeros, y, T, R, E, N, K, group);
    if (st) return st;
    if (epi.act < 0 || epi.act > 1) return QUICK_ERR_INVALID_ARG;
    if (epi.act && N % 32 != 0) return QUICK_ERR_SHAPE;
    if (R && epi.bias && !aligned(epi.bias, 8)) return QUICK_ERR_ALIGNMENT;
    Plan pl;
    st = grouped_plan(R, E, N, K, cfg, &pl);
    if (st) return st;
    st = grouped_epilogue_plan(epi, cfg, &pl);
    if (st) return st;
    Plan tp;
    const bool tail = grouped_tail_plan(R, E, N, K, cfg, pl, &tp);
    if (R == 0) return QUICK_OK;
    hipStream_t hs = (hipStream_t)stream;
    const size_t need = std::max(grouped_workspace(R, N, pl), tail ? grouped_workspace(R, N, tp) : 0);
    void* ws = nullptr;
    if (need) {
        if (workspace) {
            if (workspace_bytes < need) return QUICK_ERR_WORKSPACE;
            if (!aligned(workspace, 16)) return QUICK_ERR_ALIGNMENT;
            ws = workspace;
        } else {
            st = get_workspace(need, hs, &ws);
            if (st) return st;
        }
    }
    (void)hipGetLastError();
    // the two launches write disjoint rows of y; the second reuses the
    // workspace after the first (same stream; stream-K leaves its counters
    // zero)
    for (int part = tail ? 1 : 0; part <= (tail ? 2 : 0); ++part) {
        const GroupArgs ga{rows, offsets, (int)E, (int)R, part, kGroupTileUnit, kGroupTailKeep};
        st = launch_tiled(part == 2 ? tp : pl, static_cast<const uint16_t*>(x), static_cast<const u4_t*>(packed),
                          static_cast<const uint16_t*>(scales), static_cast<const uint32_t*>(zeros),
                          static_cast<uint16_t*>(y), static_cast<float*>(ws), (int)T, (int)N, (int)K, hs, epi, &ga);
        if (st) return st;
    }
    return hipGetLastError() == hipSuccess ? QUICK_OK : QUICK_ERR_HIP;
}

}  // namespace

extern "C" int quick_w4a16_grouped_gemm(const void* x, const int32_t* rows, const int32_t* offsets,
                                        const void* packed, const void* scales, const void* zeros, void* y,
                                        int64_t T, int64_t R, int64_t E, int64_t N, int64_t K, int64_t group,
                                        void* stream)
{
    return grouped_impl(x, rows, offsets, packed, scales, zeros, y, T, R, E, N, K, group, stream, nullptr,
                        nullptr, 0);
}

extern "C" int quick_w4a16_grouped_gemm_ex(const void* x, const int32_t* rows, const int32_t* offsets,
                                           const void* packed, const void* scales, const void* zeros, void* y,
                                           int64_t T, int64_t R, int64_t E, int64_t N, int64_t K, int64_t group,
                                           void* stream, const quick_config_t* cfg, void* workspace,
                                           size_t workspace_bytes)
{
    return grouped_impl(x, rows, offsets, packed, scales, zeros, y, T, R, E, N, K, group, stream, cfg, workspace,
                        workspace_bytes);
}

extern "C" size_t quick_grouped_workspace_bytes(int64_t R, int64_t E, int64_t N, int64_t K,
                                                const quick_config_t* cfg)
{
    if (R <= 0 || E < 1 || E > kMaxExperts || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return 0;
    Plan pl, tp;
    if (grouped_plan(R, E, N, K, cfg, &pl)) return 0;
    const bool tail = grouped_tail_plan(R, E, N, K, cfg, pl, &tp);
    return std::max(grouped_workspace(R, N, pl), tail ? grouped_workspace(R, N, tp) : 0);
}

extern "C" int quick_grouped_select_config(int64_t R, int64_t E, int64_t N, int64_t K, quick_config_t* cfg)
{
    if (!cfg) return QUICK_ERR_INVALID_ARG;
    if (R < 0 || E < 1 || E > kMaxExperts || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0)
        return QUICK_ERR_SHAPE;
    Plan pl;
    const int st = grouped_plan(R, E, N, K, nullptr, &pl);
    if (st) return st;
    cfg->variant = pl.variant;
    cfg->split_k = pl.split;
    cfg->tile_m = pl.bm;
    cfg->tile_n = pl.wn;
    return QUICK_OK;
}

// ---------------------------------------------------------------------------
// Fused epilogues: declared in quick_fused.h.
// ---------------------------------------------------------------------------
namespace {

Epi to_epi(const quick_epilogue_t* e)
{
    return e ? Epi{static_cast<const uint16_t*>(e->bias), e->activation} : Epi{nullptr, 0};
}

}  // namespace

extern "C" int quick_w4a16_gemm_fused(const void* x, const void* packed, const void* scales, const void* zeros,
                                      void* y, int64_t M, int64_t N, int64_t K, int64_t group, void* stream,
                                      const quick_epilogue_t* epi, const quick_config_t* cfg, void* workspace,
                                      size_t workspace_bytes)
{
    return gemm_impl(x, packed, scales, zeros, y, M, N, K, group, stream, cfg, workspace, workspace_bytes,
                     to_epi(epi));
}

extern "C" int quick_w4a16_grouped_gemm_fused(const void* x, const int32_t* rows, const int32_t* offsets,
                                              const void* packed, const void* scales, const void* zeros, void* y,
                                              int64_t T, int64_t R, int64_t E, int64_t N, int64_t K,
                                              int64_t group, void* stream, const quick_epilogue_t* epi,
                                              const quick_config_t* cfg, void* workspace, size_t workspace_bytes)
{
    return grouped_impl(x, rows, offsets, packed, scales, zeros, y, T, R, E, N, K, group, stream, cfg, workspace,
                        workspace_bytes, to_epi(epi));
}

extern "C" size_t quick_fused_workspace_bytes(int64_t M, int64_t N, int64_t K, const quick_config_t* cfg,
                                              const quick_epilogue_t* epi)
{
    if (M <= 0 || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return 0;
    Plan pl;
    if (make_plan(M, N, K, cfg, &pl)) return 0;
    if (epilogue_plan(to_epi(epi), cfg, &pl)) return 0;
    finish_plan(M, N, K, &pl);
    return plan_workspace(M, N, pl);
}

extern "C" size_t quick_grouped_fused_workspace_bytes(int64_t R, int64_t E, int64_t N, int64_t K,
                                                      const quick_config_t* cfg, const quick_epilogue_t* epi)
{
    if (R <= 0 || E < 1 || E > kMaxExperts || N <= 0 || K <= 0 || K % 128 != 0 || N % 16 != 0) return 0;
    Plan pl, tp;
    if (grouped_plan(R, E, N, K, cfg, &pl)) return 0;
    if (grouped_epilogue_plan(to_epi(epi), cfg, &pl)) return 0;
    const bool tail = grouped_tail_plan(R, E, N, K, cfg, pl, &tp);
    return std::max(grouped_workspace(R, N, pl), tail ? grouped_workspace(R, N, tp) : 0);
}

extern "C" int quick_interleave_gate_up(const uint8_t* q_gate, const uint8_t* z_gate, const uint16_t* s_gate,
                                        const uint8_t* q_up, const uint8_t* z_up, const uint16_t* s_up,
                                        int64_t K, int64_t Nh, int64_t group, uint8_t* q, uint8_t* z, uint16_t* s)
{
    if (!q_gate || !z_gate || !s_gate || !q_up || !z_up || !s_up || !q || !z || !s) return QUICK_ERR_INVALID_ARG;
    if (group != quick::kGroup) return QUICK_ERR_UNSUPPORTED;
    if (K <= 0 || Nh <= 0 || K % 128 != 0 || Nh % 16 != 0) return QUICK_ERR_SHAPE;
    const int64_t N = 2 * Nh;
    // output column 32t + i: gate column 16t + i (i < 16), up column 16t + i - 16
    auto cols = [&](const auto* gate, const auto* up, auto* out, int64_t rows) {
        for (int64_t r = 0; r < rows; ++r)
            for (int64_t t = 0; t < Nh / 16; ++t) {
                std::memcpy(out + r * N + 32 * t, gate + r * Nh + 16 * t, 16 * sizeof(*out));
                std::memcpy(out + r * N + 32 * t + 16, up + r * Nh + 16 * t, 16 * sizeof(*out));
            }
    };
    cols(q_gate, q_up, q, K);
    cols(z_gate, z_up, z, K / group);
    cols(s_gate, s_up, s, K / group);
    return QUICK_OK;
}

#endif  // QUICK_HOST
