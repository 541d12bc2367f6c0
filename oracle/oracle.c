/*
 * oracle.c -- CPU reference for the W4A16 mixed-precision GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no source with the HIP library.
 *
 * What it computes (paper, Section 2.1 and Section 2.3): with weight-only
 * quantization the weights are stored as small unsigned integers q together
 * with a zero point z and a scale s per group, and they are dequantized to
 * W = (q - z) * s before being multiplied by the half-precision activations
 * x.  The GEMM is y = x . W.  Here the group is `group` consecutive input
 * channels (rows k of W) of one output column n, so
 *
 *     W[k][n]     = (q[k][n] - z[k/group][n]) * s[k/group][n]
 *     y[m][n]     = sum_{k=0}^{K-1} x[m][k] * W[k][n]
 *
 * evaluated in IEEE binary64 with a plain loop over k in ascending order and
 * no final rounding.  (q - z) is an integer in [-15, 15] and s is a binary16
 * value, so W is exact in binary64.
 *
 * The offline weight reorder (paper, Section 3.1 and Section 3.2: the static
 * weights are rearranged once so that a direct load from memory already has
 * the register pattern the matrix instruction needs, and the nibbles are
 * ordered so that the dequantized values come out in sequence) is written
 * here as the plain definition of the packed layout, one element at a time:
 * oracle_pack_qpk16().  The layout itself is this project's own design for
 * the gfx950 16x16x32 f16 matrix instruction; the paper's figures of its
 * NVIDIA pattern are not used.
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC (no fast-math: the k loop must stay a
 * strict left-to-right sum).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* binary16 <-> binary64, written from the IEEE 754 format definition. */
/* ------------------------------------------------------------------ */

/* Value of a binary16 bit pattern: sign, 5-bit biased exponent (bias 15),
 * 10-bit fraction.  Exponent 0 is zero/subnormal (f * 2^-24), exponent 31 is
 * infinity (f == 0) or NaN. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);
    return sign ? -v : v;
}

/* Round a binary64 value to the nearest binary16 value, ties to even.
 * The representable values between 2^e and 2^(e+1) (e >= -14) are spaced
 * 2^(e-10); below 2^-14 the spacing stays 2^-24 (subnormals).  The value is
 * divided by that spacing (exact: a power of two), rounded to an integer
 * with rint() under the default round-to-nearest-even mode, and re-encoded.
 * Anything that rounds to 2^16 or more becomes infinity. */
uint16_t oracle_f64_to_f16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    if (isnan(v))
        return 0x7e00;
    double a = fabs(v);
    if (isinf(a))
        return sign | 0x7c00;
    if (a == 0.0)
        return sign;
    int e2;
    frexp(a, &e2);            /* a = m * 2^e2, m in [0.5, 1) */
    int ex = e2 - 1;          /* 2^ex <= a < 2^(ex+1) */
    if (ex < -14)
        ex = -14;
    if (ex > 15)
        return sign | 0x7c00; /* a >= 2^16: beyond every finite value */
    double r = rint(ldexp(a, 10 - ex)); /* integer in [0, 2048] */
    /* r counts units of 2^(ex-10); r == 2048 carries into the exponent. */
    long bits = ((long)(ex + 15) << 10) + ((long)r - 1024);
    if (ex == -14 && r < 1024)
        bits = (long)r;       /* subnormal */
    if (bits >= 0x7c00)
        return sign | 0x7c00;
    return (uint16_t)(sign | bits);
}

void oracle_f16_to_f64_array(const uint16_t* h, int64_t n, double* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_f16_to_f64(h[i]);
}

void oracle_f64_to_f16_array(const double* v, int64_t n, uint16_t* out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_f64_to_f16(v[i]);
}

/* ------------------------------------------------------------------ */
/* Dequantization and GEMM (Section 2.1, Section 2.3).                 */
/* ------------------------------------------------------------------ */

static int check_shape(int64_t M, int64_t N, int64_t K, int64_t group)
{
    if (M < 0 || N < 0 || K < 0 || group <= 0)
        return 2;
    if (K % group != 0)
        return 2;
    return 0;
}

/* W[k][n] = (q[k][n] - z[k/group][n]) * s[k/group][n], all of W in binary64.
 * q: [K][N] values 0..15, z: [K/group][N] values 0..15, s: [K/group][N]
 * binary16 bits.  Returns 0, or 2 for an invalid shape, 4 for a value > 15. */
int oracle_dequant_f64(const uint8_t* q, const uint8_t* z, const uint16_t* s,
                       int64_t K, int64_t N, int64_t group, double* W)
{
    if (check_shape(0, N, K, group))
        return 2;
    for (int64_t k = 0; k < K; ++k) {
        int64_t gi = k / group;
        for (int64_t n = 0; n < N; ++n) {
            int qv = q[k * N + n];
            int zv = z[gi * N + n];
            if (qv > 15 || zv > 15)
                return 4;
            W[k * N + n] = (double)(qv - zv) * oracle_f16_to_f64(s[gi * N + n]);
        }
    }
    return 0;
}

/* y[m][c] = sum_{k ascending} x[m][k] * W[k][cols[c]] for every row m and
 * every listed column (cols == NULL means all N columns, ncols == N).
 * x: [M][K] binary16 bits.  y: [M][ncols] binary64, row-major.
 * nthreads <= 0 uses the OpenMP default.  Parallel over columns only: every
 * output element is one sequential sum. */
int oracle_gemm_f64(const uint16_t* x, const uint8_t* q, const uint8_t* z,
                    const uint16_t* s, int64_t M, int64_t N, int64_t K,
                    int64_t group, const int64_t* cols, int64_t ncols,
                    double* y, int nthreads)
{
    if (check_shape(M, N, K, group))
        return 2;
    if (cols == NULL)
        ncols = N;
    for (int64_t c = 0; c < ncols; ++c) {
        int64_t n = cols ? cols[c] : c;
        if (n < 0 || n >= N)
            return 1;
    }
    for (int64_t i = 0; i < K * N; ++i)
        if (q[i] > 15)
            return 4;
    for (int64_t i = 0; i < (K / group) * N; ++i)
        if (z[i] > 15)
            return 4;
    if (M == 0 || ncols == 0)
        return 0;

    double* xd = (double*)malloc(sizeof(double) * (size_t)(M * K > 0 ? M * K : 1));
    if (!xd)
        return 1;
    for (int64_t i = 0; i < M * K; ++i)
        xd[i] = oracle_f16_to_f64(x[i]);

#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int failed = 0;
#pragma omp parallel
    {
        double* wcol = (double*)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
        if (!wcol) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t c = 0; c < ncols; ++c) {
                int64_t n = cols ? cols[c] : c;
                /* Dequantize column n of W. */
                for (int64_t k = 0; k < K; ++k) {
                    int64_t gi = k / group;
                    wcol[k] = (double)((int)q[k * N + n] - (int)z[gi * N + n]) *
                              oracle_f16_to_f64(s[gi * N + n]);
                }
                /* Dot product of every activation row with that column. */
                for (int64_t m = 0; m < M; ++m) {
                    const double* xr = xd + m * K;
                    double acc = 0.0;
                    for (int64_t k = 0; k < K; ++k)
                        acc += xr[k] * wcol[k];
                    y[m * ncols + c] = acc;
                }
            }
            free(wcol);
        }
    }
    free(xd);
    return failed ? 1 : 0;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------ */
/* Offline weight reorder, layout "QPK16" version 1 (Section 3.2).     */
/* ------------------------------------------------------------------ */
/*
 * Definition, element by element.  With KG = K/128 k-groups, an n-tile nt of
 * 16 output columns and a k-group kg of 128 input channels form one unit of
 * 64 lanes x 4 words of 32 bits (1 KiB).  For column n and input channel k:
 *
 *   nt = n / 16, c = n % 16                      column inside the tile
 *   kg = k / 128, r = k % 128
 *   j  = r / 32                                  which 32-wide k step (word)
 *   g  = (r % 32) / 8                            lane group 0..3
 *   e  = r % 8                                   element 0..7 of the lane's 8
 *   lane = 16 * g + c
 *   word = ((nt * KG + kg) * 64 + lane) * 4 + j
 *   nibble slot of e: the even elements 0,2,4,6 sit in slots 0..3 and the odd
 *   elements 1,3,5,7 in slots 4..7, i.e. slot = e/2 + 4*(e%2), bits
 *   4*slot .. 4*slot+3 of the word.
 *
 * Zero points: word (nt * KG + kg) * 2 + c/8 holds z[kg][n] in nibble c%8.
 * Scales:      half  (nt * KG + kg) * 16 + c holds s[kg][n].
 *
 * Requires group == 128, K % 128 == 0, N % 16 == 0, values <= 15.
 * Output arrays must hold K*N/8, K*N/1024 and K*N/128 elements and are fully
 * overwritten.  Returns 0, 2 (shape), 3 (group != 128) or 4 (value > 15).
 */
int oracle_pack_qpk16(const uint8_t* q, const uint8_t* z, const uint16_t* s,
                      int64_t K, int64_t N, int64_t group,
                      uint32_t* pw, uint32_t* pz, uint16_t* ps)
{
    if (group != 128)
        return 3;
    if (K < 0 || N < 0 || K % 128 != 0 || N % 16 != 0)
        return 2;
    const int64_t KG = K / 128;
    memset(pw, 0, sizeof(uint32_t) * (size_t)(K * N / 8));
    memset(pz, 0, sizeof(uint32_t) * (size_t)(K * N / 1024));
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t n = 0; n < N; ++n) {
            uint32_t v = q[k * N + n];
            if (v > 15)
                return 4;
            int64_t nt = n / 16, c = n % 16;
            int64_t kg = k / 128, r = k % 128;
            int64_t j = r / 32, g = (r % 32) / 8, e = r % 8;
            int64_t lane = 16 * g + c;
            int64_t word = ((nt * KG + kg) * 64 + lane) * 4 + j;
            int slot = (int)(e / 2 + 4 * (e % 2));
            pw[word] |= v << (4 * slot);
        }
    }
    for (int64_t kg = 0; kg < KG; ++kg) {
        for (int64_t n = 0; n < N; ++n) {
            uint32_t v = z[kg * N + n];
            if (v > 15)
                return 4;
            int64_t nt = n / 16, c = n % 16;
            pz[(nt * KG + kg) * 2 + c / 8] |= v << (4 * (c % 8));
            ps[(nt * KG + kg) * 16 + c] = s[kg * N + n];
        }
    }
    return 0;
}
