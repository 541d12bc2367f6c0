/*
 * Driver for the sanitizer test (tests/test_sanitize.py): links the host
 * packing code of the library (quick_pack.cpp) and the CPU oracle
 * (oracle/oracle.c), both built with AddressSanitizer and
 * UndefinedBehaviorSanitizer, and runs them on buffers allocated to their
 * exact documented sizes, so any read or write past a buffer, any use of
 * freed memory and any undefined arithmetic aborts the program.
 *
 * Checked along the way: the library pack equals the oracle's element-wise
 * pack byte for byte, unpack(pack) is the identity, every error path leaves
 * the outputs untouched, and the binary16 conversions round-trip all 65536
 * patterns.  Prints SANITIZE_OK and exits 0 when everything holds.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "quick.h"

/* oracle.c */
double oracle_f16_to_f64(uint16_t h);
uint16_t oracle_f64_to_f16(double v);
int oracle_dequant_f64(const uint8_t* q, const uint8_t* z, const uint16_t* s, int64_t K, int64_t N, int64_t group,
                       double* W);
int oracle_gemm_f64(const uint16_t* x, const uint8_t* q, const uint8_t* z, const uint16_t* s, int64_t M, int64_t N,
                    int64_t K, int64_t group, const int64_t* cols, int64_t ncols, double* y, int nthreads);
int oracle_pack_qpk16(const uint8_t* q, const uint8_t* z, const uint16_t* s, int64_t K, int64_t N, int64_t group,
                      uint32_t* pw, uint32_t* pz, uint16_t* ps);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void)
{
    /* xorshift64* */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}

static int failures = 0;
#define CHECK(cond, ...)                                  \
    do {                                                  \
        if (!(cond)) {                                    \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);                 \
            fprintf(stderr, "\n");                        \
            ++failures;                                   \
        }                                                 \
    } while (0)

static void check_f16(void)
{
    for (uint32_t h = 0; h < 65536; ++h) {
        const int nan = ((h >> 10) & 0x1f) == 0x1f && (h & 0x3ff);
        const uint16_t back = oracle_f64_to_f16(oracle_f16_to_f64((uint16_t)h));
        if (nan)
            CHECK(((back >> 10) & 0x1f) == 0x1f && (back & 0x3ff), "NaN %04x lost", h);
        else
            CHECK(back == h, "f16 %04x -> %04x", h, back);
    }
}

static void check_shape(int64_t K, int64_t N, int64_t M)
{
    const int64_t G = K / 128;
    uint8_t* q = malloc((size_t)(K * N));
    uint8_t* z = malloc((size_t)(G * N));
    uint16_t* s = malloc((size_t)(G * N) * 2);
    for (int64_t i = 0; i < K * N; ++i) q[i] = (uint8_t)(next_u32() & 15);
    for (int64_t i = 0; i < G * N; ++i) {
        z[i] = (uint8_t)(next_u32() & 15);
        s[i] = (uint16_t)(0x1C00 + (next_u32() % 0x0C00));   /* 0.0039 .. 0.03 */
    }
    size_t wb = 0, zb = 0, sb = 0;
    CHECK(quick_packed_sizes(K, N, 128, &wb, &zb, &sb) == QUICK_OK, "sizes");
    CHECK(wb == (size_t)(K * N / 2) && zb == (size_t)(K * N / 256) && sb == (size_t)(K * N / 64), "size formula");
    uint8_t* pw = malloc(wb);
    uint8_t* pz = malloc(zb);
    uint8_t* ps = malloc(sb);
    CHECK(quick_pack_weights(q, z, s, K, N, 128, pw, ps, pz) == QUICK_OK, "pack");

    uint32_t* ow = malloc(wb);
    uint32_t* oz = malloc(zb);
    uint16_t* os = malloc(sb);
    CHECK(oracle_pack_qpk16(q, z, s, K, N, 128, ow, oz, os) == 0, "oracle pack");
    CHECK(memcmp(pw, ow, wb) == 0 && memcmp(pz, oz, zb) == 0 && memcmp(ps, os, sb) == 0,
          "library pack != oracle pack at K=%lld N=%lld", (long long)K, (long long)N);

    uint8_t* q2 = malloc((size_t)(K * N));
    uint8_t* z2 = malloc((size_t)(G * N));
    uint16_t* s2 = malloc((size_t)(G * N) * 2);
    CHECK(quick_unpack_weights(pw, ps, pz, K, N, 128, q2, z2, s2) == QUICK_OK, "unpack");
    CHECK(memcmp(q, q2, (size_t)(K * N)) == 0 && memcmp(z, z2, (size_t)(G * N)) == 0 &&
              memcmp(s, s2, (size_t)(G * N) * 2) == 0,
          "unpack(pack) != id");

    /* a value above 15 (last element): RANGE, outputs untouched */
    memset(pw, 0xA5, wb);
    q[K * N - 1] = 16;
    CHECK(quick_pack_weights(q, z, s, K, N, 128, pw, ps, pz) == QUICK_ERR_RANGE, "range");
    for (size_t i = 0; i < wb; ++i)
        if (pw[i] != 0xA5) {
            CHECK(0, "RANGE left a write at byte %zu", i);
            break;
        }
    q[K * N - 1] = 3;

    /* the oracle on the same data: dequant, full GEMM and a column subset */
    uint16_t* x = malloc((size_t)(M * K) * 2);
    for (int64_t i = 0; i < M * K; ++i) x[i] = (uint16_t)(0x3000 + (next_u32() % 0x1000)) | (next_u32() & 0x8000);
    double* W = malloc((size_t)(K * N) * sizeof(double));
    double* y = malloc((size_t)(M * N) * sizeof(double));
    CHECK(oracle_dequant_f64(q, z, s, K, N, 128, W) == 0, "dequant");
    CHECK(oracle_gemm_f64(x, q, z, s, M, N, K, 128, NULL, N, y, 2) == 0, "gemm");
    int64_t cols[3] = {0, N / 2, N - 1};
    double ysub[3 * 8];
    CHECK(M <= 8, "driver: M <= 8");
    CHECK(oracle_gemm_f64(x, q, z, s, M, N, K, 128, cols, 3, ysub, 1) == 0, "gemm cols");
    for (int64_t m = 0; m < M; ++m)
        for (int c = 0; c < 3; ++c) {
            double ref = 0.0;
            for (int64_t k = 0; k < K; ++k) ref += oracle_f16_to_f64(x[m * K + k]) * W[k * N + cols[c]];
            CHECK(ysub[m * 3 + c] == ref && y[m * N + cols[c]] == ref, "gemm mismatch at (%lld, %d)",
                  (long long)m, c);
        }
    int64_t bad_col = N;
    CHECK(oracle_gemm_f64(x, q, z, s, M, N, K, 128, &bad_col, 1, ysub, 1) != 0, "column out of range accepted");

    free(x); free(W); free(y);
    free(q2); free(z2); free(s2);
    free(ow); free(oz); free(os);
    free(pw); free(pz); free(ps);
    free(q); free(z); free(s);
}

static void check_errors(void)
{
    uint8_t q[128 * 16] = {0}, z[16] = {0};
    uint16_t s[16] = {0};
    uint8_t pw[1024], pz[8], ps[32];
    size_t a;
    CHECK(quick_packed_sizes(100, 16, 128, &a, NULL, NULL) == QUICK_ERR_SHAPE, "K % 128");
    CHECK(quick_packed_sizes(128, 8, 128, NULL, &a, NULL) == QUICK_ERR_SHAPE, "N % 16");
    CHECK(quick_packed_sizes(128, 16, 64, NULL, NULL, &a) == QUICK_ERR_UNSUPPORTED, "group");
    CHECK(quick_pack_weights(NULL, z, s, 128, 16, 128, pw, ps, pz) == QUICK_ERR_INVALID_ARG, "null q");
    CHECK(quick_pack_weights(q, z, s, 128, 16, 128, NULL, ps, pz) == QUICK_ERR_INVALID_ARG, "null out");
    CHECK(quick_unpack_weights(pw, ps, NULL, 128, 16, 128, q, z, s) == QUICK_ERR_INVALID_ARG, "null in");
    z[5] = 16;
    CHECK(quick_pack_weights(q, z, s, 128, 16, 128, pw, ps, pz) == QUICK_ERR_RANGE, "zero range");
    for (int st = -1; st <= 12; ++st) CHECK(quick_status_string(st) != NULL, "status string %d", st);
    CHECK(quick_pack_format_version() == 1, "format version");
}

int main(void)
{
    check_f16();
    check_errors();
    static const int64_t shapes[][3] = {{128, 16, 1}, {256, 48, 3}, {512, 272, 5}, {1024, 32, 2}, {384, 528, 8}};
    for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i) check_shape(shapes[i][0], shapes[i][1], shapes[i][2]);
    if (failures) {
        fprintf(stderr, "%d failures\n", failures);
        return 1;
    }
    printf("SANITIZE_OK\n");
    return 0;
}
