// Offline weight reorder (paper, Section 3.1 and Section 3.2) -- host side.
//
// The static 4-bit weights are rearranged once so that one 16-byte load per
// lane delivers, for the 16x16x32 f16 matrix instruction of gfx950, exactly
// the eight k-consecutive weights that lane contributes to the instruction's
// weight operand -- for four consecutive 32-wide k steps -- and so that the
// nibbles inside each 32-bit word come out of the mask-and-shift dequantizer
// as in-order f16 pairs (the "dequant-aware" second reorder of Section 3.2).
//
// Layout QPK16 (version 1).  Unit u = nt*KG + kg for n-tile nt (16 output
// columns) and k-group kg (128 input channels), KG = K/128.  A unit is 64
// lanes x 4 words x 32 bits = 1 KiB.  Lane l covers column 16*nt + (l & 15)
// and, in word j, input channels 128*kg + 32*j + 8*(l >> 4) + e, e = 0..7.
// Nibble i of the word holds element kSlotElem[i]: the even elements in
// nibbles 0..3, the odd ones in nibbles 4..7.
//
// Zero points: per unit two words, word (c >> 3) holding column c's zero in
// nibble (c & 7).  Scales: per unit 16 binary16 values in column order.
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>
#include <algorithm>

#include "quick.h"
#include "quick_internal.h"

namespace {

// nibble index -> element (k offset inside the lane's 8 consecutive k).
constexpr int kSlotElem[8] = {0, 2, 4, 6, 1, 3, 5, 7};

template <class F>
void parallel_for(int64_t n, F&& f)
{
    unsigned hw = std::thread::hardware_concurrency();
    int64_t nth = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, 32));
    nth = std::min(nth, n);
    if (nth <= 1) {
        for (int64_t i = 0; i < n; ++i) f(i);
        return;
    }
    std::vector<std::thread> th;
    th.reserve(nth);
    for (int64_t t = 0; t < nth; ++t) {
        th.emplace_back([&, t] {
            for (int64_t i = t; i < n; i += nth) f(i);
        });
    }
    for (auto& x : th) x.join();
}

}  // namespace

namespace quick {

int check_pack_shape(int64_t K, int64_t N, int64_t group)
{
    if (group != kGroup) return QUICK_ERR_UNSUPPORTED;
    if (K <= 0 || N <= 0 || K % kGroup != 0 || N % 16 != 0) return QUICK_ERR_SHAPE;
    return QUICK_OK;
}

}  // namespace quick

extern "C" int quick_pack_format_version(void) { return 1; }

extern "C" int quick_packed_sizes(int64_t K, int64_t N, int64_t group, size_t* packed_bytes,
                                  size_t* zeros_bytes, size_t* scales_bytes)
{
    int st = quick::check_pack_shape(K, N, group);
    if (st) return st;
    if (packed_bytes) *packed_bytes = (size_t)(K * N / 2);
    if (zeros_bytes) *zeros_bytes = (size_t)(K * N / 256);
    if (scales_bytes) *scales_bytes = (size_t)(K * N / 64);
    return QUICK_OK;
}

extern "C" int quick_pack_weights(const uint8_t* q, const uint8_t* z, const uint16_t* s,
                                  int64_t K, int64_t N, int64_t group, void* packed,
                                  void* scales, void* zeros)
{
    if (!q || !z || !s || !packed || !scales || !zeros) return QUICK_ERR_INVALID_ARG;
    int st = quick::check_pack_shape(K, N, group);
    if (st) return st;
    const int64_t KG = K / quick::kGroup;
    const int64_t NT = N / 16;

    // Range check first so that a bad input leaves the outputs untouched.
    bool bad = false;
    for (int64_t i = 0; i < K * N && !bad; ++i) bad = q[i] > 15;
    for (int64_t i = 0; i < KG * N && !bad; ++i) bad = z[i] > 15;
    if (bad) return QUICK_ERR_RANGE;

    uint32_t* pw = static_cast<uint32_t*>(packed);
    uint32_t* pz = static_cast<uint32_t*>(zeros);
    uint16_t* ps = static_cast<uint16_t*>(scales);

    parallel_for(NT, [&](int64_t nt) {
        for (int64_t kg = 0; kg < KG; ++kg) {
            const int64_t unit = nt * KG + kg;
            uint32_t* dst = pw + unit * 256;
            for (int lane = 0; lane < 64; ++lane) {
                const int64_t n = nt * 16 + (lane & 15);
                for (int j = 0; j < 4; ++j) {
                    const int64_t k0 = kg * quick::kGroup + 32 * j + 8 * (lane >> 4);
                    uint32_t w = 0;
                    for (int i = 0; i < 8; ++i)
                        w |= (uint32_t)q[(k0 + kSlotElem[i]) * N + n] << (4 * i);
                    dst[lane * 4 + j] = w;
                }
            }
            for (int h = 0; h < 2; ++h) {
                uint32_t w = 0;
                for (int i = 0; i < 8; ++i)
                    w |= (uint32_t)z[kg * N + nt * 16 + 8 * h + i] << (4 * i);
                pz[unit * 2 + h] = w;
            }
            std::memcpy(ps + unit * 16, s + kg * N + nt * 16, 16 * sizeof(uint16_t));
        }
    });
    return QUICK_OK;
}

extern "C" int quick_unpack_weights(const void* packed, const void* scales, const void* zeros,
                                    int64_t K, int64_t N, int64_t group, uint8_t* q, uint8_t* z,
                                    uint16_t* s)
{
    if (!packed || !scales || !zeros || !q || !z || !s) return QUICK_ERR_INVALID_ARG;
    int st = quick::check_pack_shape(K, N, group);
    if (st) return st;
    const int64_t KG = K / quick::kGroup;
    const int64_t NT = N / 16;
    const uint32_t* pw = static_cast<const uint32_t*>(packed);
    const uint32_t* pz = static_cast<const uint32_t*>(zeros);
    const uint16_t* ps = static_cast<const uint16_t*>(scales);

    parallel_for(NT, [&](int64_t nt) {
        for (int64_t kg = 0; kg < KG; ++kg) {
            const int64_t unit = nt * KG + kg;
            const uint32_t* src = pw + unit * 256;
            for (int lane = 0; lane < 64; ++lane) {
                const int64_t n = nt * 16 + (lane & 15);
                for (int j = 0; j < 4; ++j) {
                    const int64_t k0 = kg * quick::kGroup + 32 * j + 8 * (lane >> 4);
                    const uint32_t w = src[lane * 4 + j];
                    for (int i = 0; i < 8; ++i)
                        q[(k0 + kSlotElem[i]) * N + n] = (uint8_t)((w >> (4 * i)) & 15u);
                }
            }
            for (int h = 0; h < 2; ++h) {
                const uint32_t w = pz[unit * 2 + h];
                for (int i = 0; i < 8; ++i)
                    z[kg * N + nt * 16 + 8 * h + i] = (uint8_t)((w >> (4 * i)) & 15u);
            }
            std::memcpy(s + kg * N + nt * 16, ps + unit * 16, 16 * sizeof(uint16_t));
        }
    });
    return QUICK_OK;
}

extern "C" const char* quick_status_string(int status)
{
    switch (status) {
    case QUICK_OK: return "QUICK_OK";
    case QUICK_ERR_INVALID_ARG: return "QUICK_ERR_INVALID_ARG: null pointer or invalid argument";
    case QUICK_ERR_SHAPE: return "QUICK_ERR_SHAPE: need M >= 0, K % 128 == 0, N % 16 == 0";
    case QUICK_ERR_UNSUPPORTED: return "QUICK_ERR_UNSUPPORTED: only group == 128 is supported";
    case QUICK_ERR_RANGE: return "QUICK_ERR_RANGE: a 4-bit value exceeds 15";
    case QUICK_ERR_ALIGNMENT: return "QUICK_ERR_ALIGNMENT: device pointer misaligned";
    case QUICK_ERR_HIP: return "QUICK_ERR_HIP: HIP runtime error";
    case QUICK_ERR_WORKSPACE: return "QUICK_ERR_WORKSPACE: workspace missing or too small";
    case QUICK_ERR_IO: return "QUICK_ERR_IO: tune table file unreadable or malformed";
    case QUICK_ERR_CAPTURE:
        return "QUICK_ERR_CAPTURE: the internal workspace would have to be allocated or grown while the stream "
               "is being captured (call once on that stream before capturing, or pass a workspace)";
    default: return "unknown quick status";
    }
}
