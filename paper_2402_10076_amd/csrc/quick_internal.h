// Internal declarations shared by the library's own translation units.
#pragma once
#include <cstdint>

namespace quick {

// Quantization group: consecutive input channels sharing one zero point and
// one scale.  The only group size the packed layout supports.
constexpr int64_t kGroup = 128;

// QUICK_OK or the status describing why (K, N, group) cannot be packed.
int check_pack_shape(int64_t K, int64_t N, int64_t group);

}  // namespace quick
