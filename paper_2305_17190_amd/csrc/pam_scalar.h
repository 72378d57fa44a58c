// Float32 encoding constants and the complete piecewise affine multiplication
// of two float32 encodings (Kosson & Jaggi, Sec. 2.2), shared by the matrix
// product kernels (their SPECIAL path) and the elementwise stream.  Included
// by the HIP sources only.
//
// PAM: the int32 sum of the two magnitudes' encodings minus one exponent bias
// (127 << 23); the sign is the exclusive or of the signs; zero and denormal
// operands and results whose exponent field would be <= 0 give a signed zero;
// results whose exponent field would be >= 255 saturate at +-FLT_MAX; a NaN
// operand or inf times zero gives the quiet NaN 0x7FC00000, inf times anything
// else a signed inf.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pamk {

constexpr uint32_t kSign = 0x80000000u;
constexpr uint32_t kMag = 0x7FFFFFFFu;
constexpr uint32_t kBias = 0x3F800000u;     // 127 << 23
constexpr uint32_t kMinNormal = 0x00800000u;
constexpr uint32_t kFltMax = 0x7F7FFFFFu;
constexpr uint32_t kInf = 0x7F800000u;
constexpr uint32_t kQNaN = 0x7FC00000u;
constexpr uint32_t kExpMask = 0x7F800000u;

constexpr uint32_t kSignExp = 0xFF800000u;
constexpr uint32_t kMant = 0x007FFFFFu;

// Complete PAM of two float32 encodings, every input class.
__device__ __forceinline__ uint32_t pam_full(uint32_t ua, uint32_t ub) {
    const uint32_t s = (ua ^ ub) & kSign;
    const uint32_t ma = ua & kMag;
    const uint32_t mb = ub & kMag;
    const uint32_t sum = ma + mb;                       // <= 0xFFFFFFFE, no wrap
    uint32_t r = sum - kBias;
    r = (sum < kBias + kMinNormal) ? 0u : r;            // underflow -> zero
    r = (sum > kBias + kFltMax) ? kFltMax : r;          // overflow -> FLT_MAX
    r = (ma < kMinNormal || mb < kMinNormal) ? 0u : r;  // zero / denormal operand
    uint32_t out = s | r;
    const bool a_inf = ma == kInf;
    const bool b_inf = mb == kInf;
    const bool nan_in = (ma > kInf) || (mb > kInf);
    const bool inf_zero = (a_inf && mb < kMinNormal) || (b_inf && ma < kMinNormal);
    out = (a_inf || b_inf) ? (s | kInf) : out;
    out = (nan_in || inf_zero) ? kQNaN : out;
    return out;
}

}  // namespace pamk
