// HIP kernels for the elementwise piecewise affine operations on gfx950
// (Kosson & Jaggi, Sec. 2.2-2.3): PAM itself, piecewise affine division (PAD),
// palog2 and paexp2, and the mantissa rounding of the narrow products.  All
// are HBM-bound streams; each element goes through a branch-free integer /
// float sequence of a few vector ops.
//
// PAM is the complete per-element definition shared with the matrix products
// (pam_scalar.h).
//
// PAD is the inverse of PAM: the int32 difference of the two encodings plus
// one exponent bias (127 << 23); the borrow of the subtraction realises
// 1{M_A - M_B < 0}.  Edge cases as for PAM: sign = exclusive or, denormal
// operands count as zero, NaN operand / 0 ./ 0 / inf ./ inf give 0x7FC00000,
// x ./ 0 and inf ./ x give a signed inf, 0 ./ x and x ./ inf a signed zero, a
// result exponent field <= 0 a signed zero and >= 255 +-FLT_MAX.
//
// palog2(A) = E_A + M_A is the encoding of A read as a fixed-point number with
// 23 fraction bits, minus 127: one int32 subtract and one int-to-float
// conversion (rounded to nearest even, as the conversion does), then an exact
// scaling by 2^-23.  Outside A > 0 it follows log2 (+-0 and denormals -> -inf,
// negative -> NaN, +inf -> +inf, NaN -> 0x7FC00000).
//
// paexp2(A) = 2^floor(A) (1 + A - floor(A)) is the float whose encoding is
// A * 2^23 + 127 * 2^23 read back as bits: the product is exact, rounding it
// to an integer (nearest even) rounds the result to the nearest float32, and
// a carry out of the mantissa moves into the exponent as it should.  Results
// below 2^-126 are +0, above FLT_MAX +inf; -inf -> +0, NaN -> 0x7FC00000.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "pam_internal.h"
#include "pam_scalar.h"

namespace pamk {
namespace {

constexpr uint32_t kNegInf = 0xFF800000u;

struct PamOp {
    __device__ __forceinline__ uint32_t operator()(uint32_t ua, uint32_t ub) const { return pam_full(ua, ub); }
};

struct PadOp {
    __device__ __forceinline__ uint32_t operator()(uint32_t ua, uint32_t ub) const {
        const uint32_t s = (ua ^ ub) & kSign;
        const uint32_t ma = ua & kMag;
        const uint32_t mb = ub & kMag;
        // Difference of the magnitudes, in int32 range for every input; the
        // biased result t = d + bias is checked through d so it never wraps.
        const int32_t d = (int32_t)ma - (int32_t)mb;
        uint32_t r = (uint32_t)d + kBias;
        r = (d < (int32_t)kMinNormal - (int32_t)kBias) ? 0u : r;            // exponent field <= 0
        r = (d > (int32_t)(kFltMax - kBias)) ? kFltMax : r;                  // exponent field >= 255
        const bool a_zero = ma < kMinNormal;
        const bool b_zero = mb < kMinNormal;
        const bool a_inf = ma == kInf;
        const bool b_inf = mb == kInf;
        uint32_t out = s | r;
        out = b_zero ? (s | kInf) : out;                                    // x ./ 0
        out = a_zero ? (b_zero ? kQNaN : s) : out;                          // 0 ./ x, 0 ./ 0
        out = b_inf ? s : out;                                              // x ./ inf
        out = a_inf ? (b_inf ? kQNaN : (s | kInf)) : out;                   // inf ./ x, inf ./ inf
        out = (ma > kInf || mb > kInf) ? kQNaN : out;
        return out;
    }
};

struct Palog2Op {
    __device__ __forceinline__ uint32_t operator()(uint32_t u) const {
        const uint32_t mag = u & kMag;
        const float v = (float)(int32_t)(mag - kBias) * 0x1p-23f;
        uint32_t out = __float_as_uint(v);
        out = (mag < kMinNormal) ? kNegInf : out;
        out = (u >= kSign && mag >= kMinNormal) ? kQNaN : out;
        out = (u == kInf) ? kInf : out;
        out = (mag > kInf) ? kQNaN : out;
        return out;
    }
};

struct Paexp2Op {
    __device__ __forceinline__ uint32_t operator()(uint32_t u) const {
        const uint32_t mag = u & kMag;
        float x = __uint_as_float(u);
        x = (mag < kMinNormal || mag > kInf) ? 0.0f : x;
        x = fminf(fmaxf(x, -255.0f), 255.0f);          // beyond +-255 the result is saturated anyway
        const int32_t r = (int32_t)__builtin_rintf(x * 8388608.0f);   // exact product, nearest even
        uint32_t out = (uint32_t)r + kBias;
        out = (r >= (int32_t)(kInf - kBias)) ? kInf : out;          // field >= 255
        out = (r < (int32_t)kMinNormal - (int32_t)kBias) ? 0u : out;  // field <= 0
        out = (mag > kInf) ? kQNaN : out;
        return out;
    }
};

// Rounding to 23 - drop mantissa bits (the inputs of the narrow matrix
// product), as an elementwise op.
struct RoundOp {
    uint32_t drop;
    __device__ __forceinline__ uint32_t operator()(uint32_t u) const {
        const uint32_t low = (1u << drop) - 1u;
        const uint32_t rounded = (u + (low >> 1) + ((u >> drop) & 1u)) & ~low;
        return ((u & kInf) == kInf) ? u : rounded;
    }
};

// 16-byte groups, read and written with non-temporal hints (a stream touches
// each byte once), one group per thread: with a workgroup per 256 groups the
// chip keeps far more loads in flight than a short grid-stride loop would.
// The grid-stride loop only runs past kMaxBlocks workgroups.  The pointers
// may alias (every op may run in place: each thread reads its elements
// before it writes them), so none is marked __restrict__.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename Op>
__global__ void __launch_bounds__(256) binary_vec4_kernel(const u32x4 *a, const u32x4 *b, u32x4 *out,
                                                          int64_t n4) {
    const Op op;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const u32x4 x = __builtin_nontemporal_load(a + i);
        const u32x4 y = __builtin_nontemporal_load(b + i);
        const u32x4 r = {op(x.x, y.x), op(x.y, y.y), op(x.z, y.z), op(x.w, y.w)};
        __builtin_nontemporal_store(r, out + i);
    }
}

template <typename Op>
__global__ void __launch_bounds__(256) binary_scalar_kernel(const uint32_t *a, const uint32_t *b,
                                                            uint32_t *out, int64_t n) {
    const Op op;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        __builtin_nontemporal_store(op(__builtin_nontemporal_load(a + i), __builtin_nontemporal_load(b + i)),
                                    out + i);
}

template <typename Op>
__global__ void __launch_bounds__(256) unary_vec4_kernel(const u32x4 *a, u32x4 *out, int64_t n4,
                                                         Op op) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const u32x4 x = __builtin_nontemporal_load(a + i);
        const u32x4 r = {op(x.x), op(x.y), op(x.z), op(x.w)};
        __builtin_nontemporal_store(r, out + i);
    }
}

template <typename Op>
__global__ void __launch_bounds__(256) unary_scalar_kernel(const uint32_t *a, uint32_t *out, int64_t n,
                                                           Op op) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        __builtin_nontemporal_store(op(__builtin_nontemporal_load(a + i)), out + i);
}

// Workgroups per launch at most (the grid, in threads, stays below 2^32);
// 16-byte groups when every pointer is 16-byte aligned, then the scalar
// kernel for the remaining 0..3 elements (or everything).
constexpr int64_t kMaxBlocks = 16777215;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename Op>
hipError_t launch_binary(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    int64_t head = 0;
    if (aligned16(a) && aligned16(b) && aligned16(out)) {
        const int64_t n4 = n / 4;
        if (n4 > 0) {
            const int64_t blocks = std::min<int64_t>((n4 + 255) / 256, kMaxBlocks);
            hipLaunchKernelGGL(binary_vec4_kernel<Op>, dim3((unsigned)blocks), dim3(256), 0, stream,
                               reinterpret_cast<const u32x4 *>(a), reinterpret_cast<const u32x4 *>(b),
                               reinterpret_cast<u32x4 *>(out), n4);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess)
                return e;
        }
        head = n4 * 4;
    }
    const int64_t rest = n - head;
    if (rest > 0) {
        const int64_t blocks = std::min<int64_t>((rest + 255) / 256, kMaxBlocks);
        hipLaunchKernelGGL(binary_scalar_kernel<Op>, dim3((unsigned)blocks), dim3(256), 0, stream,
                           reinterpret_cast<const uint32_t *>(a) + head, reinterpret_cast<const uint32_t *>(b) + head,
                           reinterpret_cast<uint32_t *>(out) + head, rest);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <typename Op>
hipError_t launch_unary(const float *a, float *out, int64_t n, hipStream_t stream, Op op = Op()) {
    if (n <= 0)
        return hipSuccess;
    int64_t head = 0;
    if (aligned16(a) && aligned16(out)) {
        const int64_t n4 = n / 4;
        if (n4 > 0) {
            const int64_t blocks = std::min<int64_t>((n4 + 255) / 256, kMaxBlocks);
            hipLaunchKernelGGL(unary_vec4_kernel<Op>, dim3((unsigned)blocks), dim3(256), 0, stream,
                               reinterpret_cast<const u32x4 *>(a), reinterpret_cast<u32x4 *>(out), n4, op);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess)
                return e;
        }
        head = n4 * 4;
    }
    const int64_t rest = n - head;
    if (rest > 0) {
        const int64_t blocks = std::min<int64_t>((rest + 255) / 256, kMaxBlocks);
        hipLaunchKernelGGL(unary_scalar_kernel<Op>, dim3((unsigned)blocks), dim3(256), 0, stream,
                           reinterpret_cast<const uint32_t *>(a) + head, reinterpret_cast<uint32_t *>(out) + head,
                           rest, op);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_pam_mul(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    return launch_binary<PamOp>(a, b, out, n, stream);
}

hipError_t launch_pad(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    return launch_binary<PadOp>(a, b, out, n, stream);
}

hipError_t launch_palog2(const float *a, float *out, int64_t n, hipStream_t stream) {
    return launch_unary<Palog2Op>(a, out, n, stream);
}

hipError_t launch_paexp2(const float *a, float *out, int64_t n, hipStream_t stream) {
    return launch_unary<Paexp2Op>(a, out, n, stream);
}

hipError_t launch_round_mantissa(const float *a, float *out, int64_t n, int drop, hipStream_t stream) {
    return launch_unary<RoundOp>(a, out, n, stream, RoundOp{(uint32_t)drop});
}

}  // namespace pamk
