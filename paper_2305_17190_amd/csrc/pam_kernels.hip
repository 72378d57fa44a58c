// HIP kernels for piecewise affine multiplication (PAM) on gfx950.
//
// PAM (Kosson & Jaggi, Sec. 2.2): the product of two float32 numbers is
// replaced by the int32 sum of their encodings minus one exponent bias
// (127 << 23); the sign is the exclusive or of the signs, zero/denormal
// operands and underflowing results give signed zeros, overflowing results
// saturate at +-FLT_MAX, NaN/inf follow IEEE multiplication with a canonical
// quiet NaN.  PAM matrix products (Sec. 3.2) keep float32 accumulation.
//
// The matrix product is a vector-ALU contraction (PAM is not a product, so
// the matrix cores do not apply).  Each workgroup owns a BM x BN output tile,
// each thread an 8 x 8 register micro-tile, and K advances in chunks of 16
// staged through LDS.  When a chunk is written to LDS its operands are
// re-encoded once so that the per-MAC work is as small as the chunk's values
// allow; the workgroup votes on which encoding a chunk gets:
//
//   FAST     every operand has exponent field in [64, 190], so no product
//            can leave the normal range.  LDS holds a's encoding and b's
//            encoding minus the bias; per MAC: one v_add_u32 (the sign
//            bits add mod 2^32 to their exclusive or) + one v_add_f32.
//   GENERIC  every operand is finite with |x| < 2^64 (zeros, denormals and
//            products that underflow allowed).  Magnitudes are shifted into
//            a domain where one signed-saturating add clamps every underflow
//            (and every zero/denormal operand, encoded as INT32_MIN) to
//            INT32_MIN, i.e. to magnitude 0; per MAC: v_add_i32 clamp +
//            v_add3_u32 (restores the offset and adds both sign words) +
//            v_add_f32.  Results in (0, 2^-126) come out as denormal
//            encodings; the kernels run with float32 denormals flushed, so
//            the accumulate treats them as the zero PAM defines.
//   SPECIAL  anything else (inf, NaN, |x| >= 2^64): raw encodings and the
//            complete per-MAC definition.  Never taken on finite data whose
//            magnitudes stay below 2^64.
//
// Encodings used by GENERIC (m = |x| encoding, valid m in [2^23, 0x5F7FFFFF]):
//   x_A = m_A - 0x5F7FFFFF            in [-0x5EFFFFFF, 0], or INT32_MIN
//   y_B = m_B - 0x3F800000 - 0x20800001 in [-0x5F800001, -0x00800002], or INT32_MIN
//   sat(x_A + y_B) = sat(R - 2^31),    R = m_A + m_B - 0x3F800000
// R >= 0 gives the PAM magnitude R + (-2^31) exactly; R < 0 (underflow)
// saturates.  Since x_A <= 0 and y_B < 0, a zero/denormal operand on either
// side also lands on INT32_MIN.  R <= 0x7F7FFFFE, so nothing overflows.
// Adding (sign_A ^ 2^31) + sign_B mod 2^32 then yields sign | magnitude.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "pam_internal.h"

namespace pamk {

constexpr uint32_t kSign = 0x80000000u;
constexpr uint32_t kMag = 0x7FFFFFFFu;
constexpr uint32_t kBias = 0x3F800000u;     // 127 << 23
constexpr uint32_t kMinNormal = 0x00800000u;
constexpr uint32_t kFltMax = 0x7F7FFFFFu;
constexpr uint32_t kInf = 0x7F800000u;
constexpr uint32_t kQNaN = 0x7FC00000u;
constexpr uint32_t kExpMask = 0x7F800000u;

// GENERIC-encoding offsets (see the header comment).
constexpr uint32_t kOffA = 0x5F7FFFFFu;
constexpr uint32_t kOffB = 0x60000001u;     // bias + 0x20800001
constexpr int32_t kSentinel = INT32_MIN;

enum : int { kFast = 0, kGeneric = 1, kSpecial = 2 };

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

// ---------------------------------------------------------------------------
// Elementwise PAM.  HBM-bound: 8 bytes read and 4 written per element.
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(256) pam_mul_vec4_kernel(const uint4 *__restrict__ a,
                                                           const uint4 *__restrict__ b,
                                                           uint4 *__restrict__ out, int64_t n4) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        const uint4 x = a[i];
        const uint4 y = b[i];
        uint4 r;
        r.x = pam_full(x.x, y.x);
        r.y = pam_full(x.y, y.y);
        r.z = pam_full(x.z, y.z);
        r.w = pam_full(x.w, y.w);
        out[i] = r;
    }
}

__global__ void __launch_bounds__(256) pam_mul_scalar_kernel(const uint32_t *__restrict__ a,
                                                             const uint32_t *__restrict__ b,
                                                             uint32_t *__restrict__ out, int64_t n) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = pam_full(a[i], b[i]);
}

hipError_t launch_pam_mul(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    if (n <= 0)
        return hipSuccess;
    const bool aligned = ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                           reinterpret_cast<uintptr_t>(out)) & 15u) == 0;
    const int64_t max_blocks = 256 * 16;
    int64_t head = 0;
    if (aligned) {
        const int64_t n4 = n / 4;
        if (n4 > 0) {
            const int64_t blocks = std::min<int64_t>((n4 + 255) / 256, max_blocks);
            hipLaunchKernelGGL(pam_mul_vec4_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                               reinterpret_cast<const uint4 *>(a), reinterpret_cast<const uint4 *>(b),
                               reinterpret_cast<uint4 *>(out), n4);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess)
                return e;
        }
        head = n4 * 4;
    }
    const int64_t rest = n - head;
    if (rest > 0) {
        const int64_t blocks = std::min<int64_t>((rest + 255) / 256, max_blocks);
        hipLaunchKernelGGL(pam_mul_scalar_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                           reinterpret_cast<const uint32_t *>(a) + head,
                           reinterpret_cast<const uint32_t *>(b) + head,
                           reinterpret_cast<uint32_t *>(out) + head, rest);
        return hipGetLastError();
    }
    return hipSuccess;
}

// ---------------------------------------------------------------------------
// Tiled PAM matrix product
// ---------------------------------------------------------------------------

// An operand tile of D (rows of op(A), or columns of op(B)) x kChunkK staged
// through registers.  KCONTIG: element (o, kk) of the tile sits at
// base[(o0 + o) * ld + k0 + kk] (A with op N, B with op T); otherwise at
// base[(k0 + kk) * ld + o0 + o] (A with op T, B with op N).  Each thread
// holds L float4 groups of four consecutive elements of the contiguous axis.
template <int D, int NT, bool KCONTIG>
struct TileLoader {
    static constexpr int BK = kChunkK;
    static constexpr int L = D * BK / 4 / NT;
    static_assert(L >= 1 && D * BK / 4 == L * NT, "tile does not divide over the threads");
    uint4 v[L];

    // Rows past o_lim are clamped to the last valid row (their outputs are
    // discarded); elements at k >= k_lim are zero (they must add nothing).
    __device__ __forceinline__ void load(const float *__restrict__ base, int64_t ld, int o0, int o_lim,
                                         int k0, int k_lim, bool vec, int tid) {
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const int f = tid + NT * r;
            uint32_t e[4];
            if (KCONTIG) {
                const int o = min(o0 + f / (BK / 4), o_lim - 1);
                const int kq = k0 + (f % (BK / 4)) * 4;
                const float *src = base + (int64_t)o * ld + kq;
                if (vec && kq + 3 < k_lim) {
                    const uint4 q = *reinterpret_cast<const uint4 *>(src);
                    e[0] = q.x; e[1] = q.y; e[2] = q.z; e[3] = q.w;
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        e[c] = (kq + c < k_lim) ? __float_as_uint(src[c]) : 0u;
                }
            } else {
                const int kk = k0 + f / (D / 4);
                const int oq = o0 + (f % (D / 4)) * 4;
                if (kk < k_lim) {
                    const float *row = base + (int64_t)kk * ld;
                    if (vec && oq + 3 < o_lim) {
                        const uint4 q = *reinterpret_cast<const uint4 *>(row + oq);
                        e[0] = q.x; e[1] = q.y; e[2] = q.z; e[3] = q.w;
                    } else {
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            e[c] = __float_as_uint(row[min(oq + c, o_lim - 1)]);
                    }
                } else {
                    e[0] = e[1] = e[2] = e[3] = 0u;
                }
            }
            v[r] = make_uint4(e[0], e[1], e[2], e[3]);
        }
    }

    // bit 0: some operand is outside the FAST range; bit 1: outside GENERIC.
    __device__ __forceinline__ uint32_t classify() const {
        uint32_t not_fast = 0, not_generic = 0;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                not_fast |= ((e[c] & kExpMask) - 0x20000000u) > 0x3F000000u;   // field not in [64, 190]
                not_generic |= (e[c] & kMag) >= 0x5F800000u;                   // |x| >= 2^64, inf, NaN
            }
        }
        return not_fast | (not_generic << 1);
    }

    __device__ __forceinline__ static void encode(int mode, bool is_b, uint32_t u, uint32_t &p0, uint32_t &p1) {
        if (mode == kFast) {
            p0 = is_b ? u - kBias : u;
            p1 = 0u;
        } else if (mode == kGeneric) {
            const bool zero = (u & kExpMask) == 0u;
            const uint32_t m = u & kMag;
            p0 = zero ? (uint32_t)kSentinel : m - (is_b ? kOffB : kOffA);
            p1 = is_b ? (u & kSign) : ((u & kSign) ^ kSign);
        } else {
            p0 = u;
            p1 = 0u;
        }
    }

    // Write the chunk into LDS, k-major: s[plane][kk][o].
    template <int LDS_LD>
    __device__ __forceinline__ void store(uint32_t (*s)[BK][LDS_LD], int mode, bool is_b, int tid) const {
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const int f = tid + NT * r;
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
            uint32_t p0[4], p1[4];
#pragma unroll
            for (int c = 0; c < 4; ++c)
                encode(mode, is_b, e[c], p0[c], p1[c]);
            if (KCONTIG) {
                const int o = f / (BK / 4);
                const int kq = (f % (BK / 4)) * 4;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    s[0][kq + c][o] = p0[c];
                if (mode == kGeneric) {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        s[1][kq + c][o] = p1[c];
                }
            } else {
                const int kk = f / (D / 4);
                const int oq = (f % (D / 4)) * 4;
                *reinterpret_cast<uint4 *>(&s[0][kk][oq]) = make_uint4(p0[0], p0[1], p0[2], p0[3]);
                if (mode == kGeneric)
                    *reinterpret_cast<uint4 *>(&s[1][kk][oq]) = make_uint4(p1[0], p1[1], p1[2], p1[3]);
            }
        }
    }
};

template <int LD>
__device__ __forceinline__ void lds_frag(const uint32_t (*s)[kChunkK][LD], int plane, int kk, int i0, int half,
                                         uint32_t out[8]) {
    const uint4 lo = *reinterpret_cast<const uint4 *>(&s[plane][kk][i0]);
    const uint4 hi = *reinterpret_cast<const uint4 *>(&s[plane][kk][half + i0]);
    out[0] = lo.x; out[1] = lo.y; out[2] = lo.z; out[3] = lo.w;
    out[4] = hi.x; out[5] = hi.y; out[6] = hi.z; out[7] = hi.w;
}

template <int BM, int BN, bool TA, bool TB>
__global__ void __launch_bounds__(BM * BN / 64) pam_gemm_kernel(GemmParams p) {
    constexpr int BK = kChunkK;
    constexpr int NT = BM * BN / 64;
    constexpr int NW = NT / 64;
    constexpr int TXN = BN / 8;            // threads along n
    constexpr int HM = BM / 2;
    constexpr int HN = BN / 2;
    constexpr int LDA = BM + 4;            // padded LDS rows, 16-byte aligned
    constexpr int LDB = BN + 4;

    __shared__ uint32_t sA[2][BK][LDA];    // plane 0: value word, plane 1: sign word (GENERIC)
    __shared__ uint32_t sB[2][BK][LDB];
    __shared__ uint32_t sVote[NW];

    const int tid = threadIdx.x;
    const int tx = tid % TXN;
    const int ty = tid / TXN;
    const int tm = blockIdx.x / p.tiles_n;
    const int tn = blockIdx.x % p.tiles_n;
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int split = blockIdx.y;
    const int64_t bz = blockIdx.z;
    const float *A = p.A + bz * p.strideA;
    const float *B = p.B + bz * p.strideB;
    const int kb = split * p.k_per_split;
    const int ke = min(p.k, kb + p.k_per_split);
    const int nchunks = ke > kb ? (ke - kb + BK - 1) / BK : 0;

    TileLoader<BM, NT, !TA> la;
    TileLoader<BN, NT, TB> lb;

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = 0.0f;

    if (nchunks > 0) {
        la.load(A, p.lda, m0, p.m, kb, ke, p.vec_a != 0, tid);
        lb.load(B, p.ldb, n0, p.n, kb, ke, p.vec_b != 0, tid);
    }

    for (int c = 0; c < nchunks; ++c) {
        // Workgroup vote on the chunk's encoding.
        const uint32_t f = la.classify() | lb.classify();
        const uint64_t nf = __ballot(f & 1u);
        const uint64_t ng = __ballot(f & 2u);
        if ((tid & 63) == 0)
            sVote[tid >> 6] = (nf ? 1u : 0u) | (ng ? 2u : 0u);
        __syncthreads();
        uint32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            v |= sVote[w];
        const int mode = (v & 2u) ? kSpecial : ((v & 1u) ? kGeneric : kFast);

        la.template store<LDA>(sA, mode, false, tid);
        lb.template store<LDB>(sB, mode, true, tid);
        __syncthreads();

        if (c + 1 < nchunks) {
            const int k0 = kb + (c + 1) * BK;
            la.load(A, p.lda, m0, p.m, k0, ke, p.vec_a != 0, tid);
            lb.load(B, p.ldb, n0, p.n, k0, ke, p.vec_b != 0, tid);
        }

        if (mode == kFast) {
#pragma unroll
            for (int kk = 0; kk < BK; ++kk) {
                uint32_t a[8], b[8];
                lds_frag<LDA>(sA, 0, kk, ty * 4, HM, a);
                lds_frag<LDB>(sB, 0, kk, tx * 4, HN, b);
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        acc[i][j] += __uint_as_float(a[i] + b[j]);
            }
        } else if (mode == kGeneric) {
#pragma unroll
            for (int kk = 0; kk < BK; ++kk) {
                uint32_t x[8], sa[8], y[8], sb[8];
                lds_frag<LDA>(sA, 0, kk, ty * 4, HM, x);
                lds_frag<LDA>(sA, 1, kk, ty * 4, HM, sa);
                lds_frag<LDB>(sB, 0, kk, tx * 4, HN, y);
                lds_frag<LDB>(sB, 1, kk, tx * 4, HN, sb);
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int32_t t = __builtin_elementwise_add_sat((int32_t)x[i], (int32_t)y[j]);
                        acc[i][j] += __uint_as_float((uint32_t)t + sa[i] + sb[j]);
                    }
            }
        } else {
#pragma unroll 1
            for (int kk = 0; kk < BK; ++kk) {
                uint32_t a[8], b[8];
                lds_frag<LDA>(sA, 0, kk, ty * 4, HM, a);
                lds_frag<LDB>(sB, 0, kk, tx * 4, HN, b);
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        acc[i][j] += __uint_as_float(pam_full(a[i], b[j]));
            }
        }
    }

    // Epilogue: final output, or this split's slice of the partial sums.
    float *out;
    int64_t ld;
    if (p.W != nullptr) {
        out = p.W + ((bz * p.splits + split) * (int64_t)p.m) * p.n;
        ld = p.n;
    } else {
        out = p.C + bz * p.strideC;
        ld = p.ldc;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int row = m0 + (i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4));
        if (row >= p.m)
            continue;
        float *orow = out + (int64_t)row * ld;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int col = n0 + (h == 0 ? tx * 4 : HN + tx * 4);
            if (p.vec_c && col + 3 < p.n) {
                *reinterpret_cast<float4 *>(orow + col) =
                    make_float4(acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3]);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (col + j < p.n)
                        orow[col + j] = acc[i][4 * h + j];
            }
        }
    }
}

template <int BM, int BN>
static hipError_t launch_tile(bool ta, bool tb, const GemmParams &p, dim3 grid, hipStream_t stream) {
    const dim3 block(BM * BN / 64);
    if (!ta && !tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, false, false>), grid, block, 0, stream, p);
    else if (!ta && tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, false, true>), grid, block, 0, stream, p);
    else if (ta && !tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, true, false>), grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, true, true>), grid, block, 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_pam_gemm(int tile_m, int tile_n, bool trans_a, bool trans_b, const GemmParams &p,
                           int64_t batch, hipStream_t stream) {
    const int64_t tiles_m = (p.m + tile_m - 1) / tile_m;
    const dim3 grid((unsigned)(tiles_m * p.tiles_n), (unsigned)p.splits, (unsigned)batch);
    if (tile_m == 128 && tile_n == 128)
        return launch_tile<128, 128>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 128 && tile_n == 64)
        return launch_tile<128, 64>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 64 && tile_n == 64)
        return launch_tile<64, 64>(trans_a, trans_b, p, grid, stream);
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Split-K reduction and k == 0 fill
// ---------------------------------------------------------------------------

__global__ void __launch_bounds__(256) splitk_reduce_kernel(const float *__restrict__ W, float *__restrict__ C,
                                                            int32_t m, int32_t n, int64_t ldc, int64_t strideC,
                                                            int32_t splits, int64_t total) {
    const int64_t mn = (int64_t)m * n;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t b = idx / mn;
        const int64_t r = idx - b * mn;
        const int64_t i = r / n;
        const int64_t j = r - i * n;
        const float *w = W + b * splits * mn + r;
        float s = 0.0f;
        for (int q = 0; q < splits; ++q)
            s += w[q * mn];
        C[b * strideC + i * ldc + j] = s;
    }
}

hipError_t launch_splitk_reduce(const float *W, float *C, int32_t m, int32_t n, int64_t ldc, int64_t strideC,
                                int32_t splits, int64_t batch, hipStream_t stream) {
    const int64_t total = batch * (int64_t)m * n;
    if (total <= 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 256 * 32);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, W, C, m, n, ldc, strideC,
                       splits, total);
    return hipGetLastError();
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float *__restrict__ C, int32_t m, int32_t n, int64_t ldc,
                                                        int64_t strideC, int64_t total) {
    const int64_t mn = (int64_t)m * n;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t b = idx / mn;
        const int64_t r = idx - b * mn;
        const int64_t i = r / n;
        const int64_t j = r - i * n;
        C[b * strideC + i * ldc + j] = 0.0f;
    }
}

hipError_t launch_fill_zero(float *C, int32_t m, int32_t n, int64_t ldc, int64_t strideC, int64_t batch,
                            hipStream_t stream) {
    const int64_t total = batch * (int64_t)m * n;
    if (total <= 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((total + 255) / 256, 256 * 32);
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, C, m, n, ldc, strideC, total);
    return hipGetLastError();
}

}  // namespace pamk
