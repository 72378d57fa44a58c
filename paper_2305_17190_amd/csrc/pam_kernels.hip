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
// staged through LDS.  On gfx950 the integer add and the float32 add, mul and
// fma issue at twice the rate of other vector ops (max, add3, saturating
// add), so the per-MAC work is built from those four only.
//
// SCALED encoding (written to LDS once per chunk):
//   A element a = (-1)^s 2^E (1 + M):  aM = encoding of 1 + M (exponent
//       field 127, a's mantissa) and m = a with its mantissa cleared, i.e.
//       the float +-2^E, or +-0 when a is zero/denormal.
//   B element b:  b' = encoding of b minus 0x3F800000 (zero and denormal b
//       are encoded as a signed zero first).
//   Then t = aM + b' (one int add) is the encoding of PAM(1 + M, b): adding
//   1 + M's mantissa to b's encoding is Sec. 2.2's sum with E = 0 on the A
//   side.  PAM is exact under power-of-two scaling (Fig. 2: the pattern
//   repeats per octave), so t * m = PAM(a, b) whenever the result is a normal
//   number; the float multiply also supplies the sign.  A zero b makes t a
//   denormal encoding, which the float unit (denormals flushed) reads as 0.
//
//   S2 (per MAC: v_add_u32, v_fmac_f32): acc = fma(t, m, acc).  Exact when
//      no product underflows, which holds when every nonzero operand has
//      exponent field in [64, 190].
//   S3 (per MAC: v_add_u32, v_mul_f32, v_add_f32): p = t * m is rounded on
//      its own, so an underflowing product flushes to the signed zero PAM
//      defines; exact for all finite operands with |x| < 2^64.
//   Each wave picks S2 or S3 per k step from a bit mask of the operands it
//   will read at that k ("tiny": nonzero with exponent field 1..63).
//
// SPECIAL: a chunk holding inf, NaN or |x| >= 2^64 is written raw and
// evaluated with the complete per-MAC definition (never taken on finite data
// whose magnitudes stay below 2^64).

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

constexpr uint32_t kSignExp = 0xFF800000u;
constexpr uint32_t kMant = 0x007FFFFFu;

enum : int { kScaled = 0, kSpecial = 1 };

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

    // Nonzero when some element needs the SPECIAL path: inf, NaN or |x| >= 2^64.
    __device__ __forceinline__ uint32_t needs_special() const {
        uint32_t any = 0;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int c = 0; c < 4; ++c)
                any |= (e[c] & kMag) >= 0x5F800000u;
        }
        return any;
    }

    // "Tiny": a normal number with exponent field 1..63, whose products can
    // underflow.  Zeros and denormals are not tiny (their products are exact
    // zeros in both S2 and S3).
    __device__ __forceinline__ static bool tiny(uint32_t u) {
        return (u & kExpMask) - kMinNormal < (63u << 23);
    }

    // Write the chunk into LDS, k-major: s[plane][kk][o].  SCALED: A gets
    // plane 0 = aM, plane 1 = m; B gets plane 0 = b'.  SPECIAL: raw words in
    // plane 0.  Tiny elements set bit kk of mask[w] (A: the wave that reads
    // row o, from row_wave; B: mask[b_slot], read by every wave).
    template <int LDS_LD, typename RowWave>
    __device__ __forceinline__ void store(uint32_t (*s)[BK][LDS_LD], int mode, bool is_b, int tid, uint32_t *mask,
                                          int b_slot, RowWave row_wave) const {
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const int f = tid + NT * r;
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
            uint32_t p0[4], p1[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t u = e[c];
                if (mode == kSpecial) {
                    p0[c] = u;
                    p1[c] = 0u;
                } else if (is_b) {
                    const uint32_t z = ((u & kExpMask) == 0u) ? (u & kSign) : u;   // denormal -> signed zero
                    p0[c] = z - kBias;
                    p1[c] = 0u;
                } else {
                    p0[c] = (u & kMant) | kBias;
                    p1[c] = u & kSignExp;
                }
            }
            int o, kk0;
            if (KCONTIG) {
                o = f / (BK / 4);
                kk0 = (f % (BK / 4)) * 4;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    s[0][kk0 + c][o] = p0[c];
                if (!is_b && mode != kSpecial) {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        s[1][kk0 + c][o] = p1[c];
                }
            } else {
                kk0 = f / (D / 4);
                o = (f % (D / 4)) * 4;
                *reinterpret_cast<uint4 *>(&s[0][kk0][o]) = make_uint4(p0[0], p0[1], p0[2], p0[3]);
                if (!is_b && mode != kSpecial)
                    *reinterpret_cast<uint4 *>(&s[1][kk0][o]) = make_uint4(p1[0], p1[1], p1[2], p1[3]);
            }
            if (mode != kSpecial) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if (tiny(e[c])) {
                        const int kk = KCONTIG ? kk0 + c : kk0;
                        const int oc = KCONTIG ? o : o + c;
                        atomicOr(&mask[is_b ? b_slot : row_wave(oc)], 1u << kk);
                    }
                }
            }
        }
    }
};

// S3 update of a micro-tile: the product t * m is rounded (denormal results
// flushed) before it is added, never fused into an fma.
__device__ __forceinline__ void s3_accumulate(float (&acc)[8][8], const uint32_t (&am)[8], const uint32_t (&mm)[8],
                                              const uint32_t (&bb)[8]) {
#pragma clang fp contract(off)
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float prod = __uint_as_float(am[i] + bb[j]) * __uint_as_float(mm[i]);
            acc[i][j] = acc[i][j] + prod;
        }
}

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
    constexpr int TY_PER_WAVE = 64 / TXN;  // micro-tile rows (of 2 x 4) per wave
    constexpr int HM = BM / 2;
    constexpr int HN = BN / 2;
    constexpr int LDA = BM + 4;            // padded LDS rows, 16-byte aligned
    constexpr int LDB = BN + 4;

    __shared__ uint32_t sA[2][BK][LDA];    // SCALED: plane 0 aM, plane 1 m; SPECIAL: plane 0 raw
    __shared__ uint32_t sB[1][BK][LDB];    // SCALED: b'; SPECIAL: raw
    __shared__ uint32_t sVote[NW];
    __shared__ uint32_t sMask[2][NW + 1];  // per chunk parity: tiny bits per wave (A rows) and for B

    const int tid = threadIdx.x;
    const int tx = tid % TXN;
    const int ty = tid / TXN;
    const int wave = tid >> 6;
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
    auto row_wave = [](int o) { return ((o % HM) / 4) / TY_PER_WAVE; };

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = 0.0f;

    if (tid < 2 * (NW + 1))
        (&sMask[0][0])[tid] = 0u;

    if (nchunks > 0) {
        la.load(A, p.lda, m0, p.m, kb, ke, p.vec_a != 0, tid);
        lb.load(B, p.ldb, n0, p.n, kb, ke, p.vec_b != 0, tid);
    }

    for (int c = 0; c < nchunks; ++c) {
        // Workgroup vote: SPECIAL if any operand of the chunk is inf, NaN or >= 2^64.
        const uint64_t sp = __ballot(la.needs_special() | lb.needs_special());
        if ((tid & 63) == 0)
            sVote[wave] = sp ? 1u : 0u;
        __syncthreads();
        uint32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            v |= sVote[w];
        const int mode = v ? kSpecial : kScaled;

        uint32_t *mask = sMask[c & 1];
        if (tid < NW + 1)
            sMask[(c + 1) & 1][tid] = 0u;   // next chunk's masks; last read two chunks ago
        la.template store<LDA>(sA, mode, false, tid, mask, NW, row_wave);
        lb.template store<LDB>(sB, mode, true, tid, mask, NW, row_wave);
        __syncthreads();

        if (c + 1 < nchunks) {
            const int k0 = kb + (c + 1) * BK;
            la.load(A, p.lda, m0, p.m, k0, ke, p.vec_a != 0, tid);
            lb.load(B, p.ldb, n0, p.n, k0, ke, p.vec_b != 0, tid);
        }

        if (mode == kScaled) {
            // Accumulation order is free, so a wave runs its S2 k steps first
            // and its S3 k steps after them; neither loop body branches.
            const uint32_t slow = __builtin_amdgcn_readfirstlane(mask[wave] | mask[NW]) & 0xFFFFu;
            auto s2_step = [&](int kk) {
                uint32_t am[8], mm[8], bb[8];
                lds_frag<LDA>(sA, 0, kk, ty * 4, HM, am);
                lds_frag<LDA>(sA, 1, kk, ty * 4, HM, mm);
                lds_frag<LDB>(sB, 0, kk, tx * 4, HN, bb);
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        acc[i][j] = __builtin_fmaf(__uint_as_float(am[i] + bb[j]), __uint_as_float(mm[i]), acc[i][j]);
            };
            if (slow == 0u) {
#pragma unroll
                for (int kk = 0; kk < BK; ++kk)
                    s2_step(kk);
            } else {
                for (uint32_t todo = ~slow & 0xFFFFu; todo != 0u; todo &= todo - 1u)
                    s2_step(__builtin_ctz(todo));
                for (uint32_t todo = slow; todo != 0u; todo &= todo - 1u) {
                    // S3: the product is rounded (and flushed) before the add.
                    const int kk = __builtin_ctz(todo);
                    uint32_t am[8], mm[8], bb[8];
                    lds_frag<LDA>(sA, 0, kk, ty * 4, HM, am);
                    lds_frag<LDA>(sA, 1, kk, ty * 4, HM, mm);
                    lds_frag<LDB>(sB, 0, kk, tx * 4, HN, bb);
                    s3_accumulate(acc, am, mm, bb);
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
