// Exact-derivative PAM products on gfx950 (Kosson & Jaggi, Table 1).
//
// The exact derivative of A .^ B with respect to A is the slope of the
// piecewise affine function: sgn(B) 2^(E_B + c), c = 1{M_A + M_B >= 1}, where
// A .^ B is not clamped, and 0 where it is (a zero or denormal operand, a
// result that underflows to a signed zero or saturates at +-FLT_MAX): the
// function is constant there.  For Y = X .^ W^T the two gradients are
// contractions in which every term also depends on an output-shaped operand:
//
//   dX[i,k] = sum_j dY[i,j] d(X[i,k] .^ W[j,k]) / dX[i,k]
//   dW[j,k] = sum_i dY[i,j] d(W[j,k] .^ X[i,k]) / dW[j,k]
//
// Both are C(r, c) = sum_q op(A)(r, q) g(B(q, c), Mod(r, c)) with g(b, mod) =
// d(mod .^ b) / d mod: dX is (A = dY, B = W, Mod = X), dW is (A = dY^T,
// B = X, Mod = W).  Each term A * g is exact (g is a power of two) and added
// with one rounding (fma); a denormal A counts as zero.
//
// Fast path.  Call a normal value "safe" when its exponent field is in
// [64, 190].  For safe b and safe mod the product mod .^ b can never leave the
// normal range and 2^(E_b + c) <= 2^64, so per term: t = b + M_mod (one int
// add: it carries into b's exponent exactly when M_b + M_mod >= 1), clearing
// t's mantissa (one and) leaves the float sgn(b) 2^(E_b + c), and one fma adds
// A * g.  Zero and denormal b are staged as 0, which gives g = 0.
//
// The rest, taken by the complete definition (general_fma):
//   * b that is normal but not safe ("extreme"): staged as 0 for the fast
//     path, and the LDS chunk's steps holding one are flagged; in a flagged
//     step each thread adds the general term for its columns whose b is
//     extreme.
//   * mod that is normal but not safe: the output's fast-path sum is
//     discarded; the workgroup lists such outputs in LDS (up to 512 of the
//     tile's 16384) and deals them out evenly over its threads, each keeping
//     the sums of at most two, over every k with the general term.  A tile
//     with more takes the general term for every term.
//   * zero / denormal mod: the output is zero.
// The general term needs mod's exponent field, kept for the whole tile in
// LDS as bytes; mod's mantissa stays in registers for the fast path.
//
// Tiling: 128 x 128 output tile per 256-thread workgroup, 8 x 8 register
// micro-tiles, K in LDS chunks of 16; split-K into the workspace p.W when
// several K slices run.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pam_internal.h"
#include "pam_tile.h"

namespace pamk {
namespace {

constexpr uint32_t kSafeLo = 64u;    // exponent fields [64, 190]: the fast path is exact
constexpr uint32_t kSafeHi = 190u;

// Normal (field 1..254; inf / NaN count too) but outside the safe band.
__device__ __forceinline__ bool extreme(uint32_t u) {
    const uint32_t f = (u >> 23) & 0xFFu;
    return f != 0u && (f < kSafeLo || f > kSafeHi);
}

// acc += a * d(mod .^ b)/d mod, the complete definition for finite operands:
// zero when b or mod is zero / denormal or mod .^ b is clamped (magnitude sum
// |b| + |mod| - bias outside [2^-126's, FLT_MAX's encoding]); otherwise
// sgn(b) 2^(E_b + c).  2^128 (E_b = 127 with the carry) is applied as
// (2a) * 2^127 (exact: a doubling).
__device__ __forceinline__ void general_fma(float &acc, float a, uint32_t b, uint32_t mod) {
    const uint32_t mb = b & kMag;
    const uint32_t md = mod & kMag;
    const uint32_t sum = mb + md;   // < 2^32: both magnitudes are below 2^31
    const bool live = mb >= kMinNormal && md >= kMinNormal && sum >= kBias + kMinNormal && sum <= kBias + kFltMax;
    uint32_t g = (b + (md & kMant)) & kSignExp;
    const bool top = (g & kExpMask) == kExpMask;
    g = top ? g - (1u << 23) : g;
    const float a2 = top ? a * 2.0f : a;
    g = live ? g : 0u;
    acc = fmaf(a2, __uint_as_float(g), acc);
}

// Raw operand words into one k-major LDS plane s[kk][o].
template <int LDS_LD, int D, int NT, int BK, bool KCONTIG>
__device__ __forceinline__ void store_a(const TileLoader<D, NT, BK, KCONTIG> &ld, uint32_t (*s)[LDS_LD], int tid) {
    using TL = TileLoader<D, NT, BK, KCONTIG>;
#pragma unroll
    for (int r = 0; r < TL::L; ++r) {
        const uint32_t e[4] = {ld.v[r].x, ld.v[r].y, ld.v[r].z, ld.v[r].w};
        const int o = TL::grp_o(tid, r);
        const int kk = TL::grp_k(tid, r);
        if (KCONTIG) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                s[kk + c][o] = e[c];
        } else {
            *reinterpret_cast<uint4 *>(&s[kk][o]) = make_uint4(e[0], e[1], e[2], e[3]);
        }
    }
}

// B (k-major in memory, rows kk, columns o) into two planes: plane 0 for the
// fast path (zero, denormal and extreme b as 0), plane 1 for the general
// term (zero and denormal b as 0, extreme b kept); a chunk step holding an
// extreme b sets its bit in *slow.
template <int LDS_LD, int D, int NT, int BK>
__device__ __forceinline__ void store_b(const TileLoader<D, NT, BK, false> &ld, uint32_t (*s)[BK][LDS_LD], int tid,
                                        uint32_t *slow) {
    using TL = TileLoader<D, NT, BK, false>;
#pragma unroll
    for (int r = 0; r < TL::L; ++r) {
        const uint32_t e[4] = {ld.v[r].x, ld.v[r].y, ld.v[r].z, ld.v[r].w};
        uint32_t fast[4], full[4];
        bool any = false;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t u = e[c];
            const bool zero = (u & kExpMask) == 0u;
            const bool ext = extreme(u);
            full[c] = zero ? 0u : u;
            fast[c] = (zero || ext) ? 0u : u;
            any = any || ext;
        }
        const int o = TL::grp_o(tid, r);
        const int kk = TL::grp_k(tid, r);
        *reinterpret_cast<uint4 *>(&s[0][kk][o]) = make_uint4(fast[0], fast[1], fast[2], fast[3]);
        *reinterpret_cast<uint4 *>(&s[1][kk][o]) = make_uint4(full[0], full[1], full[2], full[3]);
        if (any)
            atomicOr(slow, 1u << kk);
    }
}

// One micro-tile row: acc[j] += a * ((b[j] + mm[j]) & sign|exponent).
__device__ __forceinline__ void exact_row(float (&acc)[8], float a, const uint32_t (&b)[8], const uint32_t (&mm)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm("v_add_u32 %0, %17, %25\n\t"
        "v_add_u32 %1, %18, %26\n\t"
        "v_add_u32 %2, %19, %27\n\t"
        "v_add_u32 %3, %20, %28\n\t"
        "v_add_u32 %4, %21, %29\n\t"
        "v_add_u32 %5, %22, %30\n\t"
        "v_add_u32 %6, %23, %31\n\t"
        "v_add_u32 %7, %24, %32\n\t"
        "v_and_b32 %0, 0xff800000, %0\n\t"
        "v_and_b32 %1, 0xff800000, %1\n\t"
        "v_and_b32 %2, 0xff800000, %2\n\t"
        "v_and_b32 %3, 0xff800000, %3\n\t"
        "v_and_b32 %4, 0xff800000, %4\n\t"
        "v_and_b32 %5, 0xff800000, %5\n\t"
        "v_and_b32 %6, 0xff800000, %6\n\t"
        "v_and_b32 %7, 0xff800000, %7\n\t"
        "v_fmac_f32 %8, %16, %0\n\t"
        "v_fmac_f32 %9, %16, %1\n\t"
        "v_fmac_f32 %10, %16, %2\n\t"
        "v_fmac_f32 %11, %16, %3\n\t"
        "v_fmac_f32 %12, %16, %4\n\t"
        "v_fmac_f32 %13, %16, %5\n\t"
        "v_fmac_f32 %14, %16, %6\n\t"
        "v_fmac_f32 %15, %16, %7"
        : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7),
          "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
          "+v"(acc[7])
        : "v"(a), "v"(b[0]), "v"(b[1]), "v"(b[2]), "v"(b[3]), "v"(b[4]), "v"(b[5]), "v"(b[6]), "v"(b[7]),
          "v"(mm[0]), "v"(mm[1]), "v"(mm[2]), "v"(mm[3]), "v"(mm[4]), "v"(mm[5]), "v"(mm[6]), "v"(mm[7]));
}

template <bool TA>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
pam_exact_grad_kernel(GemmParams p) {
    constexpr int BM = 128, BN = 128, BK = kChunkK;
    constexpr int NT = 256;
    constexpr int TXN = BN / 8;
    constexpr int HM = BM / 2, HN = BN / 2;
    constexpr int LDA = BM + 4, LDB = BN + 4;
    constexpr int LDE = BN / 4 + 1;   // words per row of the Mod exponent bytes
    __shared__ __attribute__((aligned(16))) uint32_t sA[BK][LDA];
    __shared__ __attribute__((aligned(16))) uint32_t sB[2][BK][LDB];
    constexpr int kListCap = 2 * NT;   // extreme-Mod outputs a tile lists
    __shared__ uint32_t sE[BM][LDE];   // Mod exponent fields, four columns per word
    __shared__ uint32_t sSlow[2];      // [chunk parity] steps holding an extreme b
    __shared__ uint32_t sCount;        // extreme-Mod outputs of the tile
    __shared__ uint32_t sList[2][kListCap];   // their (row << 16 | column) and Mod words

    const int tid = threadIdx.x;
    const int tx = tid % TXN;
    const int ty = tid / TXN;
    const int tm = blockIdx.x / p.tiles_n;
    const int tn = blockIdx.x % p.tiles_n;
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int split = blockIdx.y;
    const int kb = split * p.k_per_split;
    const int ke = min(p.k, kb + p.k_per_split);
    const int nchunks = ke > kb ? (ke - kb + BK - 1) / BK : 0;

    // op(A) rows m0.. and B columns n0.. (B is k-major: B[q * ldb + c]).
    const float *a_base = p.A + (TA ? (int64_t)kb * p.lda + m0 : (int64_t)m0 * p.lda + kb);
    const float *b_base = p.B + (int64_t)kb * p.ldb + n0;
    const int64_t a_step = TA ? (int64_t)BK * p.lda : BK;
    const int64_t b_step = (int64_t)BK * p.ldb;
    const bool vec_a = p.vec_a != 0;
    const bool vec_b = p.vec_b != 0;

    TileLoader<BM, NT, BK, !TA> la;
    TileLoader<BN, NT, BK, false> lb;
    la.init(p.lda, m0, p.m, tid);
    lb.init(p.ldb, n0, p.n, tid);

    if (tid < 2)
        sSlow[tid] = 0u;
    if (tid == 0)
        sCount = 0u;
    __syncthreads();

    // The micro-tile's Mod mantissas, fixed for the whole K loop, and its
    // exponent fields in LDS; outputs with an extreme Mod go to the tile's
    // list.
    uint32_t mm[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int lr = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
        const int row = m0 + lr;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t fields = 0u;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int j = 4 * h + jj;
                const int lc = (h == 0 ? tx * 4 : HN + tx * 4) + jj;
                const int col = n0 + lc;
                uint32_t u = 0u;
                if (row < p.m && col < p.n)
                    u = __float_as_uint(p.Mod[(int64_t)row * p.ldm + col]);
                // kept as computed: re-deriving it inside the loop would cost
                // an op per term
                asm volatile("v_and_b32 %0, 0x7fffff, %1" : "=v"(mm[i][j]) : "v"(u));
                fields |= ((u >> 23) & 0xFFu) << (8 * jj);
                if (extreme(u)) {
                    const uint32_t e = atomicAdd(&sCount, 1u);
                    if (e < (uint32_t)kListCap) {
                        sList[0][e] = ((uint32_t)lr << 16) | (uint32_t)lc;
                        sList[1][e] = u;
                    }
                }
            }
            sE[lr][(h == 0 ? tx : HN / 4 + tx)] = fields;
        }
    }

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = 0.0f;

    if (nchunks > 0) {
        la.load(a_base, m0, p.m, kb, ke, vec_a, tid);
        lb.load(b_base, n0, p.n, kb, ke, vec_b, tid);
    }
    __syncthreads();
    const uint32_t nlist = sCount;
    const bool dense = nlist > (uint32_t)kListCap;
    // This thread's list entries: e = s * NT + slot(tid), slots dealt so that
    // consecutive entries go to different waves.
    const uint32_t slot = (uint32_t)((tid % 64) * (NT / 64) + tid / 64);
    uint32_t side_rc[2], side_mod[2];
    float side_acc[2] = {0.0f, 0.0f};
    bool side_on[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const uint32_t idx = (uint32_t)e * NT + slot;
        side_on[e] = !dense && idx < nlist;
        side_rc[e] = side_on[e] ? sList[0][idx] : 0u;
        side_mod[e] = side_on[e] ? sList[1][idx] : 0u;
    }

    for (int c = 0; c < nchunks; ++c) {
        __syncthreads();   // every wave is done reading the previous chunk
        store_a<LDA>(la, sA, tid);
        store_b<LDB>(lb, sB, tid, &sSlow[c & 1]);
        __syncthreads();
        const uint32_t slow = __builtin_amdgcn_readfirstlane(sSlow[c & 1]);
        if (tid == 0)
            sSlow[(c + 1) & 1] = 0u;   // next chunk's flags; last read one chunk ago
        if (c + 1 < nchunks) {
            const int k0 = kb + (c + 1) * BK;
            la.load(a_base + (c + 1) * a_step, m0, p.m, k0, ke, vec_a, tid);
            lb.load(b_base + (c + 1) * b_step, n0, p.n, k0, ke, vec_b, tid);
        }
        if (!dense) {
#pragma unroll 1
            for (int kk = 0; kk < BK; ++kk) {
                uint32_t av[8], bv[8];
                lds_frag<BK, LDA>(&sA, 0, kk, ty * 4, HM, av);
                lds_frag<BK, LDB>(sB, 0, kk, tx * 4, HN, bv);
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    exact_row(acc[i], __uint_as_float(av[i]), bv, mm[i]);
            }
        }
        // Steps with an extreme b (every step in a dense workgroup): the
        // general term for the columns whose b is extreme (every column).
#pragma unroll 1
        for (uint32_t todo = dense ? 0xFFFFu : slow; todo != 0u; todo &= todo - 1u) {
            const int kk = __builtin_ctz(todo);
            uint32_t av[8], bv[8];
            lds_frag<BK, LDA>(&sA, 0, kk, ty * 4, HM, av);
            lds_frag<BK, LDB>(sB, 1, kk, tx * 4, HN, bv);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (dense || extreme(bv[j])) {
                    const int h = j / 4;
                    const int sh = 8 * (j % 4);
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        const int lr = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
                        const uint32_t f = (sE[lr][(h == 0 ? tx : HN / 4 + tx)] >> sh) & 0xFFu;
                        general_fma(acc[i][j], __uint_as_float(av[i]), bv[j], (f << 23) | mm[i][j]);
                    }
                }
            }
        }
        // Outputs with an extreme Mod, every step.
        if (!dense) {
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                if (side_on[e]) {
                    const int lr = (int)(side_rc[e] >> 16);
                    const int lc = (int)(side_rc[e] & 0xFFFFu);
#pragma unroll 4
                    for (int kk = 0; kk < BK; ++kk)
                        general_fma(side_acc[e], __uint_as_float(sA[kk][lr]), sB[1][kk][lc], side_mod[e]);
                }
            }
        }
    }

    float *out;
    int64_t ld;
    if (p.W != nullptr) {
        out = p.W + (int64_t)split * p.m * p.n;
        ld = p.n;
    } else {
        out = p.C;
        ld = p.ldc;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int row = m0 + (i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4));
        if (row >= p.m)
            continue;
        float *orow = out + (int64_t)row * ld;
        const float *mrow = p.Mod + (int64_t)row * p.ldm;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int col = n0 + (j < 4 ? tx * 4 + j : HN + tx * 4 + (j - 4));
            if (col < p.n) {
                const uint32_t mu = __float_as_uint(mrow[col]);
                const bool zero_mod = (mu & kExpMask) == 0u;
                // extreme-Mod outputs are written by the owner of their list entry
                if (dense || !extreme(mu))
                    orow[col] = zero_mod ? 0.0f : acc[i][j];
            }
        }
    }
    if (!dense) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            if (side_on[e]) {
                const int row = m0 + (int)(side_rc[e] >> 16);
                const int col = n0 + (int)(side_rc[e] & 0xFFFFu);
                if (row < p.m && col < p.n)
                    out[(int64_t)row * ld + col] = side_acc[e];
            }
        }
    }
}

}  // namespace

hipError_t launch_pam_exact_grad(bool trans_a, const GemmParams &p, hipStream_t stream) {
    const int64_t tiles_m = (p.m + 127) / 128;
    const dim3 grid((unsigned)(tiles_m * p.tiles_n), (unsigned)p.splits, 1);
    if (trans_a)
        hipLaunchKernelGGL(pam_exact_grad_kernel<true>, grid, dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(pam_exact_grad_kernel<false>, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace pamk
