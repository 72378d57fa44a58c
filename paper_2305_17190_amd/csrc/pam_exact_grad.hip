// Exact-derivative PAM products on gfx950 (Kosson & Jaggi, Table 1).
//
// The exact derivative of A .^ B with respect to A is sgn(B) 2^(E_B + c),
// c = 1{M_A + M_B >= 1}: a power of two, so each backward term is exact.  For
// Y = X .^ W^T the two gradients are contractions in which every term also
// depends on an output-shaped operand through the carry c:
//
//   dX[i,k] = sum_j dY[i,j] d(X[i,k] .^ W[j,k]) / dX[i,k]
//   dW[j,k] = sum_i dY[i,j] d(W[j,k] .^ X[i,k]) / dW[j,k]
//
// Both are C(r, c) = sum_q op(A)(r, q) g(B(q, c), Mod(r, c)) with
// g(b, mod) = sgn(b) 2^(E_b + 1{M_b + M_mod >= 1}) (zero when b or mod is zero
// or denormal): dX is (A = dY, B = W, Mod = X), dW is (A = dY^T, B = X,
// Mod = W).
//
// Per term, with b's encoding staged in LDS (zero and denormal b as 0) and
// mod's mantissa field held in a register per output: t = b + M_mod (one
// int add) carries into b's exponent exactly when M_b + M_mod >= 1, and
// clearing t's mantissa (one and) leaves the float sgn(b) 2^(E_b + c); then
// one fma adds dY * g.  Three full-rate vector ops per term; the product dY *
// g is exact, and the fma adds it unrounded.  Outputs whose Mod is zero or
// denormal are zero.
//
// Tiling follows the PAM matrix product: 128 x 128 output tile per 256-thread
// workgroup, 8 x 8 register micro-tiles, K in LDS chunks of 16; split-K into
// the workspace p.W when several K slices run.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pam_internal.h"
#include "pam_tile.h"

namespace pamk {
namespace {

// Raw operand words into one k-major LDS plane s[kk][o]; with `flush`, zero
// and denormal words become +0 (the B side: such a b has a zero factor).
template <int LDS_LD, int D, int NT, int BK, bool KCONTIG>
__device__ __forceinline__ void store_plane(const TileLoader<D, NT, BK, KCONTIG> &ld, uint32_t (*s)[LDS_LD],
                                            int tid, bool flush) {
    using TL = TileLoader<D, NT, BK, KCONTIG>;
#pragma unroll
    for (int r = 0; r < TL::L; ++r) {
        uint32_t e[4] = {ld.v[r].x, ld.v[r].y, ld.v[r].z, ld.v[r].w};
        if (flush) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                e[c] = ((e[c] & kExpMask) == 0u) ? 0u : e[c];
        }
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
    __shared__ __attribute__((aligned(16))) uint32_t sA[BK][LDA];
    __shared__ __attribute__((aligned(16))) uint32_t sB[BK][LDB];

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

    // The micro-tile's Mod mantissas, fixed for the whole K loop (the
    // epilogue reads Mod again for the zero / denormal test, so no flags stay
    // live through the loop).
    uint32_t mm[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int row = m0 + (i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4));
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int col = n0 + (j < 4 ? tx * 4 + j : HN + tx * 4 + (j - 4));
            uint32_t u = 0u;
            if (row < p.m && col < p.n)
                u = __float_as_uint(p.Mod[(int64_t)row * p.ldm + col]);
            // kept as computed: re-deriving it inside the loop would cost an
            // op per term
            asm volatile("v_and_b32 %0, 0x7fffff, %1" : "=v"(mm[i][j]) : "v"(u));
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
    for (int c = 0; c < nchunks; ++c) {
        __syncthreads();   // every wave is done reading the previous chunk
        store_plane<LDA>(la, sA, tid, false);
        store_plane<LDB>(lb, sB, tid, true);
        __syncthreads();
        if (c + 1 < nchunks) {
            const int k0 = kb + (c + 1) * BK;
            la.load(a_base + (c + 1) * a_step, m0, p.m, k0, ke, vec_a, tid);
            lb.load(b_base + (c + 1) * b_step, n0, p.n, k0, ke, vec_b, tid);
        }
#pragma unroll 1
        for (int kk = 0; kk < BK; ++kk) {
            uint32_t av[8], bv[8];
            const uint4 a_lo = *reinterpret_cast<const uint4 *>(&sA[kk][ty * 4]);
            const uint4 a_hi = *reinterpret_cast<const uint4 *>(&sA[kk][HM + ty * 4]);
            const uint4 b_lo = *reinterpret_cast<const uint4 *>(&sB[kk][tx * 4]);
            const uint4 b_hi = *reinterpret_cast<const uint4 *>(&sB[kk][HN + tx * 4]);
            av[0] = a_lo.x; av[1] = a_lo.y; av[2] = a_lo.z; av[3] = a_lo.w;
            av[4] = a_hi.x; av[5] = a_hi.y; av[6] = a_hi.z; av[7] = a_hi.w;
            bv[0] = b_lo.x; bv[1] = b_lo.y; bv[2] = b_lo.z; bv[3] = b_lo.w;
            bv[4] = b_hi.x; bv[5] = b_hi.y; bv[6] = b_hi.z; bv[7] = b_hi.w;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                exact_row(acc[i], __uint_as_float(av[i]), bv, mm[i]);
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
                const bool zero_mod = (__float_as_uint(mrow[col]) & kExpMask) == 0u;
                orow[col] = zero_mod ? 0.0f : acc[i][j];
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
