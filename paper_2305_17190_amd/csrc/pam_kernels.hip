// HIP kernels for piecewise affine multiplication (PAM) matrix products on
// gfx950.
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
// Encodings written to LDS once per chunk:
//   A element a = (-1)^s 2^E (1 + M):  aM = encoding of 1 + M (exponent
//       field 127, a's mantissa), m = a with its mantissa cleared, i.e.
//       the float +-2^E, or +-0 when a is zero/denormal, and a itself.
//   B element b:  b' = encoding of b minus 0x3F800000 (zero and denormal b
//       are encoded as a signed zero first).
//
//   S1 (per MAC: v_add_u32, v_add_f32): acc += a + b'.  When both exponent
//      fields are in [64, 190] the int32 sum is PAM(a, b)'s encoding itself
//      (Sec. 2.2's addition; the magnitude sum cannot leave the normal range
//      and the carry out of the sign bits leaves their exclusive or), so one
//      float add accumulates it: no multiply at all.
//
//   SCALED form, for the other finite operands: t = aM + b' (one int add) is
//   the encoding of PAM(1 + M, b): adding
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
//   Each wave picks S1, S2 or S3 per k step from bit masks of the operands
//   it will read at that k: S1 unless one has exponent field below 64, S3 if
//   one of those is a normal number ("tiny", field 1..63), S2 otherwise
//   (zeros and denormals only).
//
// SPECIAL: a chunk holding inf, NaN or |x| >= 2^64 is written raw and
// evaluated with the complete per-MAC definition (never taken on finite data
// whose magnitudes stay below 2^64).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "pam_internal.h"
#include "pam_tile.h"

namespace pamk {

// ---------------------------------------------------------------------------
// Tiled PAM matrix product
// ---------------------------------------------------------------------------

// One micro-tile row, S1: acc[j] += a + b'[j] for j < 8.  When a and every
// b[j] have exponent fields in [64, 190], the int32 sum of a's encoding and
// b' = b - bias is the encoding of PAM(a, b) itself: the magnitude sum stays
// within [2^23, 255 * 2^23), so no range check applies, and the carry out of
// the sign bits leaves their exclusive or.  No multiply.
__device__ __forceinline__ void s1_row(float (&acc)[8], uint32_t a, const uint32_t (&bb)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm("v_add_u32 %0, %16, %17\n\t"
        "v_add_u32 %1, %16, %18\n\t"
        "v_add_u32 %2, %16, %19\n\t"
        "v_add_u32 %3, %16, %20\n\t"
        "v_add_u32 %4, %16, %21\n\t"
        "v_add_u32 %5, %16, %22\n\t"
        "v_add_u32 %6, %16, %23\n\t"
        "v_add_u32 %7, %16, %24\n\t"
        "v_add_f32 %8, %8, %0\n\t"
        "v_add_f32 %9, %9, %1\n\t"
        "v_add_f32 %10, %10, %2\n\t"
        "v_add_f32 %11, %11, %3\n\t"
        "v_add_f32 %12, %12, %4\n\t"
        "v_add_f32 %13, %13, %5\n\t"
        "v_add_f32 %14, %14, %6\n\t"
        "v_add_f32 %15, %15, %7"
        : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7),
          "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
          "+v"(acc[7])
        : "v"(a), "v"(bb[0]), "v"(bb[1]), "v"(bb[2]), "v"(bb[3]), "v"(bb[4]), "v"(bb[5]), "v"(bb[6]),
          "v"(bb[7]));
}

// A whole S1 step of the 8 x 8 micro-tile (s1_row for rows 0..7) as one
// instruction sequence: the compiler separates consecutive inline-asm blocks
// with a wait state, which one block per step avoids.
#define PAM_S1_ROW(R, A)                                                                                   \
    "v_add_u32 %[t0], %[" #A "], %[b0]\n\tv_add_u32 %[t1], %[" #A "], %[b1]\n\t"                           \
    "v_add_u32 %[t2], %[" #A "], %[b2]\n\tv_add_u32 %[t3], %[" #A "], %[b3]\n\t"                           \
    "v_add_u32 %[t4], %[" #A "], %[b4]\n\tv_add_u32 %[t5], %[" #A "], %[b5]\n\t"                           \
    "v_add_u32 %[t6], %[" #A "], %[b6]\n\tv_add_u32 %[t7], %[" #A "], %[b7]\n\t"                           \
    "v_add_f32 %[c" #R "0], %[c" #R "0], %[t0]\n\tv_add_f32 %[c" #R "1], %[c" #R "1], %[t1]\n\t"           \
    "v_add_f32 %[c" #R "2], %[c" #R "2], %[t2]\n\tv_add_f32 %[c" #R "3], %[c" #R "3], %[t3]\n\t"           \
    "v_add_f32 %[c" #R "4], %[c" #R "4], %[t4]\n\tv_add_f32 %[c" #R "5], %[c" #R "5], %[t5]\n\t"           \
    "v_add_f32 %[c" #R "6], %[c" #R "6], %[t6]\n\tv_add_f32 %[c" #R "7], %[c" #R "7], %[t7]\n\t"
#define PAM_ACC_ROW(R)                                                                                     \
    [c##R##0] "+v"(acc[R][0]), [c##R##1] "+v"(acc[R][1]), [c##R##2] "+v"(acc[R][2]),                       \
        [c##R##3] "+v"(acc[R][3]), [c##R##4] "+v"(acc[R][4]), [c##R##5] "+v"(acc[R][5]),                   \
        [c##R##6] "+v"(acc[R][6]), [c##R##7] "+v"(acc[R][7])

__device__ __forceinline__ void s1_step(float (&acc)[8][8], const uint4 &al, const uint4 &ah,
                                        const uint32_t (&bb)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm(PAM_S1_ROW(0, a0) PAM_S1_ROW(1, a1) PAM_S1_ROW(2, a2) PAM_S1_ROW(3, a3) PAM_S1_ROW(4, a4)
            PAM_S1_ROW(5, a5) PAM_S1_ROW(6, a6) PAM_S1_ROW(7, a7)
        : PAM_ACC_ROW(0), PAM_ACC_ROW(1), PAM_ACC_ROW(2), PAM_ACC_ROW(3), PAM_ACC_ROW(4), PAM_ACC_ROW(5),
          PAM_ACC_ROW(6), PAM_ACC_ROW(7), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3),
          [t4] "=&v"(t4), [t5] "=&v"(t5), [t6] "=&v"(t6), [t7] "=&v"(t7)
        : [a0] "v"(al.x), [a1] "v"(al.y), [a2] "v"(al.z), [a3] "v"(al.w), [a4] "v"(ah.x), [a5] "v"(ah.y),
          [a6] "v"(ah.z), [a7] "v"(ah.w), [b0] "v"(bb[0]), [b1] "v"(bb[1]), [b2] "v"(bb[2]), [b3] "v"(bb[3]),
          [b4] "v"(bb[4]), [b5] "v"(bb[5]), [b6] "v"(bb[6]), [b7] "v"(bb[7]));
}
#undef PAM_S1_ROW
#undef PAM_ACC_ROW

// One micro-tile row, S2: acc[j] = fma(aM + b'[j], m, acc[j]) for j < 8.
// The eight integer adds are issued before the eight fmas: a SIMD pairs the
// full-rate ops of two waves only when neither wave stalls on the result of
// its previous instruction, which a strict add/fma alternation would do.
__device__ __forceinline__ void s2_row(float (&acc)[8], uint32_t am, uint32_t m, const uint32_t (&bb)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm("v_add_u32 %0, %16, %18\n\t"
        "v_add_u32 %1, %16, %19\n\t"
        "v_add_u32 %2, %16, %20\n\t"
        "v_add_u32 %3, %16, %21\n\t"
        "v_add_u32 %4, %16, %22\n\t"
        "v_add_u32 %5, %16, %23\n\t"
        "v_add_u32 %6, %16, %24\n\t"
        "v_add_u32 %7, %16, %25\n\t"
        "v_fmac_f32 %8, %0, %17\n\t"
        "v_fmac_f32 %9, %1, %17\n\t"
        "v_fmac_f32 %10, %2, %17\n\t"
        "v_fmac_f32 %11, %3, %17\n\t"
        "v_fmac_f32 %12, %4, %17\n\t"
        "v_fmac_f32 %13, %5, %17\n\t"
        "v_fmac_f32 %14, %6, %17\n\t"
        "v_fmac_f32 %15, %7, %17"
        : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7),
          "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
          "+v"(acc[7])
        : "v"(am), "v"(m), "v"(bb[0]), "v"(bb[1]), "v"(bb[2]), "v"(bb[3]), "v"(bb[4]), "v"(bb[5]), "v"(bb[6]),
          "v"(bb[7]));
}

// One micro-tile row, S3: p = (aM + b'[j]) * m rounded on its own (an
// underflowing product is flushed to zero), then acc[j] += p; each of the
// three ops is issued for all eight columns before the next.
__device__ __forceinline__ void s3_row(float (&acc)[8], uint32_t am, uint32_t m, const uint32_t (&bb)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm("v_add_u32 %0, %16, %18\n\t"
        "v_add_u32 %1, %16, %19\n\t"
        "v_add_u32 %2, %16, %20\n\t"
        "v_add_u32 %3, %16, %21\n\t"
        "v_add_u32 %4, %16, %22\n\t"
        "v_add_u32 %5, %16, %23\n\t"
        "v_add_u32 %6, %16, %24\n\t"
        "v_add_u32 %7, %16, %25\n\t"
        "v_mul_f32 %0, %0, %17\n\t"
        "v_mul_f32 %1, %1, %17\n\t"
        "v_mul_f32 %2, %2, %17\n\t"
        "v_mul_f32 %3, %3, %17\n\t"
        "v_mul_f32 %4, %4, %17\n\t"
        "v_mul_f32 %5, %5, %17\n\t"
        "v_mul_f32 %6, %6, %17\n\t"
        "v_mul_f32 %7, %7, %17\n\t"
        "v_add_f32 %8, %8, %0\n\t"
        "v_add_f32 %9, %9, %1\n\t"
        "v_add_f32 %10, %10, %2\n\t"
        "v_add_f32 %11, %11, %3\n\t"
        "v_add_f32 %12, %12, %4\n\t"
        "v_add_f32 %13, %13, %5\n\t"
        "v_add_f32 %14, %14, %6\n\t"
        "v_add_f32 %15, %15, %7"
        : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7),
          "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
          "+v"(acc[7])
        : "v"(am), "v"(m), "v"(bb[0]), "v"(bb[1]), "v"(bb[2]), "v"(bb[3]), "v"(bb[4]), "v"(bb[5]), "v"(bb[6]),
          "v"(bb[7]));
}


// Four outputs to 16-byte aligned memory: the final C with the non-temporal
// hint (written once; streaming it leaves the cache to the operands of the
// work that follows: a w4 step of six alternating products ran 3-5% faster
// in two of three A/B runs, each product alone within 0.7%), split partial
// sums without it (the reduce reads them back soon, mostly from cache).
__device__ __forceinline__ void store_out4(float *p, float a, float b, float c, float d, bool final_c) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 v = {a, b, c, d};
    if (final_c)
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
    else
        *reinterpret_cast<f32x4 *>(p) = v;
}

// Waves each SIMD holds for a tile shape (the register budget per wave is
// 512 / waves): three for the 128 x 128 tile, whose loop fits 168 registers;
// two for the smaller tiles, which stage more operand registers per thread.
constexpr int gemm_waves_per_simd(int bm, int bn, int kw) { return (bm == 128 && bn == 128 && kw == 1) ? 3 : 2; }

// One workgroup computes a BM x BN output tile.  Each of its KW k-groups
// holds the whole tile in 8 x 8 register micro-tiles (BM * BN / 64 threads)
// and takes 16 of the 16 * KW k steps of every LDS chunk; with KW > 1 the
// groups' partial tiles are added through LDS at the end, so small outputs
// get more waves without extra HBM traffic.
template <int BM, int BN, int KW, bool TA, bool TB, typename T>
__global__ void __launch_bounds__(BM * BN / 64 * KW) __attribute__((amdgpu_waves_per_eu(gemm_waves_per_simd(BM, BN, KW))))
pam_gemm_kernel(GemmParams p) {
    constexpr int KPG = kChunkK;           // k steps per group per chunk
    constexpr int BK = KPG * KW;           // chunk depth
    constexpr int NTG = BM * BN / 64;      // threads per k-group
    constexpr int NT = NTG * KW;
    constexpr int NW = NT / 64;
    constexpr int NRW = NTG / 64;          // waves per k-group
    // A k-group's waves form a WR x WC grid, each wave 8 x 8 threads (a
    // 64 x 64 block of outputs when both operands' halves are counted): a
    // k step then reads the fewest operand values per wave, so one zero or
    // tiny value moves as few waves' steps off the two-op path as possible.
    constexpr int WC = BN / 64;            // wave columns
    constexpr int WR = NRW / WC;           // wave rows
    constexpr int NSLOT = WR + WC;         // step-mask words per k-group: one per wave row, one per wave column
    static_assert(WC >= 1 && WR * WC == NRW && BM / 64 == WR, "waves do not tile the output tile");
    constexpr int HM = BM / 2;
    constexpr int HN = BN / 2;
    constexpr int LDA = BM + 4;            // padded LDS rows, 16-byte aligned
    constexpr int LDB = BN + 4;
    constexpr int LDR = BN + 4;            // partial-tile rows (KW > 1)
    static_assert(NTG % 64 == 0, "bad tile shape");

    // The chunk in LDS, and for KW > 1 the partial tiles, which reuse the
    // same bytes after the K loop.
    constexpr int kTileWords = 3 * BK * LDA + BK * LDB;
    constexpr int kRedWords = KW > 1 ? KW * BM * LDR : 0;
    __shared__ __attribute__((aligned(16))) uint32_t smem[kTileWords > kRedWords ? kTileWords : kRedWords];
    __shared__ uint32_t sVote[NW];                 // chunk needs the SPECIAL path
    __shared__ uint32_t sMask[2][KW * NSLOT];      // [chunk parity] low / tiny bits per (group, wave row / wave column)
    uint32_t (*sA)[BK][LDA] = reinterpret_cast<uint32_t (*)[BK][LDA]>(smem);             // plane 0 aM, 1 m, 2 a
    uint32_t (*sB)[BK][LDB] = reinterpret_cast<uint32_t (*)[BK][LDB]>(smem + 3 * BK * LDA);  // b'

    const int tid = threadIdx.x;
    const int grp = tid / NTG;
    const int t = tid % NTG;
    const int wave = tid >> 6;
    const int gwave = t >> 6;              // wave within the k-group
    const int wr = gwave / WC;
    const int wc = gwave % WC;
    const int lane = tid & 63;
    const int tx = wc * 8 + (lane & 7);    // micro-tile column group (of 4, in each half)
    const int ty = wr * 8 + (lane >> 3);   // micro-tile row group
    // Work item -> (tile, K range): whole-K tiles first, then the K slices of
    // the split tiles, slice by slice (neighbouring items share operand rows).
    const uint32_t item = blockIdx.x;
    const bool whole = item < (uint32_t)p.whole;
    const uint32_t rel = item - (uint32_t)p.whole;
    const uint32_t nsplit = (uint32_t)max(p.split_tiles, 1);
    const uint32_t st = whole ? 0u : rel % nsplit;
    const int split = whole ? 0 : (int)(rel / nsplit);
    const uint32_t tile_lin = whole ? item : (uint32_t)p.whole + st;
    const int64_t bz = tile_lin / (uint32_t)p.tiles;
    const int tile = (int)(tile_lin % (uint32_t)p.tiles);
    const int tm = tile / p.tiles_n;
    const int tn = tile % p.tiles_n;
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int kb = whole ? 0 : split * p.k_per_split;
    const int ke = whole ? p.k : min(p.k, kb + p.k_per_split);
    const int nchunks = ke > kb ? (ke - kb + BK - 1) / BK : 0;

    // Chunk bases (uniform): op(A) rows m0.., op(B) columns n0.., at k = kb.
    const T *a_base = reinterpret_cast<const T *>(p.A) + bz * p.strideA +
                      (TA ? (int64_t)kb * p.lda + m0 : (int64_t)m0 * p.lda + kb);
    const T *b_base = reinterpret_cast<const T *>(p.B) + bz * p.strideB +
                      (TB ? (int64_t)n0 * p.ldb + kb : (int64_t)kb * p.ldb + n0);
    const int64_t a_step = TA ? (int64_t)BK * p.lda : BK;
    const int64_t b_step = TB ? BK : (int64_t)BK * p.ldb;
    const bool vec_a = p.vec_a != 0;
    const bool vec_b = p.vec_b != 0;

    TileLoader<BM, NT, BK, !TA, T> la;
    TileLoader<BN, NT, BK, TB, T> lb;
    la.init(p.lda, m0, p.m, tid);
    lb.init(p.ldb, n0, p.n, tid);
    auto a_slot = [](int o) { return ((o % HM) / 4) / 8; };        // wave row reading tile row o
    auto b_slot = [](int o) { return WR + ((o % HN) / 4) / 8; };   // wave column reading tile column o

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = 0.0f;

    if (tid < 2 * KW * NSLOT)
        (&sMask[0][0])[tid] = 0u;

    if (nchunks > 0) {
        la.load(a_base, m0, p.m, kb, ke, vec_a, tid);
        lb.load(b_base, n0, p.n, kb, ke, vec_b, tid);
    }

    const int k_first = grp * KPG;
    for (int c = 0; c < nchunks; ++c) {
        // The chunk's staging runs at a raised wave priority, so that a
        // workgroup reaches its barriers sooner while other workgroups'
        // waves compute (measured +0.3-0.9%); the step loops run at the
        // base priority.
        __builtin_amdgcn_s_setprio(1);
        if (p.round_drop != 0) {
            la.round_mantissa(p.round_drop);
            lb.round_mantissa(p.round_drop);
        }
        const uint32_t fa = la.scan();
        const uint32_t fb = lb.scan();
        const uint64_t sp = __ballot((fa | fb) & 2u);
        uint32_t *mask = sMask[c & 1];
        __syncthreads();   // every wave is done reading the previous chunk (and zeroing this mask)
        la.template store<LDA>(sA, false, tid, fa >> 2, mask, NSLOT, a_slot);
        lb.template store<LDB>(sB, true, tid, fb >> 2, mask, NSLOT, b_slot);
        if ((tid & 63) == 0)
            sVote[wave] = sp ? 1u : 0u;
        __syncthreads();

        uint32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            v |= sVote[w];
        const bool special = v != 0u;
        // Bits 0..15: the wave's k steps with an operand of exponent field
        // below 64; bits 16..31: those among them with a tiny normal one.
        const uint32_t low =
            __builtin_amdgcn_readfirstlane(mask[grp * NSLOT + wr] | mask[grp * NSLOT + WR + wc]);
        if (tid < KW * NSLOT)
            sMask[(c + 1) & 1][tid] = 0u;   // next chunk's masks; last read one chunk ago

        if (c + 1 < nchunks) {
            const int k0 = kb + (c + 1) * BK;
            la.load(a_base + (c + 1) * a_step, m0, p.m, k0, ke, vec_a, tid);
            lb.load(b_base + (c + 1) * b_step, n0, p.n, k0, ke, vec_b, tid);
        }

        __builtin_amdgcn_s_setprio(0);
        const uint32_t (*cA)[BK][LDA] = sA;
        const uint32_t (*cB)[BK][LDB] = sB;
        // The wave's k steps of this chunk as four bit sets, taken by four
        // loops in sequence (accumulation order is free): S1 steps (every
        // operand's exponent field in [64, 190]), S2 steps (zeros or
        // denormals among them, no tiny normals), S3 steps (tiny normals),
        // and for a SPECIAL chunk every step with the complete definition.
        // Loops in sequence, rather than alternative paths, keep the
        // accumulator tile in one set of registers.  The S1 steps, most of
        // them, are unrolled with the next step's reads issued ahead; the
        // rarer S2 / S3 steps read their operands at the start of each step
        // (reading ahead there measured no faster).
        const uint32_t s1_bits = special ? 0u : (~low & 0xFFFFu);
        const uint32_t s2_bits = special ? 0u : (low & ~(low >> 16) & 0xFFFFu);
        const uint32_t s3_bits = special ? 0u : (low >> 16);
        const uint32_t sp_bits = special ? 0xFFFFu : 0u;
        {
            // All 16 steps unrolled: the reads take compile-time offsets from
            // the wave's k-group, the next step's operands are read
            // (unconditionally) while the current one's rows are added, and a
            // uniform branch skips the rows of steps off the two-op path.
            const uint32_t *a_row = &cA[2][k_first][ty * 4];
            const uint32_t *b_row = &cB[0][k_first][tx * 4];
            uint4 al[2], ah[2];
            uint32_t bq[2][8];
            auto rd = [&](int k, int slot) {
                al[slot] = *reinterpret_cast<const uint4 *>(a_row + k * LDA);
                ah[slot] = *reinterpret_cast<const uint4 *>(a_row + k * LDA + HM);
                const uint4 lo = *reinterpret_cast<const uint4 *>(b_row + k * LDB);
                const uint4 hi = *reinterpret_cast<const uint4 *>(b_row + k * LDB + HN);
                bq[slot][0] = lo.x; bq[slot][1] = lo.y; bq[slot][2] = lo.z; bq[slot][3] = lo.w;
                bq[slot][4] = hi.x; bq[slot][5] = hi.y; bq[slot][6] = hi.z; bq[slot][7] = hi.w;
            };
            if (s1_bits != 0u) {
                rd(0, 0);
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    const int cur = k & 1;
                    if (k + 1 < 16)
                        rd(k + 1, cur ^ 1);
                    __builtin_amdgcn_sched_barrier(0);
                    if ((s1_bits >> k) & 1u) {
                        s1_step(acc, al[cur], ah[cur], bq[cur]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        for (uint32_t todo = s2_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = k_first + __builtin_ctz(todo);
            uint32_t am[8], mm[8], bb[8];
            lds_frag<BK, LDA>(cA, 0, kk, ty * 4, HM, am);
            lds_frag<BK, LDA>(cA, 1, kk, ty * 4, HM, mm);
            lds_frag<BK, LDB>(cB, 0, kk, tx * 4, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                s2_row(acc[i], am[i], mm[i], bb);
        }
        for (uint32_t todo = s3_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = k_first + __builtin_ctz(todo);
            uint32_t am[8], mm[8], bb[8];
            lds_frag<BK, LDA>(cA, 0, kk, ty * 4, HM, am);
            lds_frag<BK, LDA>(cA, 1, kk, ty * 4, HM, mm);
            lds_frag<BK, LDB>(cB, 0, kk, tx * 4, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                s3_row(acc[i], am[i], mm[i], bb);
        }
        // SPECIAL: the complete definition per MAC on the operands' own
        // encodings (A: plane 2; B: b' + bias, denormals already zero).
#pragma unroll 1
        for (uint32_t todo = sp_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = k_first + __builtin_ctz(todo);
            uint32_t aa[8], bb[8];
            lds_frag<BK, LDA>(cA, 2, kk, ty * 4, HM, aa);
            lds_frag<BK, LDB>(cB, 0, kk, tx * 4, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] += __uint_as_float(pam_full(aa[i], bb[j] + kBias));
            }
        }
    }

    // Epilogue: the output tile in C, or this K slice's partial tile (packed,
    // written whole: rows and columns past the output are never read).
    float *out;
    int64_t ld;
    int lim_m, lim_n;
    bool vec;
    if (whole) {
        out = p.C + bz * p.strideC + (int64_t)m0 * p.ldc + n0;
        ld = p.ldc;
        lim_m = p.m - m0;
        lim_n = p.n - n0;
        vec = p.vec_c != 0;
    } else {
        out = p.W + ((int64_t)split * p.split_tiles + st) * (BM * BN);
        ld = BN;
        lim_m = BM;
        lim_n = BN;
        vec = true;
    }
    if (KW == 1) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
            if (row >= lim_m)
                continue;
            float *orow = out + (int64_t)row * ld;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int col = h == 0 ? tx * 4 : HN + tx * 4;
                if (vec && col + 3 < lim_n) {
                    store_out4(orow + col, acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3],
                               whole);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (col + j < lim_n)
                            orow[col + j] = acc[i][4 * h + j];
                }
            }
        }
    } else {
        // Every group writes its partial tile over the chunk buffer (after a
        // barrier: other waves may still be reading the last chunk); each
        // thread then adds the KW partials, in group order, for BM * BN / NT
        // outputs.
        __syncthreads();
        float *red = reinterpret_cast<float *>(smem);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int col = h == 0 ? tx * 4 : HN + tx * 4;
                *reinterpret_cast<float4 *>(&red[(grp * BM + row) * LDR + col]) =
                    make_float4(acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3]);
            }
        }
        __syncthreads();
        constexpr int PER = BM * BN / NT;   // outputs per thread, a multiple of 4
        static_assert(PER % 4 == 0 && BN % PER == 0, "bad reduction split");
        const int e0 = tid * PER;
        const int row = e0 / BN;
        const int col0 = e0 % BN;
        if (row < lim_m) {
            float *orow = out + (int64_t)row * ld;
#pragma unroll
            for (int q = 0; q < PER / 4; ++q) {
                const int col = col0 + 4 * q;
                float4 sum = *reinterpret_cast<const float4 *>(&red[row * LDR + col]);
#pragma unroll
                for (int g = 1; g < KW; ++g) {
                    const float4 x = *reinterpret_cast<const float4 *>(&red[(g * BM + row) * LDR + col]);
                    sum.x += x.x;
                    sum.y += x.y;
                    sum.z += x.z;
                    sum.w += x.w;
                }
                if (vec && col + 3 < lim_n) {
                    store_out4(orow + col, sum.x, sum.y, sum.z, sum.w, whole);
                } else {
                    const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (col + j < lim_n)
                            orow[col + j] = sv[j];
                }
            }
        }
    }
}

template <int BM, int BN, int KW, typename T>
static hipError_t launch_tile(bool ta, bool tb, const GemmParams &p, dim3 grid, hipStream_t stream) {
    const dim3 block(BM * BN / 64 * KW);
    if (!ta && !tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, KW, false, false, T>), grid, block, 0, stream, p);
    else if (!ta && tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, KW, false, true, T>), grid, block, 0, stream, p);
    else if (ta && !tb)
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, KW, true, false, T>), grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL((pam_gemm_kernel<BM, BN, KW, true, true, T>), grid, block, 0, stream, p);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_shape(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, const GemmParams &p,
                               dim3 grid, hipStream_t stream) {
    if (tile_m == 128 && tile_n == 128 && kgroups == 1)
        return launch_tile<128, 128, 1, T>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 128 && tile_n == 64 && kgroups == 1)
        return launch_tile<128, 64, 1, T>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 64 && tile_n == 64 && kgroups == 1)
        return launch_tile<64, 64, 1, T>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 64 && tile_n == 64 && kgroups == 4)
        return launch_tile<64, 64, 4, T>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 128 && tile_n == 64 && kgroups == 2)
        return launch_tile<128, 64, 2, T>(trans_a, trans_b, p, grid, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_pam_gemm(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, bool bf16,
                           const GemmParams &p, hipStream_t stream) {
    const int64_t items = (int64_t)p.whole + (int64_t)p.split_tiles * p.splits;
    if (items <= 0 || items > kMaxLaunchItems)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)items);
    if (bf16)
        return launch_shape<uint16_t>(tile_m, tile_n, kgroups, trans_a, trans_b, p, grid, stream);
    // float32 operands: the kernel whose chunks are copied into LDS by the
    // memory pipeline (same results bit for bit).
    return launch_pam_gemm_dma(tile_m, tile_n, kgroups, trans_a, trans_b, p, stream);
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

// Each workgroup adds the K slices of a 256 x 4-output part of one split
// tile (grid-stride over the parts); each thread four consecutive outputs,
// slice by slice.
__global__ void __launch_bounds__(256) split_tile_reduce_kernel(GemmParams p, int bm, int bn) {
    const int gpr = bn / 4;                      // four-output groups per tile row
    const int parts = bm * bn / 4 / 256;         // parts per tile
    const int64_t tile_elems = (int64_t)bm * bn;
    const int64_t slice = (int64_t)p.split_tiles * tile_elems;
    const int64_t nparts = (int64_t)p.split_tiles * parts;
    for (int64_t b = blockIdx.x; b < nparts; b += gridDim.x) {
        const int64_t t = b / parts;
        const int g = (int)(b % parts) * 256 + threadIdx.x;
        const int64_t tile_lin = p.whole + t;
        const int64_t bz = tile_lin / p.tiles;
        const int tile = (int)(tile_lin % p.tiles);
        const int m0 = (tile / p.tiles_n) * bm;
        const int n0 = (tile % p.tiles_n) * bn;
        const int r = g / gpr;
        const int c = (g % gpr) * 4;
        if (m0 + r >= p.m || n0 + c >= p.n)
            continue;
        const float *w = p.W + t * tile_elems + r * bn + c;
        float4 sum = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        // Eight slices' loads in flight before their adds (in slice order):
        // a thread's loads are independent, only the sum is sequential.
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        int q = 0;
        for (; q + 8 <= p.splits; q += 8) {
            f32x4 x[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                x[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(w + (q + u) * slice));
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                sum.x += x[u].x;
                sum.y += x[u].y;
                sum.z += x[u].z;
                sum.w += x[u].w;
            }
        }
        for (; q < p.splits; ++q) {
            const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(w + q * slice));
            sum.x += x.x;
            sum.y += x.y;
            sum.z += x.z;
            sum.w += x.w;
        }
        float *crow = p.C + bz * p.strideC + (int64_t)(m0 + r) * p.ldc + n0;
        if (p.vec_c && n0 + c + 3 < p.n) {
            store_out4(crow + c, sum.x, sum.y, sum.z, sum.w, true);
        } else {
            const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
            for (int j = 0; j < 4; ++j)
                if (n0 + c + j < p.n)
                    crow[c + j] = sv[j];
        }
    }
}

hipError_t launch_split_tile_reduce(int tile_m, int tile_n, const GemmParams &p, hipStream_t stream) {
    if (p.split_tiles <= 0)
        return hipSuccess;
    const int64_t parts = (int64_t)p.split_tiles * (tile_m * tile_n / 4 / 256);
    const int64_t blocks = std::min<int64_t>(parts, 256 * 32);
    hipLaunchKernelGGL(split_tile_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, p, tile_m, tile_n);
    return hipGetLastError();
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

// ---------------------------------------------------------------------------
// Static split-K scratch of pam_gemm_batched_noalloc
// ---------------------------------------------------------------------------

// File-scope device memory: every device the library runs on holds one copy
// until the process ends.  Host code must not pass `scratch` itself to a
// kernel or a copy (on the host it names a stand-in, not device memory): the
// device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 256;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t scratch_address(void **out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        // Once per device, with that device current (hipGetDevice above).
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (ptr == nullptr)
            return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace pamk
