// PAM matrix products on gfx950, for float32 and bfloat16 operands.
//
// PAM (Kosson & Jaggi, Sec. 2.2): the product of two float32 numbers is
// replaced by the int32 sum of their encodings minus one exponent bias
// (127 << 23); the sign is the exclusive or of the signs, zero / denormal
// operands and underflowing results give signed zeros, overflowing results
// saturate at +-FLT_MAX, NaN / inf follow IEEE multiplication with a
// canonical quiet NaN.  PAM matrix products (Sec. 3.2) keep float32
// accumulation.
//
// The product is a vector-ALU contraction (PAM is not a product, so the
// matrix cores do not apply).  Each workgroup owns a BM x BN output tile,
// each thread an 8 x 8 register micro-tile, and K advances in LDS chunks of
// 16 steps per k-group.  On gfx950 the integer add and the float32 add, mul
// and fma issue at twice the rate of other vector ops, so the per-MAC work is
// built from those four only.
//
// Encodings in LDS, written once per chunk: A as it is; B as b' = b -
// 0x3F800000 (a denormal b first flushed to its signed zero).
//   S1 (per MAC: v_add_u32, v_add_f32): acc += a + b'.  When both exponent
//      fields are in [64, 190] the int32 sum is PAM(a, b)'s encoding itself
//      (Sec. 2.2's addition; the magnitude sum cannot leave the normal range
//      and the carry out of the sign bits leaves their exclusive or): no
//      multiply at all.
//   SCALED form, for the other finite operands: with aM the encoding of
//   1 + M_A (exponent field 127, a's mantissa) and m = a with its mantissa
//   cleared (the float +-2^E_A, or +-0), t = aM + b' is the encoding of
//   PAM(1 + M_A, b); PAM is exact under power-of-two scaling (Fig. 2: the
//   pattern repeats per octave), so t * m = PAM(a, b) whenever the result is
//   a normal number, the float multiply supplying the sign.  A zero b makes t
//   a denormal encoding, which the float unit (denormals flushed) reads as 0.
//   aM and m are derived per row from A's encoding (two bit operations).
//   S2 (per MAC: v_add_u32, v_fmac_f32): acc = fma(t, m, acc).  Exact when
//      no product underflows: every nonzero operand has exponent field in
//      [64, 190].
//   S3 (per MAC: v_add_u32, v_mul_f32, v_add_f32): p = t * m rounded on its
//      own, so an underflowing product flushes to the signed zero PAM
//      defines; exact for all finite operands with |x| < 2^64.
//   Each wave takes S1, S2 or S3 per k step from bit masks of the operands
//   it reads at that k: S1 unless one has exponent field below 64, S3 if one
//   of those is a normal number ("tiny", field 1..63), S2 otherwise (zeros
//   and denormals only); the S1 steps first, then S2, then S3.
//   SPECIAL: a chunk holding inf, NaN or |x| >= 2^64 takes the complete
//   per-MAC definition (never on finite data below 2^64).
//
// Staging:
//
// * Each chunk's operand pieces (16 bytes: four float32 or eight bfloat16
//   elements consecutive in memory) are copied by the memory pipeline
//   (gfx950's global_load_lds_dwordx4) into an LDS landing buffer.  No
//   register holds a chunk while its copy is in flight, so the kernel keeps
//   only the accumulators and the compute step's operands live across the K
//   loop, and the 128 x 128 tile fits four waves per SIMD.
// * At the chunk boundary each thread re-reads segments of four elements
//   its own wave copied (so no barrier is needed for them), widens bfloat16
//   elements exactly to float32 encodings, scans and encodes them, and writes
//   them k-major into the compute buffer.  A thread holds L rows of one k
//   quad of a K-contiguous operand and writes each k as one L-word store;
//   the lanes of a wave write consecutive columns of one k row, so the
//   stores are free of bank conflicts.  Float32 and bfloat16 operands are
//   staged into the same segments, so a bfloat16 product equals the float32
//   product of its widened operands bit for bit.
// * The chunk after next is copied while a chunk is computed; segments that
//   cannot be copied whole (the K tail, an unaligned operand, a piece
//   straddling the last column) are loaded element by element from global
//   memory when the chunk is encoded.
//
// With k-groups (KW > 1) the groups other than the first write their
// partial tiles to LDS, and the first group adds them in group order and
// stores the tile.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pam_internal.h"
#include "pam_scalar.h"

namespace pamk {

// One 16-byte copy per lane from global memory into LDS: lane i's bytes at
// base + off land at LDS byte address lds_base + IMM + 16 i (the block
// address in M0, the same for the whole wave).  Issued from inline asm, so
// that the compiler does not make later LDS reads of other buffers wait for
// the copy (it cannot tell the landing buffer from the compute buffers of
// the same array); every read of the landing buffer is preceded by an
// explicit wait for the vector-memory counter.  The kernels' compiled code uses M0 for nothing else (no other
// LDS copies, no indexed register moves), so setting it here disturbs no
// value the compiler keeps there.
template <int IMM>
__device__ __forceinline__ void dma_copy16(const char *base, uint32_t off, uint32_t lds_base) {
    // base and lds_base are the same for the whole wave; reading them from
    // the first lane puts them in scalar registers, as the instruction
    // requires.
    const uint2 b = __builtin_bit_cast(uint2, base);
    const uint64_t sb = __builtin_bit_cast(
        uint64_t, make_uint2(__builtin_amdgcn_readfirstlane(b.x), __builtin_amdgcn_readfirstlane(b.y)));
    const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_base);
    // One wait state between the scalar write of M0 and the copy that reads
    // it (the LDS-DMA read-after-SALU-write hazard of this generation).
    asm volatile("s_add_u32 m0, %2, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(sb), "s"(lb), "i"(IMM)
                 : "memory", "m0", "scc");
}

// LDS byte address of an element of a __shared__ array: the low 32 bits of
// its generic address (no null-pointer test as in a cast to the LDS space).
__device__ __forceinline__ uint32_t lds_addr(const uint32_t *p) { return (uint32_t)(uintptr_t)p; }

// One micro-tile row of an S2 or S3 step from A's own encoding a: first
// 1 + M_A (exponent field 127, a's mantissa) and +-2^E_A (a with its mantissa
// cleared, +-0 for zero / denormal a), then the SCALED products with the
// eight b' values.  S2: acc[j] = fma(aM + b'[j], m, acc[j]); S3: the product
// rounded on its own (an underflowing product flushes to zero), then added.
// One asm block per row keeps the derived values' lifetime to the row.
#define PAM_DMA_ROW_OPERANDS                                                                               \
    : [am] "=&v"(am), [m] "=&v"(m), [t0] "=&v"(t0), [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3),       \
      [t4] "=&v"(t4), [t5] "=&v"(t5), [t6] "=&v"(t6), [t7] "=&v"(t7), [c0] "+v"(acc[0]), [c1] "+v"(acc[1]), \
      [c2] "+v"(acc[2]), [c3] "+v"(acc[3]), [c4] "+v"(acc[4]), [c5] "+v"(acc[5]), [c6] "+v"(acc[6]),        \
      [c7] "+v"(acc[7])                                                                                    \
    : [a] "v"(a), [b0] "v"(bb[0]), [b1] "v"(bb[1]), [b2] "v"(bb[2]), [b3] "v"(bb[3]), [b4] "v"(bb[4]),     \
      [b5] "v"(bb[5]), [b6] "v"(bb[6]), [b7] "v"(bb[7]), [mant] "v"(kMant), [bias] "v"(kBias),              \
      [se] "v"(kSignExp)
#define PAM_DMA_ROW_HEAD                                                                                   \
    "v_and_or_b32 %[am], %[a], %[mant], %[bias]\n\tv_and_b32 %[m], %[a], %[se]\n\t"                        \
    "v_add_u32 %[t0], %[am], %[b0]\n\tv_add_u32 %[t1], %[am], %[b1]\n\t"                                   \
    "v_add_u32 %[t2], %[am], %[b2]\n\tv_add_u32 %[t3], %[am], %[b3]\n\t"                                   \
    "v_add_u32 %[t4], %[am], %[b4]\n\tv_add_u32 %[t5], %[am], %[b5]\n\t"                                   \
    "v_add_u32 %[t6], %[am], %[b6]\n\tv_add_u32 %[t7], %[am], %[b7]\n\t"

__device__ __forceinline__ void dma_s2_row(float (&acc)[8], uint32_t a, const uint32_t (&bb)[8]) {
    uint32_t am, m, t0, t1, t2, t3, t4, t5, t6, t7;
    asm(PAM_DMA_ROW_HEAD
        "v_fmac_f32 %[c0], %[t0], %[m]\n\tv_fmac_f32 %[c1], %[t1], %[m]\n\t"
        "v_fmac_f32 %[c2], %[t2], %[m]\n\tv_fmac_f32 %[c3], %[t3], %[m]\n\t"
        "v_fmac_f32 %[c4], %[t4], %[m]\n\tv_fmac_f32 %[c5], %[t5], %[m]\n\t"
        "v_fmac_f32 %[c6], %[t6], %[m]\n\tv_fmac_f32 %[c7], %[t7], %[m]"
        PAM_DMA_ROW_OPERANDS);
}

__device__ __forceinline__ void dma_s3_row(float (&acc)[8], uint32_t a, const uint32_t (&bb)[8]) {
    uint32_t am, m, t0, t1, t2, t3, t4, t5, t6, t7;
    asm(PAM_DMA_ROW_HEAD
        "v_mul_f32 %[t0], %[t0], %[m]\n\tv_mul_f32 %[t1], %[t1], %[m]\n\t"
        "v_mul_f32 %[t2], %[t2], %[m]\n\tv_mul_f32 %[t3], %[t3], %[m]\n\t"
        "v_mul_f32 %[t4], %[t4], %[m]\n\tv_mul_f32 %[t5], %[t5], %[m]\n\t"
        "v_mul_f32 %[t6], %[t6], %[m]\n\tv_mul_f32 %[t7], %[t7], %[m]\n\t"
        "v_add_f32 %[c0], %[c0], %[t0]\n\tv_add_f32 %[c1], %[c1], %[t1]\n\t"
        "v_add_f32 %[c2], %[c2], %[t2]\n\tv_add_f32 %[c3], %[c3], %[t3]\n\t"
        "v_add_f32 %[c4], %[c4], %[t4]\n\tv_add_f32 %[c5], %[c5], %[t5]\n\t"
        "v_add_f32 %[c6], %[c6], %[t6]\n\tv_add_f32 %[c7], %[c7], %[t7]"
        PAM_DMA_ROW_OPERANDS);
}
#undef PAM_DMA_ROW_HEAD
#undef PAM_DMA_ROW_OPERANDS

// A whole S1 step (acc[i][j] += a_i + b'_j for the 8 x 8 micro-tile) as one
// instruction sequence.
#define PAM_DMA_S1_ROW(R, A)                                                                               \
    "v_add_u32 %[t0], %[" #A "], %[b0]\n\tv_add_u32 %[t1], %[" #A "], %[b1]\n\t"                           \
    "v_add_u32 %[t2], %[" #A "], %[b2]\n\tv_add_u32 %[t3], %[" #A "], %[b3]\n\t"                           \
    "v_add_u32 %[t4], %[" #A "], %[b4]\n\tv_add_u32 %[t5], %[" #A "], %[b5]\n\t"                           \
    "v_add_u32 %[t6], %[" #A "], %[b6]\n\tv_add_u32 %[t7], %[" #A "], %[b7]\n\t"                           \
    "v_add_f32 %[c" #R "0], %[c" #R "0], %[t0]\n\tv_add_f32 %[c" #R "1], %[c" #R "1], %[t1]\n\t"           \
    "v_add_f32 %[c" #R "2], %[c" #R "2], %[t2]\n\tv_add_f32 %[c" #R "3], %[c" #R "3], %[t3]\n\t"           \
    "v_add_f32 %[c" #R "4], %[c" #R "4], %[t4]\n\tv_add_f32 %[c" #R "5], %[c" #R "5], %[t5]\n\t"           \
    "v_add_f32 %[c" #R "6], %[c" #R "6], %[t6]\n\tv_add_f32 %[c" #R "7], %[c" #R "7], %[t7]\n\t"
#define PAM_DMA_ACC_ROW(R)                                                                                 \
    [c##R##0] "+v"(acc[R][0]), [c##R##1] "+v"(acc[R][1]), [c##R##2] "+v"(acc[R][2]),                       \
        [c##R##3] "+v"(acc[R][3]), [c##R##4] "+v"(acc[R][4]), [c##R##5] "+v"(acc[R][5]),                   \
        [c##R##6] "+v"(acc[R][6]), [c##R##7] "+v"(acc[R][7])

__device__ __forceinline__ void dma_s1_step(float (&acc)[8][8], const uint4 &al, const uint4 &ah,
                                            const uint32_t (&bb)[8]) {
    uint32_t t0, t1, t2, t3, t4, t5, t6, t7;
    asm(PAM_DMA_S1_ROW(0, a0) PAM_DMA_S1_ROW(1, a1) PAM_DMA_S1_ROW(2, a2) PAM_DMA_S1_ROW(3, a3)
            PAM_DMA_S1_ROW(4, a4) PAM_DMA_S1_ROW(5, a5) PAM_DMA_S1_ROW(6, a6) PAM_DMA_S1_ROW(7, a7)
        : PAM_DMA_ACC_ROW(0), PAM_DMA_ACC_ROW(1), PAM_DMA_ACC_ROW(2), PAM_DMA_ACC_ROW(3), PAM_DMA_ACC_ROW(4),
          PAM_DMA_ACC_ROW(5), PAM_DMA_ACC_ROW(6), PAM_DMA_ACC_ROW(7), [t0] "=&v"(t0), [t1] "=&v"(t1),
          [t2] "=&v"(t2), [t3] "=&v"(t3), [t4] "=&v"(t4), [t5] "=&v"(t5), [t6] "=&v"(t6), [t7] "=&v"(t7)
        : [a0] "v"(al.x), [a1] "v"(al.y), [a2] "v"(al.z), [a3] "v"(al.w), [a4] "v"(ah.x), [a5] "v"(ah.y),
          [a6] "v"(ah.z), [a7] "v"(ah.w), [b0] "v"(bb[0]), [b1] "v"(bb[1]), [b2] "v"(bb[2]), [b3] "v"(bb[3]),
          [b4] "v"(bb[4]), [b5] "v"(bb[5]), [b6] "v"(bb[6]), [b7] "v"(bb[7]));
}
#undef PAM_DMA_S1_ROW
#undef PAM_DMA_ACC_ROW

// Eight values of one k row of a compute buffer: four at p, four at p + half.
__device__ __forceinline__ void dma_frag(const uint32_t *p, int half, uint32_t (&out)[8]) {
    const uint4 lo = *reinterpret_cast<const uint4 *>(p);
    const uint4 hi = *reinterpret_cast<const uint4 *>(p + half);
    out[0] = lo.x; out[1] = lo.y; out[2] = lo.z; out[3] = lo.w;
    out[4] = hi.x; out[5] = hi.y; out[6] = hi.z; out[7] = hi.w;
}

// One operand's D x BK chunk (D = rows of op(A) or columns of op(B)) in
// segments of four elements consecutive in memory; T is the operand's
// element type (float or bfloat16 bits).
//
// KCONTIG: a segment is (row o, k quad).  Thread t stages the L rows
// j * L .. j * L + L - 1 of one k quad kq, so that it can write each k of them
// as one L-word LDS store.  Lane 16 * q + i of a wave takes row group
// j = 16 * (wave / (BK / 16)) + i and k quad kq = q + 4 * (wave % (BK / 16)):
// with float32 operands, one copy instruction reads 16 rows x 64 contiguous
// bytes (16 cache lines), and the 16 lanes of each store pass write 16
// consecutive row groups of one k row (no bank conflicts).
//
// Otherwise a segment is (k, column quad); thread t's segment r is number
// t + r * NT, so consecutive lanes hold consecutive column quads of one k.
template <int D, int BK, int NT, bool KCONTIG, typename T>
struct DmaTile {
    static constexpr int SEGS = D * BK / 4;
    static constexpr int L = SEGS / NT;                  // segments per thread
    static constexpr int G = D / L;                      // KCONTIG: row groups
    static constexpr int KS = BK / 16;                   // KCONTIG: waves per 16 row groups
    static constexpr int NW = NT / 64;
    static constexpr bool kWide = sizeof(T) == 4;        // float32 operands; else bfloat16
    static constexpr int EPC = 16 / (int)sizeof(T);      // elements per 16-byte copy
    static constexpr int CL = D * BK / EPC / NT;         // copies per thread
    static_assert(L * NT == SEGS && (L == 2 || L == 4), "chunk does not divide over the threads");
    static_assert(CL * EPC * NT == D * BK && CL >= 1, "chunk copies do not divide over the threads");
    static_assert(!KCONTIG || (G % 16 == 0 && BK % 16 == 0 && (G / 16) * KS == NW), "bad K-contiguous segment split");

    uint4 v[L];          // the segments being encoded (live only at the chunk boundary)

    static __device__ __forceinline__ int seg_o(int t, int r) {
        return KCONTIG ? (16 * ((t >> 6) / KS) + (t & 15)) * L + r : ((t + r * NT) % (D / 4)) * 4;
    }
    static __device__ __forceinline__ int seg_k(int t, int r) {
        return KCONTIG ? (((t & 63) >> 4) + 4 * ((t >> 6) % KS)) * 4 : (t + r * NT) / (D / 4);
    }

    // Copies.  A float32 copy is one segment (seg_o / seg_k).  A bfloat16
    // copy is eight elements consecutive in memory, and a wave copies exactly
    // the elements its own lanes stage (so that, after its own wait for the
    // copies, it reads no other wave's): copy r of lane i takes q = i + 64 r
    // of the wave's pieces.  K-contiguous: the wave stages 16 L rows x 16 k
    // (row groups 16 (w / KS) + 0..15, k quads 4 (w % KS) + 0..3), piece q is
    // row q / 2 of them, k octet q % 2.  Otherwise the wave's segments r' =
    // 0..L-1 are 64 consecutive column quads each (from quad 64 w + r' NT of
    // the k-major order), piece q is octet q % 32 of run q / 32.  Either way
    // consecutive lanes read consecutive 16-byte pieces of the operand.
    static __device__ __forceinline__ int copy_o(int t, int r) {
        if constexpr (kWide)
            return seg_o(t, r);
        const int q = (t & 63) + 64 * r;
        if (KCONTIG)
            return 16 * L * ((t >> 6) / KS) + q / 2;
        return (((64 * (t >> 6) + (q / 32) * NT) / 2 + q % 32) % (D / 8)) * 8;
    }
    static __device__ __forceinline__ int copy_k(int t, int r) {
        if constexpr (kWide)
            return seg_k(t, r);
        const int q = (t & 63) + 64 * r;
        if (KCONTIG)
            return 16 * ((t >> 6) % KS) + 8 * (q & 1);
        return ((64 * (t >> 6) + (q / 32) * NT) / 2 + q % 32) / (D / 8);
    }

    // Byte offset of copy r from its chunk's base.  Rows past o_lim are
    // clamped to the last valid row (their outputs are discarded); a copy
    // straddling the last valid column is not made (copyable) and its
    // segments are loaded element by element.  In builds for three or four
    // waves per SIMD recomputed per chunk from the thread index, so that no
    // per-thread offsets stay live across the K loop.  The leading dimension
    // is below 2^22 elements (the library rejects larger ones), so its bytes
    // and the row or k index fit a 24-bit multiply.
    static __device__ __forceinline__ uint32_t boff(int tid, int r, int64_t ld, int o0, int o_lim) {
        const int o = copy_o(tid, r);
        const int kk = copy_k(tid, r);
        const uint32_t es = (uint32_t)sizeof(T);
        const uint32_t ldb = (uint32_t)ld * es;
        if (KCONTIG)
            return __umul24((uint32_t)min(o, o_lim - 1 - o0), ldb) + (uint32_t)kk * es;
        return __umul24((uint32_t)kk, ldb) + (uint32_t)o * es;
    }
    static __device__ __forceinline__ bool copyable(int tid, int r, int o0, int o_lim) {
        return KCONTIG || o0 + copy_o(tid, r) + EPC - 1 < o_lim;
    }
    // Every copy of the tile is made (the same for the whole workgroup): the
    // tile lies inside the operand, or it is K-contiguous.
    static __device__ __forceinline__ bool all_copyable(int o0, int o_lim) { return KCONTIG || o0 + D <= o_lim; }

    // Start copying the chunk at `base` into the landing buffer at byte
    // RAW_OFF of the LDS array; lds_w is the LDS byte address of that array
    // plus 1024 per wave index, so that copy r of wave w lands in block
    // (r * NW + w) at lds_w + RAW_OFF + r * NW * 1024 (16 bytes per lane).
    // Called only for an interior chunk of an aligned operand.
    template <int RAW_OFF, int R>
    static __device__ __forceinline__ void copy_seg(const char *cb, uint32_t lds_w, int tid, int64_t ld, int o0,
                                                    int o_lim) {
        dma_copy16<RAW_OFF + R * NW * 1024>(cb, boff(tid, R, ld, o0, o_lim), lds_w);
    }
    template <int RAW_OFF>
    static __device__ __forceinline__ void copy(const T *__restrict__ base, uint32_t lds_w, int tid, int64_t ld,
                                                int o0, int o_lim) {
        const char *cb = reinterpret_cast<const char *>(base);
        static_assert(CL == 1 || CL == 2 || CL == 4, "copies per thread");
        if (all_copyable(o0, o_lim)) {
            copy_seg<RAW_OFF, 0>(cb, lds_w, tid, ld, o0, o_lim);
            if constexpr (CL >= 2)
                copy_seg<RAW_OFF, 1>(cb, lds_w, tid, ld, o0, o_lim);
            if constexpr (CL == 4) {
                copy_seg<RAW_OFF, 2>(cb, lds_w, tid, ld, o0, o_lim);
                copy_seg<RAW_OFF, 3>(cb, lds_w, tid, ld, o0, o_lim);
            }
            return;
        }
        if (copyable(tid, 0, o0, o_lim))
            copy_seg<RAW_OFF, 0>(cb, lds_w, tid, ld, o0, o_lim);
        if constexpr (CL >= 2) {
            if (copyable(tid, 1, o0, o_lim))
                copy_seg<RAW_OFF, 1>(cb, lds_w, tid, ld, o0, o_lim);
        }
        if constexpr (CL == 4) {
            if (copyable(tid, 2, o0, o_lim))
                copy_seg<RAW_OFF, 2>(cb, lds_w, tid, ld, o0, o_lim);
            if (copyable(tid, 3, o0, o_lim))
                copy_seg<RAW_OFF, 3>(cb, lds_w, tid, ld, o0, o_lim);
        }
    }

    // Where segment r of this thread (wave w, lane) sits in the landing
    // buffer: the word offset of its 16 (float32) or 8 (bfloat16) bytes.  A
    // float32 segment is the lane's own copy r (block r * NW + w); a bfloat16
    // segment is half of the copy of its eight elements, made by a lane of
    // the same wave.
    static __device__ __forceinline__ uint32_t slot_of(int w, int lane, int r) {
        if constexpr (kWide)
            return (uint32_t)((r * NW + w) * 256 + lane * 4);
        const int q = KCONTIG ? ((lane & 15) * L + r) * 2 + (lane >> 5) : r * 32 + lane / 2;
        const int half = KCONTIG ? (lane >> 4) & 1 : lane & 1;
        return (uint32_t)(((q / 64) * NW + w) * 256 + (q % 64) * 4 + half * 2);
    }
    // Whether the copy holding segment r was made (see copyable).
    static __device__ __forceinline__ bool seg_copied(int tid, int r, int o0, int o_lim) {
        if constexpr (kWide)
            return copyable(tid, r, o0, o_lim);
        return KCONTIG || o0 + (seg_o(tid, r) & ~7) + 7 < o_lim;
    }
    // Reads through an LDS-space pointer: the compiler then cannot merge a
    // landing-buffer read with the element-by-element global loads of the
    // other branch into one generic (flat) load.
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    typedef __attribute__((address_space(3))) const u32x4 lds_u32x4;
    typedef __attribute__((address_space(3))) const u32x2 lds_u32x2;
    static __device__ __forceinline__ uint4 read_slot(const uint32_t *raw, uint32_t off) {
        if constexpr (kWide) {
            const u32x4 x = *(lds_u32x4 *)(raw + off);
            return make_uint4(x[0], x[1], x[2], x[3]);
        }
        const u32x2 y = *(lds_u32x2 *)(raw + off);
        const uint2 d = make_uint2(y[0], y[1]);
        // Four bfloat16 elements widened exactly to float32 encodings.
        return make_uint4(d.x << 16, d.x & 0xFFFF0000u, d.y << 16, d.y & 0xFFFF0000u);
    }

    // The thread's segments of chunk [k0, k0 + BK): from the landing buffer
    // when they were copied, else element by element from global memory
    // (elements at k >= k_lim are zero).
    __device__ __forceinline__ void fetch(const uint32_t *raw, int w, int lane, bool copied,
                                          const T *__restrict__ base, int64_t ld, int o0, int o_lim, int k0,
                                          int k_lim, int tid) {
        if (copied && all_copyable(o0, o_lim)) {
            // The common case, one branch for all segments: the reads issue
            // back to back and are waited for once.
#pragma unroll
            for (int r = 0; r < L; ++r)
                v[r] = read_slot(raw, slot_of(w, lane, r));
            return;
        }
#pragma unroll
        for (int r = 0; r < L; ++r) {
            if (copied && seg_copied(tid, r, o0, o_lim))
                v[r] = read_slot(raw, slot_of(w, lane, r));
            else
                v[r] = load_elements(base, r, ld, o0, o_lim, k0, k_lim, tid);
        }
    }

    static __device__ __forceinline__ uint32_t widen(float x) { return __float_as_uint(x); }
    static __device__ __forceinline__ uint32_t widen(uint16_t h) { return (uint32_t)h << 16; }

    static __device__ __forceinline__ uint4 load_elements(const T *base, int r, int64_t ld, int o0, int o_lim, int k0,
                                                          int k_lim, int tid) {
        const int o = seg_o(tid, r);
        const int kk = seg_k(tid, r);
        uint32_t e[4];
        if (KCONTIG) {
            // (a float32 segment is its own copy: boff is its offset)
            const T *src = kWide ? reinterpret_cast<const T *>(reinterpret_cast<const char *>(base) +
                                                               boff(tid, r, ld, o0, o_lim))
                                 : base + (int64_t)(min(o0 + o, o_lim - 1) - o0) * ld + kk;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                e[c] = (k0 + kk + c < k_lim) ? widen(src[c]) : 0u;
        } else {
            const T *row = kWide ? reinterpret_cast<const T *>(reinterpret_cast<const char *>(base) +
                                                               boff(tid, r, ld, o0, o_lim)) - o
                                 : base + (int64_t)kk * ld;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                e[c] = (k0 + kk < k_lim) ? widen(row[min(o0 + o + c, o_lim - 1) - o0]) : 0u;
        }
        return make_uint4(e[0], e[1], e[2], e[3]);
    }

    // Round every held element to 23 - drop mantissa bits, nearest even (inf
    // and NaN unchanged).
    __device__ __forceinline__ void round_mantissa(int drop) {
        const uint32_t low = (1u << drop) - 1u;
        const uint32_t half_m1 = low >> 1;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t u = e[c];
                const uint32_t rounded = (u + half_m1 + ((u >> drop) & 1u)) & ~low;
                e[c] = ((u & kExpMask) == kExpMask) ? u : rounded;
            }
            v[r] = make_uint4(e[0], e[1], e[2], e[3]);
        }
    }

    // One pass over the held elements with the exponent field moved to the
    // top byte and the sign dropped (x << 1): per segment r the least such
    // value (below 64 << 24 iff the segment holds an element below the S1
    // range: a zero, denormal or |x| < 2^-63), and the largest over all
    // elements, returned (at least 191 << 24 iff one needs the SPECIAL
    // path: |x| >= 2^64, inf, NaN).
    __device__ __forceinline__ uint32_t scan(uint32_t (&smin)[L]) const {
        uint32_t mx = 0;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const uint32_t j0 = v[r].x << 1, j1 = v[r].y << 1, j2 = v[r].z << 1, j3 = v[r].w << 1;
            smin[r] = min(min(j0, j1), min(j2, j3));
            mx = max(mx, max(max(j0, j1), max(j2, j3)));
        }
        return mx;
    }
    static __device__ __forceinline__ bool low_seg(uint32_t smin) { return smin < (64u << 24); }

    // A denormal element to its signed zero (multiplying by 1.0 flushes it;
    // NaN stays NaN).  Needed for B only, and only where scan() found an
    // element below the S1 range.
    __device__ __forceinline__ void flush_denormals() {
#pragma unroll
        for (int r = 0; r < L; ++r) {
            uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int c = 0; c < 4; ++c)
                asm("v_mul_f32 %0, 1.0, %1" : "=v"(e[c]) : "v"(e[c]));
            v[r] = make_uint4(e[0], e[1], e[2], e[3]);
        }
    }

    // Element encodings: A as it is; B as b' = b - bias (denormals already
    // flushed).
    static __device__ __forceinline__ uint32_t enc(uint32_t u, bool is_b) { return is_b ? u - kBias : u; }

    // Write the encoded chunk k-major into s[k * D + o] and mark the step
    // masks: bit k % KPG of the word of k-group k / KPG.
    template <int KPG, typename SlotOf>
    __device__ __forceinline__ void store(uint32_t *s, bool is_b, int tid, const uint32_t (&smin)[L], uint32_t *mask,
                                          int slots, SlotOf slot_of) const {
        if (KCONTIG) {
            // One address; the four k rows at constant offsets from it.
            uint32_t *const row0 = s + seg_k(tid, 0) * D + seg_o(tid, 0);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uint32_t w[L];
#pragma unroll
                for (int r = 0; r < L; ++r) {
                    const uint32_t u = c == 0 ? v[r].x : c == 1 ? v[r].y : c == 2 ? v[r].z : v[r].w;
                    w[r] = enc(u, is_b);
                }
                uint32_t *dst = row0 + c * D;
                if constexpr (L == 2)
                    *reinterpret_cast<uint2 *>(dst) = make_uint2(w[0], w[1]);
                else
                    *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
            }
        } else {
#pragma unroll
            for (int r = 0; r < L; ++r) {
                const int o = seg_o(tid, r);
                const int kk = seg_k(tid, r);
                *reinterpret_cast<uint4 *>(s + kk * D + o) =
                    make_uint4(enc(v[r].x, is_b), enc(v[r].y, is_b), enc(v[r].z, is_b), enc(v[r].w, is_b));
            }
        }
#pragma unroll
        for (int r = 0; r < L; ++r) {
            // Rare: the wave skips this unless one of its lanes holds such an
            // element in segment r.
            if (low_seg(smin[r])) {
                const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
                const int o = seg_o(tid, r);
                const int kk = seg_k(tid, r);
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t ex = e[c] & kExpMask;
                    if (ex < (64u << 23)) {
                        const int k = KCONTIG ? kk + c : kk;
                        const uint32_t bit = 1u << (k % KPG);
                        atomicOr(&mask[(k / KPG) * slots + slot_of(KCONTIG ? o : o + c)],
                                 ex != 0u ? (bit | (bit << 16)) : bit);
                    }
                }
            }
        }
    }
};

// Waves per SIMD the tile is compiled for (registers per wave 512 / waves),
// matching what its LDS footprint allows on a 160 KB compute unit.
constexpr int dma_waves_per_simd(int bm, int bn, int kw) {
    return (bm == 128 && bn == 128 && kw == 1) ? 4 : (bm == 128 && bn == 64 && kw == 2) ? 3 : 2;
}

// k steps per k-group per LDS chunk: the same for every tile shape (the
// step masks hold one bit per step of a chunk in each half of a 32-bit word).
constexpr int dma_kpg(int, int, int) { return kChunkK; }

// Minimum LDS words per workgroup.  Workgroups of one or two waves can be
// placed unevenly on a compute unit's four SIMDs when more fit than the
// launch fills (measured: one workgroup in a launch with three waves on a
// SIMD ran 1.4x as long as the others).  Their LDS is padded so that no more
// than two waves per SIMD fit: four 128 x 64 or eight 64 x 64 workgroups.
// The 128 x 64 two-group tile built for two waves per SIMD is padded to two
// workgroups per compute unit for the same reason.
constexpr int dma_min_lds_words(int bm, int bn, int kw, int wps) {
    return (bm == 128 && bn == 64 && kw == 1)   ? (33 << 10) / 4
           : (bm == 64 && bn == 64 && kw == 1)  ? (18 << 10) / 4
           : (bm == 128 && bn == 64 && kw == 2 && wps == 2) ? (54 << 10) / 4
                                                           : 0;
}

// WPS: waves per SIMD the kernel is compiled for.  At two (256 registers a
// wave), and at three for a row-major A (168 registers, measured to fit), the
// per-thread staging addresses are computed once, before the K loop;
// otherwise they are recomputed per chunk, since registers held across the
// loop would not fit beside the accumulators.
template <int BM, int BN, int KW, bool TA, bool TB, int WPS, typename T>
__global__ void __launch_bounds__(BM * BN / 64 * KW) __attribute__((amdgpu_waves_per_eu(WPS)))
pam_gemm_dma_kernel(GemmParams p) {
    constexpr bool kKeepAddresses = WPS <= 2 || (WPS == 3 && !TA);
    constexpr int KPG = dma_kpg(BM, BN, KW);   // k steps per group per chunk
    constexpr int BK = KPG * KW;
    constexpr int NTG = BM * BN / 64;
    constexpr int NT = NTG * KW;
    constexpr int NRW = NTG / 64;
    constexpr int WC = BN / 64;
    constexpr int WR = NRW / WC;
    constexpr int NSLOT = WR + WC;
    static_assert(WC >= 1 && WR * WC == NRW && BM / 64 == WR, "waves do not tile the output tile");
    constexpr int HM = BM / 2;
    constexpr int HN = BN / 2;
    constexpr int LDR = BN;                // partial-tile rows (KW > 1)
    using TileA = DmaTile<BM, BK, NT, !TA, T>;
    using TileB = DmaTile<BN, BK, NT, TB, T>;
    constexpr int kRawA = TileA::CL * NT * 4;   // 16 bytes per copy
    constexpr int kRawB = TileB::CL * NT * 4;
    constexpr int kStage = kRawA + kRawB + BK * BM + BK * BN;
    // Partial tiles held at once by the LDS after the K loop (KW > 1).
    constexpr int kRedTiles = KW == 1 ? 0 : (kStage / (BM * LDR) >= KW - 1 ? KW - 1 : kStage / (BM * LDR));
    static_assert(KW == 1 || kRedTiles >= 1, "no room for a partial tile");
    constexpr int kRed = kRedTiles * BM * LDR;
    // Landing buffers, then the k-major compute buffers; for KW > 1 the
    // partial tiles reuse the same bytes after the K loop.
    constexpr int kWords0 = kStage > kRed ? kStage : kRed;
    constexpr int kMinWords = dma_min_lds_words(BM, BN, KW, WPS);
    __shared__ __attribute__((aligned(16))) uint32_t smem[kWords0 > kMinWords ? kWords0 : kMinWords];
    // Step masks of the two chunks in flight (k-group g's slot words at
    // g * NSLOT), and after them the chunk's SPECIAL vote.
    __shared__ uint32_t sMask[2][KW * NSLOT + 1];
    static_assert(2 * (KW * NSLOT + 1) <= NT, "the mask words are cleared one per thread");
    uint32_t *rawA = smem;
    uint32_t *rawB = smem + kRawA;
    uint32_t *encA = smem + kRawA + kRawB;
    uint32_t *encB = encA + BK * BM;

    const int tid = threadIdx.x;
    const int grp = tid / NTG;
    const int t = tid % NTG;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds_w = __builtin_amdgcn_readfirstlane(lds_addr(smem) + (uint32_t)wave * 1024u);
    const int gwave = t >> 6;
    const int wr = gwave / WC;
    const int wc = gwave % WC;
    const int lane = tid & 63;
    const int tx = wc * 8 + (lane & 7);
    const int ty = wr * 8 + (lane >> 3);
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

    const T *a_base = reinterpret_cast<const T *>(p.A) + bz * p.strideA +
                      (TA ? (int64_t)kb * p.lda + m0 : (int64_t)m0 * p.lda + kb);
    const T *b_base = reinterpret_cast<const T *>(p.B) + bz * p.strideB +
                      (TB ? (int64_t)n0 * p.ldb + kb : (int64_t)kb * p.ldb + n0);
    const int64_t a_step = TA ? (int64_t)BK * p.lda : BK;
    const int64_t b_step = TB ? BK : (int64_t)BK * p.ldb;
    const bool vec_a = p.vec_a != 0;
    const bool vec_b = p.vec_b != 0;
    // The launch's flags as one scalar word, tested afresh in each chunk
    // (kept as three lane masks across the loop they took six scalar
    // registers, spilled).
    const uint32_t flags = (vec_a ? 1u : 0u) | (vec_b ? 2u : 0u) | (p.round_drop != 0 ? 4u : 0u);

    TileA la;
    TileB lb;
    auto a_slot = [](int o) { return (int)(((uint32_t)o % HM) / 32u); };
    auto b_slot = [](int o) { return WR + (int)(((uint32_t)o % HN) / 32u); };

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[i][j] = 0.0f;

    if (tid < 2 * (KW * NSLOT + 1))
        (&sMask[0][0])[tid] = 0u;

    // Chunk c is copied when it is whole (k0 + BK <= ke) and its operand
    // aligned.
    if (nchunks > 0 && kb + BK <= ke) {
        if (vec_a)
            TileA::template copy<0>(a_base, lds_w, tid, p.lda, m0, p.m);
        if (vec_b)
            TileB::template copy<kRawA * 4>(b_base, lds_w, tid, p.ldb, n0, p.n);
    }

    const int k_first = grp * KPG;
    for (int c = 0; c < nchunks; ++c) {
        const int k0 = kb + c * BK;
        const bool interior = k0 + BK <= ke;
        uint32_t fl = __builtin_amdgcn_readfirstlane(flags);
        asm volatile("" : "+s"(fl));
        // The thread index through an empty asm: staging addresses derived
        // from it are recomputed per chunk instead of being hoisted out of
        // the loop into registers that would stay live during the steps.
        int tid_c = tid;
        if constexpr (!kKeepAddresses)
            asm volatile("" : "+v"(tid_c));
        __builtin_amdgcn_s_setprio(1);
        // This thread's copies of chunk c have landed (the only vector-memory
        // operations outstanding).
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        la.fetch(rawA, wave, tid_c & 63, interior && (fl & 1u), a_base + c * a_step, p.lda, m0, p.m, k0, ke, tid_c);
        lb.fetch(rawB, wave, tid_c & 63, interior && (fl & 2u), b_base + c * b_step, p.ldb, n0, p.n, k0, ke, tid_c);

        if (fl & 4u) {
            la.round_mantissa(p.round_drop);
            lb.round_mantissa(p.round_drop);
        }
        uint32_t smin_a[TileA::L], smin_b[TileB::L];
        const uint32_t mx = max(la.scan(smin_a), lb.scan(smin_b));
        uint32_t low_b = smin_b[0];
#pragma unroll
        for (int r = 1; r < TileB::L; ++r)
            low_b = min(low_b, smin_b[r]);
        if (TileB::low_seg(low_b))   // rare per thread: B's denormals to zero
            lb.flush_denormals();
        uint32_t *mask = sMask[c & 1];
        __syncthreads();   // every wave is done reading the previous chunk (and zeroing this mask)
        la.template store<KPG>(encA, false, tid_c, smin_a, mask, NSLOT, a_slot);
        lb.template store<KPG>(encB, true, tid_c, smin_b, mask, NSLOT, b_slot);
        // The workgroup's SPECIAL vote: one more mask word.
        if (mx >= (191u << 24))
            atomicOr(&mask[KW * NSLOT], 1u);
        __syncthreads();

        const bool special = __builtin_amdgcn_readfirstlane(mask[KW * NSLOT]) != 0u;
        const uint32_t low =
            __builtin_amdgcn_readfirstlane(mask[grp * NSLOT + wr] | mask[grp * NSLOT + WR + wc]);
        if (tid < KW * NSLOT + 1)
            (&sMask[0][0])[(((uint32_t)c + 1u) & 1u) * (KW * NSLOT + 1) + (uint32_t)tid] = 0u;

        // The next chunk's copies land while this one is computed (the
        // landing slots are this thread's own and were read above).
        if (c + 1 < nchunks && k0 + 2 * BK <= ke) {
            if (fl & 1u)
                TileA::template copy<0>(a_base + (c + 1) * a_step, lds_w, tid_c, p.lda, m0, p.m);
            if (fl & 2u)
                TileB::template copy<kRawA * 4>(b_base + (c + 1) * b_step, lds_w, tid_c, p.ldb, n0, p.n);
        }

        __builtin_amdgcn_s_setprio(0);

        constexpr uint32_t kStepMask = (1u << KPG) - 1u;
        const uint32_t s1_bits = special ? 0u : (~low & kStepMask);
        const uint32_t s2_bits = special ? 0u : (low & ~(low >> 16) & kStepMask);
        const uint32_t s3_bits = special ? 0u : (low >> 16);
        const uint32_t sp_bits = special ? kStepMask : 0u;
        const uint32_t *a_row = encA + k_first * BM + ty * 4;
        const uint32_t *b_row = encB + k_first * BN + tx * 4;
        {
            uint4 al[2], ah[2];
            uint32_t bq[2][8];
            auto rd = [&](int k, int slot) {
                al[slot] = *reinterpret_cast<const uint4 *>(a_row + k * BM);
                ah[slot] = *reinterpret_cast<const uint4 *>(a_row + k * BM + HM);
                const uint4 lo = *reinterpret_cast<const uint4 *>(b_row + k * BN);
                const uint4 hi = *reinterpret_cast<const uint4 *>(b_row + k * BN + HN);
                bq[slot][0] = lo.x; bq[slot][1] = lo.y; bq[slot][2] = lo.z; bq[slot][3] = lo.w;
                bq[slot][4] = hi.x; bq[slot][5] = hi.y; bq[slot][6] = hi.z; bq[slot][7] = hi.w;
            };
            if (s1_bits != 0u) {
                rd(0, 0);
#pragma unroll
                for (int k = 0; k < KPG; ++k) {
                    const int cur = k & 1;
                    if (k + 1 < KPG)
                        rd(k + 1, cur ^ 1);
                    __builtin_amdgcn_sched_barrier(0);
                    if ((s1_bits >> k) & 1u)
                        dma_s1_step(acc, al[cur], ah[cur], bq[cur]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        // S2 steps, then S3 steps (1 + M_A and +-2^E_A derived per row).
        for (uint32_t todo = s2_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = __builtin_ctz(todo);
            uint32_t aa[8], bb[8];
            dma_frag(a_row + kk * BM, HM, aa);
            dma_frag(b_row + kk * BN, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                dma_s2_row(acc[i], aa[i], bb);
        }
        for (uint32_t todo = s3_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = __builtin_ctz(todo);
            uint32_t aa[8], bb[8];
            dma_frag(a_row + kk * BM, HM, aa);
            dma_frag(b_row + kk * BN, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                dma_s3_row(acc[i], aa[i], bb);
        }
        // SPECIAL: the complete definition per MAC (B: b' + bias, denormals
        // already zero).
#pragma unroll 1
        for (uint32_t todo = sp_bits; todo != 0u; todo &= todo - 1u) {
            const int kk = __builtin_ctz(todo);
            uint32_t aa[8], bb[8];
            dma_frag(a_row + kk * BM, HM, aa);
            dma_frag(b_row + kk * BN, HN, bb);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[i][j] += __uint_as_float(pam_full(aa[i], bb[j] + kBias));
            }
        }
    }

    // Epilogue: the output tile in C, or this K slice's partial tile (packed,
    // written whole).
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
    if constexpr (KW > 1) {
        // Groups 1.. write their partial tiles, as many at a time as the LDS
        // holds (kRedTiles); group 0 adds them, in group order, to its own.
        float *red = reinterpret_cast<float *>(smem);
#pragma unroll
        for (int g0 = 1; g0 < KW; g0 += kRedTiles) {
            __syncthreads();   // the LDS is free: every wave is past its last chunk / the previous round's adds
            if (grp >= g0 && grp < g0 + kRedTiles) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int row = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int col = h == 0 ? tx * 4 : HN + tx * 4;
                        *reinterpret_cast<float4 *>(&red[((grp - g0) * BM + row) * LDR + col]) =
                            make_float4(acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3]);
                    }
                }
            }
            __syncthreads();
            if (grp == 0) {
                // Row by row: the row's partial values, then its adds (in
                // inline asm, in group order, so that the compiler neither
                // loads every partial tile up front nor moves the adds past
                // the next row's loads).
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    asm volatile("" ::: "memory");
                    const int row = i < 4 ? ty * 4 + i : HM + ty * 4 + (i - 4);
#pragma unroll
                    for (int g = g0; g < g0 + kRedTiles && g < KW; ++g) {
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const int col = h == 0 ? tx * 4 : HN + tx * 4;
                            const float4 x =
                                *reinterpret_cast<const float4 *>(&red[((g - g0) * BM + row) * LDR + col]);
                            asm volatile("v_add_f32 %0, %0, %4\n\tv_add_f32 %1, %1, %5\n\t"
                                         "v_add_f32 %2, %2, %6\n\tv_add_f32 %3, %3, %7"
                                         : "+v"(acc[i][4 * h]), "+v"(acc[i][4 * h + 1]), "+v"(acc[i][4 * h + 2]),
                                           "+v"(acc[i][4 * h + 3])
                                         : "v"(x.x), "v"(x.y), "v"(x.z), "v"(x.w));
                        }
                    }
                }
            }
        }
        if (grp > 0)
            return;
    }
    typedef float f32x4 __attribute__((ext_vector_type(4)));
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
                const f32x4 v = {acc[i][4 * h], acc[i][4 * h + 1], acc[i][4 * h + 2], acc[i][4 * h + 3]};
                // The final C with the non-temporal hint (written once);
                // split partial sums without it (the reduce reads them soon).
                if (whole)
                    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(orow + col));
                else
                    *reinterpret_cast<f32x4 *>(orow + col) = v;
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (col + j < lim_n)
                        orow[col + j] = acc[i][4 * h + j];
            }
        }
    }
}

template <typename T, int BM, int BN, int KW, int WPS = dma_waves_per_simd(BM, BN, KW)>
static hipError_t launch_dma_tile(bool ta, bool tb, const GemmParams &p, dim3 grid, hipStream_t stream) {
    const dim3 block(BM * BN / 64 * KW);
    if (!ta && !tb)
        hipLaunchKernelGGL((pam_gemm_dma_kernel<BM, BN, KW, false, false, WPS, T>), grid, block, 0, stream, p);
    else if (!ta && tb)
        hipLaunchKernelGGL((pam_gemm_dma_kernel<BM, BN, KW, false, true, WPS, T>), grid, block, 0, stream, p);
    else if (ta && !tb)
        hipLaunchKernelGGL((pam_gemm_dma_kernel<BM, BN, KW, true, false, WPS, T>), grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL((pam_gemm_dma_kernel<BM, BN, KW, true, true, WPS, T>), grid, block, 0, stream, p);
    return hipGetLastError();
}

template <typename T>
static hipError_t launch_dma_shape(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b,
                                   const GemmParams &p, int64_t items, hipStream_t stream) {
    const dim3 grid((unsigned)items);
    if (tile_m == 128 && tile_n == 128 && kgroups == 1)
        return launch_dma_tile<T, 128, 128, 1>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 128 && tile_n == 64 && kgroups == 1)
        return launch_dma_tile<T, 128, 64, 1>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 128 && tile_n == 64 && kgroups == 2)
    {
        // A launch that two workgroups per compute unit hold at once runs
        // the build for two waves per SIMD (staging addresses kept in
        // registers); its occupancy is two anyway.
        if (items <= 2 * 256)
            return launch_dma_tile<T, 128, 64, 2, 2>(trans_a, trans_b, p, grid, stream);
        return launch_dma_tile<T, 128, 64, 2>(trans_a, trans_b, p, grid, stream);
    }
    if (tile_m == 64 && tile_n == 64 && kgroups == 1)
        return launch_dma_tile<T, 64, 64, 1>(trans_a, trans_b, p, grid, stream);
    if (tile_m == 64 && tile_n == 64 && kgroups == 4)
        return launch_dma_tile<T, 64, 64, 4>(trans_a, trans_b, p, grid, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_pam_gemm_dma(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, bool bf16,
                               const GemmParams &p, hipStream_t stream) {
    const int64_t items = (int64_t)p.whole + (int64_t)p.split_tiles * p.splits;
    if (items <= 0 || items > kMaxLaunchItems)
        return hipErrorInvalidValue;
    if (bf16)
        return launch_dma_shape<uint16_t>(tile_m, tile_n, kgroups, trans_a, trans_b, p, items, stream);
    return launch_dma_shape<float>(tile_m, tile_n, kgroups, trans_a, trans_b, p, items, stream);
}

}  // namespace pamk
