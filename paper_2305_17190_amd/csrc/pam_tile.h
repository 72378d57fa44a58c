// Operand tile staging through registers, used by the exact-derivative
// products (pam_exact_grad.hip): the per-thread global-memory loader of a
// D x BK operand tile (16-byte loads at fixed per-thread offsets, ragged
// edges, k tail), its scans and the SCALED-encoding LDS store, and the
// 8-value LDS fragment read.  Included by the HIP sources only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pam_internal.h"
#include "pam_scalar.h"

namespace pamk {

// float32 encodings of the operand elements: a float32 is its own encoding;
// a bfloat16 (the high 16 bits of a float32) widens exactly by a shift.
__device__ __forceinline__ uint32_t widen(float x) { return __float_as_uint(x); }
__device__ __forceinline__ uint32_t widen(uint16_t h) { return (uint32_t)h << 16; }

// An operand tile of D (rows of op(A), or columns of op(B)) x kChunkK, staged
// through registers, from float32 or bfloat16 (T) elements.  KCONTIG: element (o, kk) of chunk c sits at
// base + (o0 + o) * ld + k0 + kk (A with op N, B with op T); otherwise at
// base + (k0 + kk) * ld + o0 + o (A with op T, B with op N).  Each thread
// holds L groups of four elements consecutive in memory.  The byte offset of
// each group from the chunk's base is fixed for the whole K loop, so the base
// (uniform, in scalar registers) is the only address that moves.
template <int D, int NT, int BK, bool KCONTIG, typename T = float>
struct TileLoader {
    static constexpr int ES = (int)sizeof(T);   // bytes per element
    static constexpr int L = D * BK / 4 / NT;
    static_assert(L >= 1 && D * BK / 4 == L * NT, "tile does not divide over the threads");
    uint4 v[L];
    uint32_t boff[L];   // byte offset of the group from the chunk base
    uint32_t edge;      // bit r: group r straddles the last valid row (OCONTIG) -- per-element path

    // Group r of thread tid: KCONTIG -> (row o, k offset kq); else (k row kk, first o oq).
    static __device__ __forceinline__ int grp_o(int tid, int r) {
        const int f = tid + NT * r;
        return KCONTIG ? f / (BK / 4) : (f % (D / 4)) * 4;
    }
    static __device__ __forceinline__ int grp_k(int tid, int r) {
        const int f = tid + NT * r;
        return KCONTIG ? (f % (BK / 4)) * 4 : f / (D / 4);
    }

    // Rows past o_lim are clamped to the last valid row (their outputs are
    // discarded); the clamp is fixed for the whole K loop.
    __device__ __forceinline__ void init(int64_t ld, int o0, int o_lim, int tid) {
        edge = 0;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const int o = grp_o(tid, r);
            const int kk = grp_k(tid, r);
            if (KCONTIG) {
                const int row = min(o0 + o, o_lim - 1) - o0;
                boff[r] = (uint32_t)((row * ld + kk) * ES);
            } else {
                boff[r] = (uint32_t)((kk * ld + o) * ES);
                if (o0 + o + 3 >= o_lim)
                    edge |= 1u << r;
            }
        }
    }

    // Load chunk elements [k0, k0 + BK) of the panel whose chunk base is
    // `base`.  Elements at k >= k_lim are zero (they must add nothing).
    __device__ __forceinline__ void load(const T *__restrict__ base, int o0, int o_lim, int k0, int k_lim,
                                         bool vec, int tid) {
        const char *cb = reinterpret_cast<const char *>(base);
        if (vec && k0 + BK <= k_lim) {
            // Interior chunk, aligned operand: one 16-byte load per group.
#pragma unroll
            for (int r = 0; r < L; ++r) {
                if (KCONTIG || !((edge >> r) & 1u))
                    v[r] = load_group(cb + boff[r]);
                else
                    v[r] = load_elements(cb, r, o0, o_lim, k0, k_lim, tid);
            }
        } else {
#pragma unroll
            for (int r = 0; r < L; ++r)
                v[r] = load_elements(cb, r, o0, o_lim, k0, k_lim, tid);
        }
    }

    // Four consecutive elements at a 16-byte (float32) or 8-byte (bfloat16)
    // aligned address, as float32 encodings.
    static __device__ __forceinline__ uint4 load_group(const char *p) {
        if constexpr (sizeof(T) == 4) {
            return *reinterpret_cast<const uint4 *>(p);
        } else {
            const uint2 h = *reinterpret_cast<const uint2 *>(p);   // elements 0, 1 in h.x; 2, 3 in h.y
            return make_uint4(h.x << 16, h.x & 0xFFFF0000u, h.y << 16, h.y & 0xFFFF0000u);
        }
    }

    // Group r element by element, with the K tail and (OCONTIG) the last
    // valid row applied.
    __device__ __forceinline__ uint4 load_elements(const char *cb, int r, int o0, int o_lim, int k0, int k_lim,
                                                   int tid) const {
        const T *src = reinterpret_cast<const T *>(cb + boff[r]);
        const int kk = grp_k(tid, r);
        uint32_t e[4];
        if (KCONTIG) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
                e[c] = (k0 + kk + c < k_lim) ? widen(src[c]) : 0u;
        } else {
            const int o = grp_o(tid, r);
            const T *row = src - o;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                e[c] = (k0 + kk < k_lim) ? widen(row[min(o0 + o + c, o_lim - 1) - o0]) : 0u;
        }
        return make_uint4(e[0], e[1], e[2], e[3]);
    }

    // Round every held element to 23 - drop mantissa bits, nearest even: the
    // dropped bits plus (half - 1) plus the kept part's lowest bit carry into
    // the kept part exactly when it must round up; a carry out of the
    // mantissa moves into the exponent (past the largest one, onto inf).
    // inf and NaN stay as they are.
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

    // Scan the held elements.  Returns bit 0 when some element has exponent
    // field below 64 (zero, denormal, or "tiny": a normal number whose
    // products can underflow), bit 1 when some element needs the SPECIAL
    // path (inf, NaN or |x| >= 2^64), and bit 2 + r when group r holds an
    // element of the first kind.
    __device__ __forceinline__ uint32_t scan() const {
        uint32_t hi = 0, groups = 0;
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
            uint32_t lo = 0xFFFFFFFFu;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t ex = e[c] & kExpMask;
                hi = max(hi, ex);
                lo = min(lo, ex);
            }
            if (lo < (64u << 23))
                groups |= 1u << r;
        }
        return (groups != 0u ? 1u : 0u) | (hi >= (191u << 23) ? 2u : 0u) | (groups << 2);
    }

    // Write the chunk into LDS buffer s, k-major: s[plane][kk][o].  A: plane 0
    // aM (1 + M), plane 1 m (+-2^E or +-0), plane 2 a itself; B: plane 0 b'
    // (b - bias, zero and denormal b as a signed zero first).  In the groups
    // flagged in `low_groups` (bit r: group r, as scan() reports), an element
    // at chunk step k with exponent field below 64 sets bit k % 16 of
    // mask[(k / 16) * slots + slot_of(o)], and a normal one among them (tiny)
    // also bit 16 + k % 16; slot_of(o) names the waves that read the element
    // of tile row (A) or column (B) o.
    template <int LDS_LD, typename SlotOf>
    __device__ __forceinline__ void store(uint32_t (*s)[BK][LDS_LD], bool is_b, int tid, uint32_t low_groups,
                                          uint32_t *mask, int slots, SlotOf slot_of) const {
#pragma unroll
        for (int r = 0; r < L; ++r) {
            const uint32_t e[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
            uint32_t p0[4], p1[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t u = e[c];
                if (is_b) {
                    // Multiplying by 1.0 flushes a denormal to the signed
                    // zero (denormals are flushed); everything else passes
                    // unchanged (a NaN stays a NaN).
                    uint32_t f;
                    asm("v_mul_f32 %0, 1.0, %1" : "=v"(f) : "v"(u));
                    p0[c] = f - kBias;
                    p1[c] = 0u;
                } else {
                    p0[c] = (u & kMant) | kBias;
                    p1[c] = u & kSignExp;
                }
            }
            const int o = grp_o(tid, r);
            const int kk = grp_k(tid, r);
            if (KCONTIG) {
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    s[0][kk + c][o] = p0[c];
                if (!is_b) {
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        s[1][kk + c][o] = p1[c];
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        s[2][kk + c][o] = e[c];
                }
            } else {
                *reinterpret_cast<uint4 *>(&s[0][kk][o]) = make_uint4(p0[0], p0[1], p0[2], p0[3]);
                if (!is_b) {
                    *reinterpret_cast<uint4 *>(&s[1][kk][o]) = make_uint4(p1[0], p1[1], p1[2], p1[3]);
                    *reinterpret_cast<uint4 *>(&s[2][kk][o]) = v[r];
                }
            }
            // Rare: a branch per group, which the wave skips unless one of
            // its lanes holds such an element in this group.
            if ((low_groups >> r) & 1u) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t ex = e[c] & kExpMask;
                    if (ex < (64u << 23)) {
                        const int k = KCONTIG ? kk + c : kk;
                        const uint32_t bit = 1u << (k % 16);
                        atomicOr(&mask[(k / 16) * slots + slot_of(KCONTIG ? o : o + c)],
                                 ex != 0u ? (bit | (bit << 16)) : bit);
                    }
                }
            }
        }
    }
};

template <int BK, int LD>
__device__ __forceinline__ void lds_frag(const uint32_t (*s)[BK][LD], int plane, int kk, int i0, int half,
                                         uint32_t out[8]) {
    const uint4 lo = *reinterpret_cast<const uint4 *>(&s[plane][kk][i0]);
    const uint4 hi = *reinterpret_cast<const uint4 *>(&s[plane][kk][half + i0]);
    out[0] = lo.x; out[1] = lo.y; out[2] = lo.z; out[3] = lo.w;
    out[4] = hi.x; out[5] = hi.y; out[6] = hi.z; out[7] = hi.w;
}

}  // namespace pamk
