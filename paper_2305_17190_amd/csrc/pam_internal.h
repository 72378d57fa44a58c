// Internal interface between the C-ABI layer (pam_api.cpp) and the HIP
// kernels (pam_gemm_dma.hip, pam_kernels.hip, pa_ops.hip,
// pam_exact_grad.hip).  Not installed; not part of the public ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime_api.h>

namespace pamk {

// K extent of one LDS chunk.
constexpr int kChunkK = 16;

// Arguments of one (batched, possibly split-K) PAM matrix product launch.
//
// Matrix product launches run whole + split_tiles * splits work items: tiles
// are numbered batch-major, then by tile row, then tile column (`tiles` per
// matrix, `tiles_n` per tile row); item i < whole computes tile i over the
// whole K into C; item whole + s * split_tiles + t computes K slice s (k in
// [s * k_per_split, (s + 1) * k_per_split)) of tile whole + t into the
// tile-packed partial sums W[s][t][tile_m][tile_n].
struct GemmParams {
    const float *A;    // operands (bfloat16 elements for the bfloat16 products)
    const float *B;
    float *C;          // final output
    float *W;          // partial sums of the split tiles, or nullptr (layout per kernel)
    int64_t lda, ldb, ldc;
    int64_t strideA, strideB, strideC;
    int32_t m, n, k;
    int32_t k_per_split;  // multiple of kChunkK
    int32_t splits;
    int32_t tiles_n;
    int32_t tiles;        // matrix products: tiles per matrix
    int32_t whole;        // matrix products: whole-K work items
    int32_t split_tiles;  // matrix products: tiles split into `splits` K slices
    int32_t vec_a;        // float4 global loads of A are aligned
    int32_t vec_b;        // float4 global loads of B are aligned
    int32_t vec_c;        // float4 stores of the output are aligned
    int32_t round_drop;   // 0, or 23 - m: round every input to m mantissa bits first
    // Exact-derivative products only: the output-shaped operand whose
    // mantissas set each term's carry (row-major, leading dimension ldm).
    const float *Mod;
    int64_t ldm;
};

hipError_t launch_pam_mul(const float *a, const float *b, float *out, int64_t n, hipStream_t stream);

// Elementwise PAD, palog2 and paexp2 (pa_ops.hip).
hipError_t launch_pad(const float *a, const float *b, float *out, int64_t n, hipStream_t stream);
hipError_t launch_palog2(const float *a, float *out, int64_t n, hipStream_t stream);
hipError_t launch_paexp2(const float *a, float *out, int64_t n, hipStream_t stream);
// Round to 23 - drop mantissa bits, nearest even (drop in [1, 23]).
hipError_t launch_round_mantissa(const float *a, float *out, int64_t n, int drop, hipStream_t stream);

// (tile_m, tile_n, kgroups) in {(128,128,1), (128,64,1), (64,64,1), (64,64,4)};
// a one-dimensional grid of p.whole + p.split_tiles * p.splits workgroups.
// bf16: p.A and p.B hold bfloat16 elements (leading dimensions and strides
// in elements), widened exactly to float32 as they are loaded.
hipError_t launch_pam_gemm(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, bool bf16,
                           const GemmParams &p, hipStream_t stream);

// The kernel behind launch_pam_gemm (pam_gemm_dma.hip): operand chunks
// copied into LDS by the memory pipeline.  With bf16, the copies need the
// operand 16-byte aligned with leading dimension and stride multiples of 8
// elements (p.vec_a / p.vec_b), else its elements are loaded one by one.
hipError_t launch_pam_gemm_dma(int tile_m, int tile_n, int kgroups, bool trans_a, bool trans_b, bool bf16,
                               const GemmParams &p, hipStream_t stream);

// C of the split tiles of a matrix product launch: element by element the sum
// over s = 0, 1, ... of W[s][t][.][.], in that order.
hipError_t launch_split_tile_reduce(int tile_m, int tile_n, const GemmParams &p, hipStream_t stream);

// Bytes of the static split-K scratch pam_gemm_batched_noalloc uses, and its
// device address on the current device (looked up once per device).
constexpr size_t kScratchBytes = (size_t)64 << 20;
hipError_t scratch_address(void **out);

// Workgroups one matrix product launch may hold (its grid, in threads, stays
// below 2^32).
constexpr int64_t kMaxLaunchItems = 16777215;

// Exact-derivative product (pam_exact_grad.hip): C(r, c) = sum_q op(A)(r, q)
// d(Mod(r, c) .^ B(q, c)) / dMod(r, c); 128 x 128 tiles, grid (tiles, splits).
hipError_t launch_pam_exact_grad(bool trans_a, const GemmParams &p, hipStream_t stream);

// Exact-derivative products: C[b][i][j] = sum_s W[b][s][i][j], s in
// increasing order.
hipError_t launch_splitk_reduce(const float *W, float *C, int32_t m, int32_t n, int64_t ldc,
                                int64_t strideC, int32_t splits, int64_t batch, hipStream_t stream);

// C[b][i][j] = +0.0f for a k == 0 product.
hipError_t launch_fill_zero(float *C, int32_t m, int32_t n, int64_t ldc, int64_t strideC,
                            int64_t batch, hipStream_t stream);

}  // namespace pamk
