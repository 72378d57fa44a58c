/*
 * pam.h -- C ABI of the piecewise affine multiplication (PAM) library for
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Kosson & Jaggi, "Multiplication-Free Transformer Training via
 * Piecewise Affine Operations" (NeurIPS 2023).
 *
 * PAM (Sec. 2.2) replaces the product of two float32 numbers
 *   A = (-1)^S_A 2^E_A (1 + M_A),  B = (-1)^S_B 2^E_B (1 + M_B)
 * by (-1)^(S_A+S_B) 2^(E_A+E_B+c) (1 + M_A + M_B - c), c = 1{M_A + M_B >= 1},
 * which is the int32 sum of the two encodings minus one exponent bias
 * (127 << 23).  The same passage asks for clamped exponent under/overflow,
 * flushed denormals and explicit NaN/inf handling; this library fixes those
 * cases as follows (identical in every entry point):
 *   - sign of the result = exclusive or of the operand signs, also for zeros;
 *   - a zero or denormal operand gives a signed zero;
 *   - a result whose exponent field would be <= 0 is a signed zero;
 *   - a result whose exponent field would be >= 255 is +-FLT_MAX;
 *   - a NaN operand, or inf times a zero/denormal, gives 0x7FC00000;
 *     inf times any other value gives a signed inf.
 *
 * PAM matrix products (Sec. 3.2, Table 1 approximate derivative) replace
 * every scalar product of a matrix multiply by PAM and keep ordinary float32
 * addition for the accumulation (App. "Hardware Cost", App. "PAM with
 * Narrower Mantissas").  The summation order is not part of the contract:
 * results agree with an exact-order sum to within float32 rounding, and
 * denormal partial sums may be flushed to zero.
 *
 * Conventions for every call:
 *   - All matrix/array pointers are DEVICE pointers (memory of the current
 *     HIP device); the caller owns every buffer.
 *   - Every call is asynchronous on `stream` (NULL = the null stream) and
 *     never synchronises.  Execution errors surface at the caller's next
 *     synchronisation.
 *   - Matrices are row-major with leading dimensions in elements.  For a
 *     matrix product, op(A) is m x k and op(B) is k x n:
 *       op(A)(i, p) = A[i*lda + p]  if transA == PAM_OP_N,  A[p*lda + i]  if PAM_OP_T
 *       op(B)(p, j) = B[p*ldb + j]  if transB == PAM_OP_N,  B[j*ldb + p]  if PAM_OP_T
 *     and C(i, j) = C[i*ldc + j] is overwritten (there is no alpha/beta:
 *     scaling would be a multiplication).
 *   - Arguments are validated before anything is launched; on failure the
 *     call returns PAM_ERROR_INVALID_VALUE and pam_last_error() says why.
 *   - Output regions overlapping an input are undefined (not checked), except
 *     that the elementwise calls (pam_mul, pam_pad, pam_palog2, pam_paexp2,
 *     pam_round_mantissa) may run in place (out == a or out == b).
 *   - The library allocates no memory.  Products that split K keep the
 *     partial sums of the K slices in a workspace the caller passes (the
 *     *_ws, with_plan and bf16 entry points); the entry points without a
 *     workspace argument use the fastest plan that does not split K.
 *   - The library keeps no state across calls but a per-thread error text
 *     and device check; it changes no process-wide setting.
 */
#ifndef PAM_H_
#define PAM_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PAM_SUCCESS = 0,
    PAM_ERROR_INVALID_VALUE = 1, /* bad size, leading dimension, pointer or option */
    PAM_ERROR_LAUNCH = 2,        /* a HIP launch or query failed */
    PAM_ERROR_NOT_SUPPORTED = 3  /* device is not gfx950 */
} pam_status_t;

/* An int-sized enum.  Any other value is refused with PAM_ERROR_INVALID_VALUE;
 * C++ sees a fixed underlying type, so such a value is still a valid object. */
#ifdef __cplusplus
typedef enum : int32_t { PAM_OP_N = 0, PAM_OP_T = 1 } pam_op_t;
#else
typedef enum { PAM_OP_N = 0, PAM_OP_T = 1 } pam_op_t;
#endif

/*
 * Elementwise PAM (Sec. 2.2): out[i] = a[i] .^ b[i] for 0 <= i < n.
 * a, b, out: device arrays of n float32.  n >= 0 (n == 0 launches nothing).
 * Bit-exact: every one of the 2^64 operand pairs has exactly one result.
 */
pam_status_t pam_mul(const float *a, const float *b, float *out, int64_t n, hipStream_t stream);

/*
 * Elementwise piecewise affine division (PAD, Sec. 2.3), the inverse of PAM:
 * out[i] = a[i] ./ b[i], the int32 difference of the encodings plus one
 * exponent bias (127 << 23), whose borrow realises 1{M_A - M_B < 0} (the
 * printed exponent / mantissa lines of Sec. 2.3 are read with this borrow).
 * Sign = exclusive or; denormal operands count as zero; a NaN operand,
 * 0 ./ 0 and inf ./ inf give 0x7FC00000; x ./ 0 and inf ./ x give a signed
 * inf; 0 ./ x and x ./ inf a signed zero; a result exponent field <= 0 a
 * signed zero, >= 255 +-FLT_MAX.  Bit-exact: one result per operand pair.
 * a, b, out: device arrays of n float32 (out may alias a or b); n >= 0.
 */
pam_status_t pam_pad(const float *a, const float *b, float *out, int64_t n, hipStream_t stream);

/*
 * Elementwise palog2 (Sec. 2.3): out[i] = E + M for a[i] = 2^E (1 + M) > 0,
 * rounded to the nearest float32 (ties to even).  +-0 and denormals give
 * -inf, negative inputs NaN (0x7FC00000), +inf +inf, NaN 0x7FC00000.
 * a, out: device arrays of n float32 (out may alias a); n >= 0.
 */
pam_status_t pam_palog2(const float *a, float *out, int64_t n, hipStream_t stream);

/*
 * Elementwise paexp2 (Sec. 2.3): out[i] = 2^floor(x) (1 + x - floor(x)) for
 * x = a[i], rounded to the nearest float32 (ties to even).  Results below
 * 2^-126 are +0, above FLT_MAX +inf; -inf gives +0, NaN 0x7FC00000;
 * denormal inputs count as zero.  a, out: device arrays of n float32 (out
 * may alias a); n >= 0.
 */
pam_status_t pam_paexp2(const float *a, float *out, int64_t n, hipStream_t stream);

/*
 * PAM matrix product (Sec. 3.2): C(i, j) = sum_p op(A)(i, p) .^ op(B)(p, j)
 * for 0 <= i < m, 0 <= j < n, float32 accumulation.
 * The forward pass of a linear layer Y = X W^T is (N, T); its approximate
 * backward products (Table 1) are dX = dY W (N, N) and dW = dY^T X (T, N).
 * Requirements: 0 <= m, n, k < 2^31; lda >= max(1, transA == N ? k : m);
 * ldb >= max(1, transB == N ? n : k); ldc >= max(1, n); lda, ldb < 2^22
 * (else PAM_ERROR_NOT_SUPPORTED); A, B non-NULL when m*k resp. k*n > 0;
 * C non-NULL when m*n > 0.  m == 0 or n == 0 launches nothing; k == 0
 * writes +0.0f to C.  No workspace: the plan does not split K
 * (pam_gemm_batched_ws takes one and may).
 */
pam_status_t pam_gemm(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                      const float *A, int64_t lda, const float *B, int64_t ldb,
                      float *C, int64_t ldc, hipStream_t stream);

/*
 * `batch` independent PAM matrix products, as in the attention products of
 * Sec. 3.2 (Q K^T, P V and their backward products).  Product z reads
 * A + z*strideA and B + z*strideB and writes C + z*strideC, each with the
 * layout of pam_gemm.  Strides are in elements, >= 0 (a zero A or B stride
 * broadcasts that operand); batch >= 0.  Same requirements as pam_gemm; no
 * workspace, so no split K.
 */
pam_status_t pam_gemm_batched(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                              const float *A, int64_t lda, int64_t strideA,
                              const float *B, int64_t ldb, int64_t strideB,
                              float *C, int64_t ldc, int64_t strideC,
                              int64_t batch, hipStream_t stream);

/*
 * How a product is tiled: output tile tile_m x tile_n per workgroup;
 * kgroups waves per micro-tile position that share each LDS chunk's k steps
 * and add their partial tiles in LDS; the number of K slices whose partial
 * sums are added by a second kernel (1 = none); and with splits > 1, how many
 * tiles take the whole K in the same launch instead: the first whole_tiles
 * tiles, numbered batch-major, then by tile row, then tile column (0 = every
 * tile is split; >= the tile count = none is).  Splitting only the last
 * tiles fills the last round of workgroups with shorter ones.
 */
typedef struct {
    int32_t tile_m;
    int32_t tile_n;
    int32_t splits;
    int32_t kgroups;
    int64_t whole_tiles;
} pam_plan_t;

/* The plan pam_gemm_batched_ws (and pam_gemm_workspace_size) uses for these
 * sizes, split K allowed.  m, n, batch > 0; k >= 0. */
pam_status_t pam_gemm_plan(int64_t m, int64_t n, int64_t k, int64_t batch, pam_plan_t *plan);

/* The fastest plan (by the library's cost model) whose split-K partial sums
 * fit in max_workspace_bytes: 0 gives the plan of the entry points without a
 * workspace argument (no split K), SIZE_MAX that of pam_gemm_plan. */
pam_status_t pam_gemm_plan_for_workspace(int64_t m, int64_t n, int64_t k, int64_t batch,
                                         size_t max_workspace_bytes, pam_plan_t *plan);

/*
 * pam_gemm_batched with an explicit plan (for tests and tuning).
 * (tile_m, tile_n, kgroups) is (128,128,1), (128,64,1), (128,64,2),
 * (64,64,1) or (64,64,4); 1 <= splits <= 64; whole_tiles >= 0.  The result is
 * the same product as with the automatic plan, up to float32 summation order.
 * A plan that splits K keeps its partial sums in `workspace`: device memory
 * of workspace_bytes >= pam_gemm_plan_workspace_size's value, 16-byte aligned,
 * that nothing else touches until this call's kernels on `stream` are done
 * (NULL when that value is 0).  A plan with 0 < whole_tiles < tiles runs as
 * one launch and fails with PAM_ERROR_INVALID_VALUE when its workgroups exceed
 * 2^24 - 1.
 */
pam_status_t pam_gemm_batched_with_plan(pam_op_t transA, pam_op_t transB,
                                        int64_t m, int64_t n, int64_t k,
                                        const float *A, int64_t lda, int64_t strideA,
                                        const float *B, int64_t ldb, int64_t strideB,
                                        float *C, int64_t ldc, int64_t strideC,
                                        int64_t batch, const pam_plan_t *plan,
                                        void *workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/* Workspace bytes pam_gemm_batched_with_plan needs for these sizes under
 * `plan` (0 when it does not split K).  m, n, k, batch >= 0 and below 2^31. */
pam_status_t pam_gemm_plan_workspace_size(int64_t m, int64_t n, int64_t k, int64_t batch,
                                          const pam_plan_t *plan, size_t *bytes);

/*
 * Narrower-mantissa PAM matrix products (App. "PAM with Narrower
 * Mantissas"): every element of op(A) and op(B) is first rounded to
 * `mantissa_bits` mantissa bits (nearest, ties to even; a carry moves into
 * the exponent, a finite value rounding past FLT_MAX becomes inf; inf and
 * NaN unchanged), then multiplied with PAM and accumulated in float32 as in
 * pam_gemm_batched.  The caller's A and B are not modified.  mantissa_bits in
 * [0, 23] (23 = pam_gemm_batched); arguments otherwise as pam_gemm_batched.
 */
pam_status_t pam_gemm_narrow(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                             const float *A, int64_t lda, int64_t strideA,
                             const float *B, int64_t ldb, int64_t strideB,
                             float *C, int64_t ldc, int64_t strideC,
                             int64_t batch, int32_t mantissa_bits, hipStream_t stream);

/*
 * The same rounding as an elementwise op: out[i] = a[i] rounded to
 * `mantissa_bits` mantissa bits (App. "PAM with Narrower Mantissas"), e.g. to
 * keep narrow copies of weights.  a, out: device arrays of n float32 (out may
 * alias a); n >= 0; mantissa_bits in [0, 23].
 */
pam_status_t pam_round_mantissa(const float *a, float *out, int64_t n, int32_t mantissa_bits,
                                hipStream_t stream);

/*
 * Exact-derivative PAM products (Table 1; the true derivative of the
 * piecewise affine product, Sec. "Derivatives"): the derivative of
 * Mod .^ B with respect to Mod is sgn(B) 2^(E_B + 1{M_Mod + M_B >= 1}), a
 * power of two, where Mod .^ B is not clamped, and 0 where it is: a zero or
 * denormal Mod or B, a product that underflows to a signed zero, one that
 * saturates at +-FLT_MAX.  This call computes
 *   C(r, c) = sum_q op(A)(r, q) * d(Mod(r, c) .^ B(q, c)) / dMod(r, c)
 * for 0 <= r < m, 0 <= c < n, q < k: each term exact (a denormal op(A)
 * element counts as zero), float32 accumulation.  For Y = X .^ W^T
 * (X: T x K, W: N x K, dY: T x N):
 *   dX = (transA = N, A = dY, B = W, Mod = X)   m = T, n = K, k = N
 *   dW = (transA = T, A = dY, B = X, Mod = W)   m = N, n = K, k = T
 * op(A) as in pam_gemm; B(q, c) = B[q*ldb + c]; Mod(r, c) = Mod[r*ldm + c];
 * C(r, c) = C[r*ldc + c] overwritten.  Requirements as pam_gemm (transB = N)
 * plus ldm >= max(1, n) and Mod non-NULL when m*n > 0.  Every finite
 * operand value is covered; inf / NaN operands give unspecified values.
 * Long K may split K; without a workspace (this entry point) it does not.
 */
pam_status_t pam_gemm_exact_grad(pam_op_t transA, int64_t m, int64_t n, int64_t k,
                                 const float *A, int64_t lda, const float *B, int64_t ldb,
                                 const float *Mod, int64_t ldm, float *C, int64_t ldc,
                                 hipStream_t stream);

/*
 * Caller-provided split-K workspace.  For long-K / few-tile shapes the
 * fastest plan splits K into slices whose partial sums are then added in a
 * fixed order; these entry points take the buffer for those partial sums from
 * the caller (e.g. from torch's caching allocator) and allocate nothing.
 *
 * pam_gemm_workspace_size: *bytes = the workspace bytes that
 * pam_gemm_batched_ws (and pam_gemm_batched_bf16 with a workspace) needs for
 * these sizes with the library's plan; 0 when the plan does not split K.
 * m, n, k, batch >= 0 and below 2^31; bytes non-NULL.
 *
 * pam_gemm_batched_ws: pam_gemm_narrow's product (mantissa_bits = 23:
 * pam_gemm_batched's), arguments as there, with the library's plan (split K
 * allowed) and the partial sums in `workspace`: device memory of
 * workspace_bytes bytes, 16-byte aligned, that nothing else reads or writes
 * until this call's kernels on `stream` have finished (stream order: a later
 * call on the same stream may reuse it).  workspace_bytes >=
 * pam_gemm_workspace_size's value, else PAM_ERROR_INVALID_VALUE before any
 * launch; workspace may be NULL when that value is 0.  The caller owns the
 * workspace; its contents afterwards are unspecified.
 *
 * pam_gemm_exact_grad_workspace_size / pam_gemm_exact_grad_ws: the same for
 * pam_gemm_exact_grad (whose plan then may split K).
 */
pam_status_t pam_gemm_workspace_size(int64_t m, int64_t n, int64_t k, int64_t batch, size_t *bytes);

pam_status_t pam_gemm_batched_ws(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                 const float *A, int64_t lda, int64_t strideA,
                                 const float *B, int64_t ldb, int64_t strideB,
                                 float *C, int64_t ldc, int64_t strideC,
                                 int64_t batch, int32_t mantissa_bits,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): pam_gemm_batched_ws's product without a workspace argument.
 * Split-K partial sums go to a static scratch of 64 MiB in device memory
 * that the library holds on every device it runs on until the process ends
 * (no hipMalloc, hipFree or other allocation by this call).  The plan is the
 * fastest whose partial sums fit in the scratch (pam_gemm_plan_for_workspace
 * with 64 MiB): pam_gemm_plan's when its workspace is at most 64 MiB, else a
 * shorter split, else none; a plan needing more is refused with
 * PAM_ERROR_INVALID_VALUE (never chosen).  Arguments as pam_gemm_batched_ws
 * without workspace and workspace_bytes.  Every call on a device shares that
 * device's scratch and leaves its contents behind (each call writes every
 * partial sum it reads, so nothing must start at zero): calls that overlap
 * on one device -- on different streams or from different threads -- race;
 * serialize them (one stream, or events).
 */
pam_status_t pam_gemm_batched_noalloc(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                      const float *A, int64_t lda, int64_t strideA,
                                      const float *B, int64_t ldb, int64_t strideB,
                                      float *C, int64_t ldc, int64_t strideC,
                                      int64_t batch, int32_t mantissa_bits, hipStream_t stream);

/*
 * bfloat16 operands (App. "PAM with Narrower Mantissas"; storage of 7-bit
 * mantissa operands in half the bytes): A and B hold bfloat16 values (the
 * high 16 bits of float32 encodings), leading dimensions and batch strides
 * in elements.  Each element is widened exactly to float32 as it is loaded;
 * the product is then pam_gemm_batched's on the widened operands, bit for bit
 * (same plan), with float32 C.  Requirements as pam_gemm_batched.  workspace
 * NULL: the plan of pam_gemm_batched (no split K); otherwise that of
 * pam_gemm_batched_ws (workspace_bytes >= pam_gemm_workspace_size's value).
 */
pam_status_t pam_gemm_batched_bf16(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                   const uint16_t *A, int64_t lda, int64_t strideA,
                                   const uint16_t *B, int64_t ldb, int64_t strideB,
                                   float *C, int64_t ldc, int64_t strideC, int64_t batch,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream);

pam_status_t pam_gemm_exact_grad_workspace_size(int64_t m, int64_t n, int64_t k, size_t *bytes);

pam_status_t pam_gemm_exact_grad_ws(pam_op_t transA, int64_t m, int64_t n, int64_t k,
                                    const float *A, int64_t lda, const float *B, int64_t ldb,
                                    const float *Mod, int64_t ldm, float *C, int64_t ldc,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Figures of `device` that set the vector-ALU roofline: compute units and
 * peak engine clock (kHz) from the HIP runtime, SIMDs per compute unit from
 * HSA, the wavefront size, and the lanes a SIMD retires per clock for the
 * full-rate ops of the PAM matrix product (int32 add, float32 add, mul and
 * fma).  lanes_per_simd is not a device query: it is the library's constant
 * 32 for gfx950, calibrated by issue-rate measurements (two waves per SIMD
 * pair these ops; other vector ops retire 16).
 * valu_lane_ops_per_s = cus * simds_per_cu * lanes_per_simd * clock.
 */
typedef struct {
    int32_t compute_units;
    int32_t simds_per_cu;
    int32_t lanes_per_simd;
    int32_t clock_khz;
    int32_t wavefront_size;
    double valu_lane_ops_per_s;
    char arch[64];
} pam_device_info_t;

pam_status_t pam_device_info(int device, pam_device_info_t *info);

/* Static text for a status code. */
const char *pam_status_string(pam_status_t status);

/* Detail of the last failure on the calling thread ("" if none). */
const char *pam_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PAM_H_ */
