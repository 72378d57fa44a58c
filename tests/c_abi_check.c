/*
 * C-only check of the PAM library's C ABI (include/pam.h): device buffers
 * from hipMalloc, products through the library's entry points, results
 * against the plain C oracle (oracle/pam_oracle.c) on the host.  No Python,
 * no torch.  Test program: built by __graft_entry__.build(), run on the GPU
 * by tests/test_gpu_c_abi.py; prints "c_abi_check: OK" and exits 0 when every
 * case passes.
 *
 * Cases: pam_mul (bit-exact, including zeros, denormals, inf, NaN and a tail
 * of 3 elements); pam_gemm with op(B) transposed on a ragged shape;
 * pam_gemm_batched_ws with a caller workspace on a long-K batched shape whose
 * plan splits K; pam_gemm_batched on the same shape (no workspace: its plan
 * keeps K whole), against the oracle and against that plan forced through
 * pam_gemm_batched_with_plan bit for bit; one refused argument.
 * GEMM tolerance: |C - C_ref| <= 1e-5 sqrt(K) S + K 2^-126 per element, with
 * S = sum of |terms| (the oracle's float64 sums).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "pam.h"

/* The oracle's entry points (oracle/pam_oracle.c). */
void pam_oracle_mul(const float *a, const float *b, float *out, int64_t n);
void pam_oracle_gemm(int ta, int tb, int64_t k, const float *A, int64_t lda, int64_t stride_a, const float *B,
                     int64_t ldb, int64_t stride_b, const int64_t *batches, int64_t nb, const int64_t *rows,
                     int64_t nr, const int64_t *cols, int64_t nc, double *C, double *S);

static int failures = 0;

#define CHECK_HIP(x)                                                                              \
    do {                                                                                          \
        hipError_t e_ = (x);                                                                      \
        if (e_ != hipSuccess) {                                                                   \
            fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_));   \
            exit(2);                                                                              \
        }                                                                                         \
    } while (0)

#define CHECK_PAM(x)                                                                              \
    do {                                                                                          \
        pam_status_t s_ = (x);                                                                    \
        if (s_ != PAM_SUCCESS) {                                                                  \
            fprintf(stderr, "%s:%d: %s: %s (%s)\n", __FILE__, __LINE__, #x, pam_status_string(s_), \
                    pam_last_error());                                                            \
            exit(3);                                                                              \
        }                                                                                         \
    } while (0)

/* splitmix64: the seeded input generator (no PAM arithmetic). */
static uint64_t rng_state;
static uint64_t next_u64(void) {
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
/* Uniform in (-2, 2), with about 1% exact zeros. */
static float next_value(void) {
    uint64_t r = next_u64();
    if (r % 100 == 0)
        return 0.0f;
    return (float)((double)(r >> 11) * (4.0 / 9007199254740992.0) - 2.0);
}
static uint32_t bits_of(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    return u;
}
static float float_of(uint32_t u) {
    float x;
    memcpy(&x, &u, 4);
    return x;
}

static float *to_device(const float *h, size_t n) {
    float *d = NULL;
    CHECK_HIP(hipMalloc((void **)&d, n * sizeof(float) + 16));
    CHECK_HIP(hipMemcpy(d, h, n * sizeof(float), hipMemcpyHostToDevice));
    return d;
}

static void check_mul(hipStream_t stream) {
    const int64_t n = 100003; /* 4-element groups and a tail of 3 */
    float *a = malloc(n * sizeof(float)), *b = malloc(n * sizeof(float));
    float *got = malloc(n * sizeof(float)), *want = malloc(n * sizeof(float));
    const uint32_t specials[] = {0x00000000u, 0x80000000u, 0x00000001u, 0x807FFFFFu, 0x00800000u, 0x3F800000u,
                                 0x7F7FFFFFu, 0x7F800000u, 0xFF800000u, 0x7FC00000u, 0x20000000u, 0x1F800000u};
    const int ns = (int)(sizeof specials / sizeof specials[0]);
    int64_t i;
    for (i = 0; i < n; i++) {
        a[i] = next_value();
        b[i] = next_value();
    }
    for (i = 0; i < ns * ns; i++) { /* every pair of special encodings */
        a[i] = float_of(specials[i / ns]);
        b[i] = float_of(specials[i % ns]);
    }
    float *da = to_device(a, n), *db = to_device(b, n), *dc = to_device(a, n);
    CHECK_PAM(pam_mul(da, db, dc, n, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(got, dc, n * sizeof(float), hipMemcpyDeviceToHost));
    pam_oracle_mul(a, b, want, n);
    int64_t bad = 0;
    for (i = 0; i < n; i++)
        if (bits_of(got[i]) != bits_of(want[i])) {
            if (bad < 5)
                fprintf(stderr, "pam_mul %lld: %08x .^ %08x = %08x, oracle %08x\n", (long long)i, bits_of(a[i]),
                        bits_of(b[i]), bits_of(got[i]), bits_of(want[i]));
            bad++;
        }
    printf("pam_mul n=%lld: %lld mismatches\n", (long long)n, (long long)bad);
    failures += bad != 0;
    CHECK_HIP(hipFree(da));
    CHECK_HIP(hipFree(db));
    CHECK_HIP(hipFree(dc));
    free(a);
    free(b);
    free(got);
    free(want);
}

/* Compare a batch x m x n device result with the oracle on every element. */
static void compare_gemm(const char *what, const float *got, int ta, int tb, int64_t m, int64_t n, int64_t k,
                         const float *A, int64_t lda, int64_t sa, const float *B, int64_t ldb, int64_t sb,
                         int64_t batch, int64_t ldc, int64_t sc) {
    int64_t *bs = malloc(batch * sizeof(int64_t)), *rs = malloc(m * sizeof(int64_t)), *cs = malloc(n * sizeof(int64_t));
    double *C = malloc(batch * m * n * sizeof(double)), *S = malloc(batch * m * n * sizeof(double));
    int64_t z, i, j, bad = 0;
    for (z = 0; z < batch; z++)
        bs[z] = z;
    for (i = 0; i < m; i++)
        rs[i] = i;
    for (j = 0; j < n; j++)
        cs[j] = j;
    pam_oracle_gemm(ta, tb, k, A, lda, sa, B, ldb, sb, bs, batch, rs, m, cs, n, C, S);
    for (z = 0; z < batch; z++)
        for (i = 0; i < m; i++)
            for (j = 0; j < n; j++) {
                const double ref = C[(z * m + i) * n + j];
                const double tol = 1e-5 * sqrt((double)k) * S[(z * m + i) * n + j] + (double)k * ldexp(1.0, -126);
                const double g = (double)got[z * sc + i * ldc + j];
                if (!(fabs(g - ref) <= tol)) {
                    if (bad < 5)
                        fprintf(stderr, "%s [%lld,%lld,%lld]: %.9g vs oracle %.9g (tol %.3g)\n", what, (long long)z,
                                (long long)i, (long long)j, g, ref, tol);
                    bad++;
                }
            }
    printf("%s: %lld of %lld outside the tolerance\n", what, (long long)bad, (long long)(batch * m * n));
    failures += bad != 0;
    free(bs);
    free(rs);
    free(cs);
    free(C);
    free(S);
}

static void check_gemm_nt(hipStream_t stream) {
    /* Y = X .^ W^T: X 203 x 333, W 150 x 333 (op(B) = W^T), ldc padded. */
    const int64_t m = 203, n = 150, k = 333, ldc = 152;
    float *x = malloc(m * k * sizeof(float)), *w = malloc(n * k * sizeof(float));
    float *y = malloc(m * ldc * sizeof(float));
    int64_t i;
    for (i = 0; i < m * k; i++)
        x[i] = next_value();
    for (i = 0; i < n * k; i++)
        w[i] = next_value();
    float *dx = to_device(x, m * k), *dw = to_device(w, n * k), *dy = NULL;
    CHECK_HIP(hipMalloc((void **)&dy, m * ldc * sizeof(float)));
    CHECK_PAM(pam_gemm(PAM_OP_N, PAM_OP_T, m, n, k, dx, k, dw, k, dy, ldc, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(y, dy, m * ldc * sizeof(float), hipMemcpyDeviceToHost));
    compare_gemm("pam_gemm NT 203x150x333", y, 0, 1, m, n, k, x, k, 0, w, k, 0, 1, ldc, 0);
    CHECK_HIP(hipFree(dx));
    CHECK_HIP(hipFree(dw));
    CHECK_HIP(hipFree(dy));
    free(x);
    free(w);
    free(y);
}

static void check_gemm_batched_ws(hipStream_t stream) {
    /* Long K, few tiles: the library's plan splits K. */
    const int64_t m = 70, n = 90, k = 12000, batch = 3;
    const int64_t sa = m * k, sb = k * n, sc = m * n;
    float *a = malloc(batch * sa * sizeof(float)), *b = malloc(batch * sb * sizeof(float));
    float *c = malloc(batch * sc * sizeof(float));
    int64_t i;
    for (i = 0; i < batch * sa; i++)
        a[i] = next_value();
    for (i = 0; i < batch * sb; i++)
        b[i] = next_value();
    float *da = to_device(a, batch * sa), *db = to_device(b, batch * sb), *dc = NULL;
    CHECK_HIP(hipMalloc((void **)&dc, batch * sc * sizeof(float)));
    pam_plan_t plan;
    CHECK_PAM(pam_gemm_plan(m, n, k, batch, &plan));
    size_t bytes = 0;
    CHECK_PAM(pam_gemm_workspace_size(m, n, k, batch, &bytes));
    printf("plan %dx%d, %d slices, %d k-groups, %lld whole tiles; workspace %zu bytes\n", plan.tile_m, plan.tile_n,
           plan.splits, plan.kgroups, (long long)plan.whole_tiles, bytes);
    if (plan.splits < 2 || bytes == 0) {
        fprintf(stderr, "expected a split-K plan with a workspace\n");
        failures++;
    }
    void *ws = NULL;
    CHECK_HIP(hipMalloc(&ws, bytes > 0 ? bytes : 16));
    /* too small a workspace is refused before any launch */
    if (bytes > 0 && pam_gemm_batched_ws(PAM_OP_N, PAM_OP_N, m, n, k, da, k, sa, db, n, sb, dc, n, sc, batch, 23, ws,
                                         bytes - 4, stream) != PAM_ERROR_INVALID_VALUE) {
        fprintf(stderr, "a too small workspace was not refused\n");
        failures++;
    }
    CHECK_PAM(pam_gemm_batched_ws(PAM_OP_N, PAM_OP_N, m, n, k, da, k, sa, db, n, sb, dc, n, sc, batch, 23, ws, bytes,
                                  stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(c, dc, batch * sc * sizeof(float), hipMemcpyDeviceToHost));
    compare_gemm("pam_gemm_batched_ws 3x70x90x12000", c, 0, 0, m, n, k, a, k, sa, b, n, sb, batch, n, sc);
    /* the entry point without a workspace: the plan that keeps K whole, the
       same bits as that plan forced through pam_gemm_batched_with_plan */
    float *c2 = malloc(batch * sc * sizeof(float)), *c3 = malloc(batch * sc * sizeof(float));
    CHECK_HIP(hipMemset(dc, 0xFF, batch * sc * sizeof(float)));
    CHECK_PAM(pam_gemm_batched(PAM_OP_N, PAM_OP_N, m, n, k, da, k, sa, db, n, sb, dc, n, sc, batch, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(c2, dc, batch * sc * sizeof(float), hipMemcpyDeviceToHost));
    compare_gemm("pam_gemm_batched 3x70x90x12000", c2, 0, 0, m, n, k, a, k, sa, b, n, sb, batch, n, sc);
    pam_plan_t whole;
    CHECK_PAM(pam_gemm_plan_for_workspace(m, n, k, batch, 0, &whole));
    size_t whole_bytes = 1;
    CHECK_PAM(pam_gemm_plan_workspace_size(m, n, k, batch, &whole, &whole_bytes));
    if (whole.splits != 1 || whole_bytes != 0) {
        fprintf(stderr, "the plan without a workspace splits K\n");
        failures++;
    }
    CHECK_HIP(hipMemset(dc, 0xFF, batch * sc * sizeof(float)));
    CHECK_PAM(pam_gemm_batched_with_plan(PAM_OP_N, PAM_OP_N, m, n, k, da, k, sa, db, n, sb, dc, n, sc, batch, &whole,
                                         NULL, 0, stream));
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(c3, dc, batch * sc * sizeof(float), hipMemcpyDeviceToHost));
    if (memcmp(c2, c3, batch * sc * sizeof(float)) != 0) {
        fprintf(stderr, "pam_gemm_batched and its plan forced differ\n");
        failures++;
    }
    free(c3);
    CHECK_HIP(hipFree(ws));
    CHECK_HIP(hipFree(da));
    CHECK_HIP(hipFree(db));
    CHECK_HIP(hipFree(dc));
    free(a);
    free(b);
    free(c);
    free(c2);
}

static void check_refusal(void) {
    /* lda below k for op(A) = A: refused before any launch, with a message. */
    const pam_status_t s = pam_gemm(PAM_OP_N, PAM_OP_N, 4, 4, 8, (const float *)256, 4, (const float *)256, 4,
                                    (float *)256, 4, NULL);
    if (s != PAM_ERROR_INVALID_VALUE || pam_last_error()[0] == '\0') {
        fprintf(stderr, "bad lda: status %d, message \"%s\"\n", (int)s, pam_last_error());
        failures++;
    }
}

int main(void) {
    rng_state = 20230527u;
    hipStream_t stream;
    CHECK_HIP(hipSetDevice(0));
    CHECK_HIP(hipStreamCreate(&stream));
    pam_device_info_t info;
    CHECK_PAM(pam_device_info(0, &info));
    printf("device %s: %d CUs, %.1f T lane-op/s\n", info.arch, info.compute_units, info.valu_lane_ops_per_s / 1e12);
    check_mul(stream);
    check_gemm_nt(stream);
    check_gemm_batched_ws(stream);
    check_refusal();
    CHECK_HIP(hipStreamDestroy(stream));
    if (failures) {
        printf("c_abi_check: %d case(s) FAILED\n", failures);
        return 1;
    }
    printf("c_abi_check: OK\n");
    return 0;
}
