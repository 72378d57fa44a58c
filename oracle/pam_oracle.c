/*
 * Plain C oracle for piecewise affine multiplication (PAM) and PAM matrix
 * products.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests and by the benchmark's CPU
 * baseline.  It shares no code, header or constant table with the HIP
 * library.  Scalar code, no intrinsics; build without fast-math.
 *
 * Source: Kosson & Jaggi, "Multiplication-Free Transformer Training via
 * Piecewise Affine Operations", Sec. 2.2 (PAM of two float32 numbers as the
 * int32 sum of their encodings minus one exponent bias, with under/overflow
 * clamped, denormals flushed and NaN/inf handled explicitly) and Sec. 3.2
 * (matrix products whose scalar products are PAM, accumulated by ordinary
 * addition).  Readings, as in the Python oracle:
 *   sign = exclusive or of the signs; zero and denormal operands give a signed
 *   zero; an underflowing result (exponent field <= 0) gives a signed zero; an
 *   overflowing result (exponent field >= 255) saturates to +-FLT_MAX; NaN in
 *   gives the quiet NaN 0x7FC00000, inf times zero/denormal gives that NaN,
 *   inf times anything else gives a signed inf.
 * Accumulation is in double, in increasing k.
 */
#include <stdint.h>
#include <string.h>
#include <math.h>

uint32_t pam_oracle_bits(uint32_t ua, uint32_t ub)
{
    uint32_t s = (ua ^ ub) & 0x80000000u;
    int64_t ma = (int64_t)(ua & 0x7FFFFFFFu);
    int64_t mb = (int64_t)(ub & 0x7FFFFFFFu);
    int64_t t;

    if (ma > 0x7F800000 || mb > 0x7F800000)
        return 0x7FC00000u;
    if (ma == 0x7F800000 || mb == 0x7F800000) {
        int64_t other = (ma == 0x7F800000) ? mb : ma;
        if (other < 0x00800000)
            return 0x7FC00000u;
        return s | 0x7F800000u;
    }
    if (ma < 0x00800000 || mb < 0x00800000)
        return s;
    t = ma + mb - 0x3F800000;
    if (t < 0x00800000)
        return s;
    if (t > 0x7F7FFFFF)
        return s | 0x7F7FFFFFu;
    return s | (uint32_t)t;
}

static float pam_oracle_f(float a, float b)
{
    uint32_t ua, ub, r;
    float out;
    memcpy(&ua, &a, 4);
    memcpy(&ub, &b, 4);
    r = pam_oracle_bits(ua, ub);
    memcpy(&out, &r, 4);
    return out;
}

void pam_oracle_mul(const float *a, const float *b, float *out, int64_t n)
{
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < n; i++)
        out[i] = pam_oracle_f(a[i], b[i]);
}

/*
 * Sub-grid of a (batched) PAM matrix product.  op(A) is m x k with element
 * (i, kk) at A[i*lda + kk] (ta == 0) or A[kk*lda + i] (ta != 0); op(B) is
 * k x n likewise.  For each batch index z in batches[0..nb), each row
 * rows[r] and each column cols[c]:
 *   C[(z*nr + r)*nc + c] = sum_kk pam(op(A_z)(rows[r], kk), op(B_z)(kk, cols[c]))
 * and S the same sum of absolute values.  Operands of batch z start at
 * A + z*stride_a and B + z*stride_b.
 */
void pam_oracle_gemm(int ta, int tb, int64_t k,
                     const float *A, int64_t lda, int64_t stride_a,
                     const float *B, int64_t ldb, int64_t stride_b,
                     const int64_t *batches, int64_t nb,
                     const int64_t *rows, int64_t nr,
                     const int64_t *cols, int64_t nc,
                     double *C, double *S)
{
    int64_t task;
#pragma omp parallel for schedule(dynamic, 1)
    for (task = 0; task < nb * nr; task++) {
        int64_t z = task / nr, r = task % nr, c, kk;
        const float *Az = A + batches[z] * stride_a;
        const float *Bz = B + batches[z] * stride_b;
        int64_t i = rows[r];
        for (c = 0; c < nc; c++) {
            int64_t j = cols[c];
            double acc = 0.0, mag = 0.0;
            for (kk = 0; kk < k; kk++) {
                float av = ta ? Az[kk * lda + i] : Az[i * lda + kk];
                float bv = tb ? Bz[j * ldb + kk] : Bz[kk * ldb + j];
                double p = (double)pam_oracle_f(av, bv);
                acc += p;
                mag += fabs(p);
            }
            C[task * nc + c] = acc;
            S[task * nc + c] = mag;
        }
    }
}

int pam_oracle_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sets the thread count of the parallel loops that follow (n < 1 -> 1). */
void pam_oracle_set_threads(int n)
{
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n > 0 ? n : 1);
}
