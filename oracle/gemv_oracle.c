/*
 * Oracle for the fp32 matrix-vector product y = A * x, evaluated in IEEE
 * fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header or constant with the
 * GPU path.
 *
 * What it computes (the plain definition).  The paper's second benchmark is
 * a full-precision fp32 GEMV (Section 6): for a row-major M x K matrix A and
 * a vector x of K values,
 *
 *     y[i] = sum_{k = 0 .. K-1} A[i*lda + k] * x[k]
 *
 * with the sum taken in ascending k, in fp64.  Alongside it the oracle
 * returns the tolerance scale
 *
 *     s[i] = sum_k | A[i][k] * x[k] |
 *
 * Exactness.  Every fp32 value is a double.  A product of two fp32 values
 * has at most 48 significant bits and an exponent between -298 and +256, so
 * it is exact in fp64 (subnormal fp32 inputs included).  The only rounding is
 * the fp64 summation, bounded by (K-1) * 2^-53 * s.
 *
 * Build with -ffp-contract=off and without -ffast-math: no reassociation and
 * no fused multiply-add (the product must be formed exactly before it is
 * added, which it is anyway in fp64, but contraction would change the
 * rounding of the sum).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/*
 * Selected rows: for r < nrows, y[r] = y_{rows[r]} and s[r] = s_{rows[r]}
 * (s may be NULL).  Returns 1 for invalid arguments.
 */
int oracle_gemv_rows(int64_t M, int64_t K, const float *A, int64_t lda, const float *x,
                     const int64_t *rows, int64_t nrows, double *y, double *s, int nthreads)
{
    if (M < 0 || K < 0 || lda < K || nrows < 0)
        return 1;
    if ((M > 0 && K > 0 && !A) || (K > 0 && !x) || (nrows > 0 && (!rows || !y)))
        return 1;
    for (int64_t r = 0; r < nrows; ++r)
        if (rows[r] < 0 || rows[r] >= M)
            return 1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int64_t r;
#pragma omp parallel for schedule(dynamic, 4)
    for (r = 0; r < nrows; ++r) {
        const float *a = A + rows[r] * lda;
        double acc = 0.0, mag = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double p = (double)a[k] * (double)x[k];
            acc += p;
            mag += fabs(p);
        }
        y[r] = acc;
        if (s)
            s[r] = mag;
    }
    return 0;
}

/* Every row 0 .. M-1. */
int oracle_gemv(int64_t M, int64_t K, const float *A, int64_t lda, const float *x, double *y, double *s,
                int nthreads)
{
    if (M < 0)
        return 1;
    int64_t *rows = (int64_t *)malloc(sizeof(int64_t) * (size_t)(M > 0 ? M : 1));
    if (!rows)
        return 2;
    for (int64_t i = 0; i < M; ++i)
        rows[i] = i;
    const int rc = oracle_gemv_rows(M, K, A, lda, x, rows, M, y, s, nthreads);
    free(rows);
    return rc;
}
