/*
 * Oracle for the dense GEMM hot path: C = A * B with 16-bit (bf16 or fp16)
 * inputs, evaluated in IEEE fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header or constant with the
 * GPU path.
 *
 * What it computes (the plain definition).  The paper's starting point is a
 * simple sequential GEMM program whose meaning every optimised schedule must
 * preserve (Introduction; Section 2.3, chain of equivalence).  For every
 * output element
 *
 *     C[i][j] = sum_{k = 0 .. K-1} dec(A[i*lda + k]) * dec(B[k*ldb + j])
 *
 * with the sum taken in ascending k, in fp64.  Alongside it the oracle returns
 * the tolerance scale
 *
 *     S[i][j] = sum_k | dec(A[i][k]) * dec(B[k][j]) |
 *
 * against which a GPU result is accepted when |C_gpu - C| <= 1e-4 * S.
 *
 * Exactness.  dec() is exact (every bf16 / fp16 value is a double).  Each
 * product is exact in fp64: bf16 significands carry 8 bits and fp16 11 bits,
 * so a product has at most 22 significant bits and its exponent stays inside
 * the fp64 normal range.  The only rounding is the fp64 summation, bounded by
 * (K-1) * 2^-53 * S.
 *
 * Layout: row-major with leading dimensions in elements, as the GPU library
 * takes them.  The "row" entry point computes whole rows of C with the k loop
 * outside the j loop; every element still receives its terms in ascending k,
 * so the per-element summation order is exactly the definition's.
 *
 * Build with -ffp-contract=off and without -ffast-math: no reassociation.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_BF16 = 0, ORACLE_FP16 = 1 };

/*
 * bfloat16: sign bit, 8 exponent bits (bias 127), 7 fraction bits; the same
 * field widths as the upper half of an IEEE binary32.
 *   exponent field 0:   (-1)^s * 2^-126 * (f / 128)            (zero/subnormal)
 *   exponent field 255: infinity (f == 0) or NaN
 *   otherwise:          (-1)^s * 2^(e - 127) * (1 + f / 128)
 */
double oracle_decode_bf16(uint16_t bits)
{
    int s = (bits >> 15) & 1;
    int e = (bits >> 7) & 0xFF;
    int f = bits & 0x7F;
    double v;
    if (e == 0)
        v = ldexp((double)f, -126 - 7);
    else if (e == 0xFF)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(128 + f), e - 127 - 7);
    return s ? -v : v;
}

/*
 * IEEE 754 binary16: sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 *   exponent field 0:  (-1)^s * 2^-14 * (f / 1024)             (zero/subnormal)
 *   exponent field 31: infinity (f == 0) or NaN
 *   otherwise:         (-1)^s * 2^(e - 15) * (1 + f / 1024)
 */
double oracle_decode_fp16(uint16_t bits)
{
    int s = (bits >> 15) & 1;
    int e = (bits >> 10) & 0x1F;
    int f = bits & 0x3FF;
    double v;
    if (e == 0)
        v = ldexp((double)f, -14 - 10);
    else if (e == 0x1F)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 15 - 10);
    return s ? -v : v;
}

static double dec(uint16_t bits, int dtype)
{
    return dtype == ORACLE_BF16 ? oracle_decode_bf16(bits) : oracle_decode_fp16(bits);
}

/* Decode `n` stored values into doubles. */
int oracle_decode(const uint16_t *src, int64_t n, int dtype, double *dst)
{
    if (n < 0 || (n > 0 && (!src || !dst)) || (dtype != ORACLE_BF16 && dtype != ORACLE_FP16))
        return 1;
    for (int64_t t = 0; t < n; ++t)
        dst[t] = dec(src[t], dtype);
    return 0;
}

static int bad_args(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda,
                    const uint16_t *B, int64_t ldb, int dtype)
{
    if (M < 0 || N < 0 || K < 0)
        return 1;
    if (lda < K || ldb < N)
        return 1;
    if (dtype != ORACLE_BF16 && dtype != ORACLE_FP16)
        return 1;
    if ((M > 0 && K > 0 && !A) || (K > 0 && N > 0 && !B))
        return 1;
    return 0;
}

/*
 * Whole rows of C and S.  rows[r] (0 <= rows[r] < M) selects a row of C; the
 * result goes to C[r*ldc + j] and S[r*lds + j] for j < N.  S may be NULL.
 * B is decoded once into a K x N fp64 array; each selected row is then the
 * ascending-k sum of its terms.  Rows are independent and spread over
 * `nthreads` OpenMP threads (0 = the OpenMP default).
 */
int oracle_gemm_rows(int64_t M, int64_t N, int64_t K,
                     const uint16_t *A, int64_t lda,
                     const uint16_t *B, int64_t ldb, int dtype,
                     const int64_t *rows, int64_t nrows,
                     double *C, int64_t ldc, double *S, int64_t lds, int nthreads)
{
    if (bad_args(M, N, K, A, lda, B, ldb, dtype) || nrows < 0 || ldc < N)
        return 1;
    if (S && lds < N)
        return 1;
    if (nrows > 0 && (!rows || (N > 0 && !C)))
        return 1;
    for (int64_t r = 0; r < nrows; ++r)
        if (rows[r] < 0 || rows[r] >= M)
            return 1;
    if (nrows == 0 || N == 0)
        return 0;

    double *Bd = NULL;
    if (K > 0) {
        Bd = (double *)malloc(sizeof(double) * (size_t)K * (size_t)N);
        if (!Bd)
            return 2;
        for (int64_t k = 0; k < K; ++k)
            for (int64_t j = 0; j < N; ++j)
                Bd[k * N + j] = dec(B[k * ldb + j], dtype);
    }
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int64_t r;
#pragma omp parallel for schedule(dynamic, 1)
    for (r = 0; r < nrows; ++r) {
        const int64_t i = rows[r];
        double *c = C + r * ldc;
        double *s = S ? S + r * lds : NULL;
        for (int64_t j = 0; j < N; ++j) {
            c[j] = 0.0;
            if (s)
                s[j] = 0.0;
        }
        for (int64_t k = 0; k < K; ++k) {
            const double a = dec(A[i * lda + k], dtype);
            const double *b = Bd + k * N;
            for (int64_t j = 0; j < N; ++j) {
                const double p = a * b[j];
                c[j] += p;
                if (s)
                    s[j] += fabs(p);
            }
        }
    }
    free(Bd);
    return 0;
}

/* The full product: every row 0..M-1. */
int oracle_gemm(int64_t M, int64_t N, int64_t K,
                const uint16_t *A, int64_t lda,
                const uint16_t *B, int64_t ldb, int dtype,
                double *C, int64_t ldc, double *S, int64_t lds, int nthreads)
{
    if (M < 0)
        return 1;
    int64_t *rows = (int64_t *)malloc(sizeof(int64_t) * (size_t)(M > 0 ? M : 1));
    if (!rows)
        return 2;
    for (int64_t i = 0; i < M; ++i)
        rows[i] = i;
    int rc = oracle_gemm_rows(M, N, K, A, lda, B, ldb, dtype, rows, M, C, ldc, S, lds, nthreads);
    free(rows);
    return rc;
}

/*
 * Scattered entries: out_c[t] = C[rows[t]][cols[t]], out_s[t] = S[...] (out_s
 * may be NULL).  Each entry is one ascending-k dot product read straight from
 * the stored bits; used to check outputs of problems too large to form whole.
 */
int oracle_gemm_entries(int64_t M, int64_t N, int64_t K,
                        const uint16_t *A, int64_t lda,
                        const uint16_t *B, int64_t ldb, int dtype,
                        const int64_t *rows, const int64_t *cols, int64_t count,
                        double *out_c, double *out_s, int nthreads)
{
    if (bad_args(M, N, K, A, lda, B, ldb, dtype) || count < 0)
        return 1;
    if (count > 0 && (!rows || !cols || !out_c))
        return 1;
    for (int64_t t = 0; t < count; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N)
            return 1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int64_t t;
#pragma omp parallel for schedule(dynamic, 16)
    for (t = 0; t < count; ++t) {
        const int64_t i = rows[t], j = cols[t];
        double c = 0.0, s = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double p = dec(A[i * lda + k], dtype) * dec(B[k * ldb + j], dtype);
            c += p;
            s += fabs(p);
        }
        out_c[t] = c;
        if (out_s)
            out_s[t] = s;
    }
    return 0;
}

/* Number of threads an OpenMP parallel region would use with `nthreads`. */
int oracle_thread_count(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
    return n;
#else
    (void)nthreads;
    return 1;
#endif
}
