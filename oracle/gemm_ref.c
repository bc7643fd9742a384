/*
 * Oracle: C = A * B over bf16 inputs, accumulated in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library includes, links or
 * calls this file; it is compiled on its own with gcc into oracle/_gemm_ref.so.
 *
 * Definition followed: the problem statement of Section II.A (A is M x K, B is
 * K x N, C is M x N) with the overwrite semantics of Listing 1 (the C block is
 * zeroed before the first contraction, reading A7):
 *     C[i][j] = sum_{k=0}^{K-1} a[i][k] * b[k][j]
 * where a and b are the bf16 inputs taken as exact real numbers.  Every product
 * of two bf16 values is exact in fp64 (8+8 significant bits), and the sum is
 * accumulated in fp64 in ascending k for every element.
 *
 * Alongside C it produces R[i][j] = sum_k |a[i][k]| * |b[k][j]|, the scale the
 * elementwise tolerance is stated against.
 *
 * Layout: row-major, A[i][k] at A[i*lda + k], B[k][j] at B[k*ldb + j]; bf16 is
 * passed as its 16-bit pattern.  Outputs are dense fp64 (leading dimension N
 * for the row version, one value per point for the point version).
 *
 * Loop order: i, then k, then j; each element therefore sees its k terms in
 * ascending order.  Rows are independent and shared among OpenMP threads.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* bf16 -> fp64, exact: a bf16 pattern is the upper half of an IEEE binary32. */
static double bf16_to_f64(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Rows [row0, row0 + nrows) of C and R, each written to out[(i - row0) * N + j]. */
void gemm_ref_rows(int64_t row0, int64_t nrows, int64_t N, int64_t K,
                   const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                   double *C, double *R) {
    int64_t r;
#pragma omp parallel for schedule(dynamic, 1)
    for (r = 0; r < nrows; ++r) {
        const int64_t i = row0 + r;
        double *c = C + r * N;
        double *s = R + r * N;
        int64_t j, k;
        for (j = 0; j < N; ++j) { c[j] = 0.0; s[j] = 0.0; }
        for (k = 0; k < K; ++k) {
            const double a = bf16_to_f64(A[i * lda + k]);
            const double aa = fabs(a);
            const uint16_t *brow = B + k * ldb;
            for (j = 0; j < N; ++j) {
                const double b = bf16_to_f64(brow[j]);
                c[j] += a * b;
                s[j] += aa * fabs(b);
            }
        }
    }
}

/* Single elements: out[p] = C[rows[p]][cols[p]] (and R likewise). */
void gemm_ref_points(int64_t npts, const int64_t *rows, const int64_t *cols, int64_t K,
                     const uint16_t *A, int64_t lda, const uint16_t *B, int64_t ldb,
                     double *C, double *R) {
    int64_t p;
#pragma omp parallel for schedule(static)
    for (p = 0; p < npts; ++p) {
        const int64_t i = rows[p], j = cols[p];
        double c = 0.0, s = 0.0;
        int64_t k;
        for (k = 0; k < K; ++k) {
            const double a = bf16_to_f64(A[i * lda + k]);
            const double b = bf16_to_f64(B[k * ldb + j]);
            c += a * b;
            s += fabs(a) * fabs(b);
        }
        C[p] = c;
        R[p] = s;
    }
}

/* The number of OpenMP threads a parallel region would use (for reporting). */
int gemm_ref_threads(void) {
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
