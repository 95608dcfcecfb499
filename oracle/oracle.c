/*
 * CPU ORACLE for the dense matrix-vector family -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  The product path (the HIP library and its binding)
 * never calls it; the two share no code, header, helper or constant.
 *
 * What it computes.  The paper evaluates its framework on PolyBench kernels
 * named ATAX, BICG and GESUMMV (Tables 1 and 2, Sec. 4.2) but never writes
 * out what they compute; the definitions used here are the textbook ones for
 * those names: the matrix-vector product y = A x, the transposed product
 * z = A^T w, the BICG pair q = A p, s = A^T r, the chain y = A^T (A x)
 * (ATAX) and the scaled sum y = alpha A x + beta B x (GESUMMV).
 *
 * How.  Plain loops in fp64: every input is promoted exactly to double before
 * this library sees it, every output element is one sum taken in ascending
 * index order by a single thread, each product is rounded once and then added
 * (no fused multiply-add: built with -ffp-contract=off).  OpenMP only splits
 * the set of output elements between threads, so the result is bit-identical
 * for any thread count.
 *
 * GEMVER, which Tables 1-2 also name without a definition, follows the BLAS
 * Technical Forum standard: Ahat = A + u1 v1^T + u2 v2^T, x = beta Ahat^T y + z,
 * w = alpha Ahat x.
 *
 * Two further streaming kernels of the paper's AMD APP SDK table (Table 3,
 * "reduction" and "vectoradd") are defined here too: the sum of a vector and
 * the elementwise sum of two vectors.
 *
 * Layout.  A and B are row-major and contiguous, m rows by n columns:
 * A_ij = A[i*n + j].  x, p have length n; w, r, t, q have length m; z, s and
 * the ATAX output y have length n; the outputs of y = A x and of the scaled
 * sum have length m.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared oracle.c
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads the oracle uses (OpenMP's current setting). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* y_i = sum_{j=0}^{n-1} A_ij x_j  (matrix-vector product, length m). */
void oracle_matvec(int64_t m, int64_t n, const double* A, const double* x, double* y)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double acc = 0.0;
        for (int64_t j = 0; j < n; ++j)
            acc += A[i * n + j] * x[j];
        y[i] = acc;
    }
}

/* z_j = sum_{i=0}^{m-1} A_ij w_i  (transposed product, length n).
 * Each thread owns a contiguous strip of columns and sweeps all rows, so
 * z_j is still summed over ascending i by one thread. */
void oracle_matvec_t(int64_t m, int64_t n, const double* A, const double* w, double* z)
{
#pragma omp parallel
    {
        int64_t nt = 1, tid = 0;
#ifdef _OPENMP
        nt = omp_get_num_threads();
        tid = omp_get_thread_num();
#endif
        int64_t j0 = n * tid / nt;
        int64_t j1 = n * (tid + 1) / nt;
        for (int64_t j = j0; j < j1; ++j)
            z[j] = 0.0;
        for (int64_t i = 0; i < m; ++i)
            for (int64_t j = j0; j < j1; ++j)
                z[j] += A[i * n + j] * w[i];
    }
}

/* ATAX: t = A x (kept in fp64, never rounded to the input type), then
 * y = A^T t.  t may be NULL when the caller does not want it. */
void oracle_ata_x(int64_t m, int64_t n, const double* A, const double* x, double* t, double* y)
{
    double* tt = t;
    if (tt == NULL) {
        tt = (double*)malloc((size_t)(m > 0 ? m : 1) * sizeof(double));
        if (tt == NULL)
            abort();
    }
    oracle_matvec(m, n, A, x, tt);
    oracle_matvec_t(m, n, A, tt, y);
    if (t == NULL)
        free(tt);
}

/* BICG pair: q = A p and s = A^T r, two independent products of one A. */
void oracle_bicg(int64_t m, int64_t n, const double* A, const double* p, const double* r,
                 double* q, double* s)
{
    oracle_matvec(m, n, A, p, q);
    oracle_matvec_t(m, n, A, r, s);
}

/* GESUMMV: y_i = alpha * (A_i . x) + beta * (B_i . x), both dot products in
 * ascending j, then two products and one sum, each rounded once. */
void oracle_axpby_mv(int64_t m, int64_t n, double alpha, const double* A, double beta,
                     const double* B, const double* x, double* y)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double da = 0.0, db = 0.0;
        for (int64_t j = 0; j < n; ++j)
            da += A[i * n + j] * x[j];
        for (int64_t j = 0; j < n; ++j)
            db += B[i * n + j] * x[j];
        y[i] = alpha * da + beta * db;
    }
}

/* s = sum_{i=0}^{n-1} x_i, ascending i, in fp64 (the "reduction" sample). */
double oracle_reduce_sum(int64_t n, const double* x)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i)
        s += x[i];
    return s;
}

/* c_i = a_i + b_i (the "vectoradd" sample), in fp64. */
void oracle_vector_add(int64_t n, const double* a, const double* b, double* c)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        c[i] = a[i] + b[i];
}

/* GEMVER: Ahat_ij = (A_ij + u1_i v1_j) + u2_i v2_j;
 * x_j = beta * (sum_i Ahat_ij y_i) + z_j  (ascending i);
 * w_i = alpha * (sum_j Ahat_ij x_j)       (ascending j).
 * A, Ahat: m x n; u1, u2, y, w: m; v1, v2, z, x: n.  All fp64. */
void oracle_gemver(int64_t m, int64_t n, double alpha, double beta, const double* A, const double* u1,
                   const double* v1, const double* u2, const double* v2, const double* y,
                   const double* z, double* Ahat, double* x, double* w)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j)
            Ahat[i * n + j] = (A[i * n + j] + u1[i] * v1[j]) + u2[i] * v2[j];
    oracle_matvec_t(m, n, Ahat, y, x);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j)
        x[j] = beta * x[j] + z[j];
    oracle_matvec(m, n, Ahat, x, w);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i)
        w[i] = alpha * w[i];
}
