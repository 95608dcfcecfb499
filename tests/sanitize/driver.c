/*
 * Host driver for the sanitizer test: runs every function of the CPU oracle
 * and of the seeded input generator on small, ragged shapes under
 * AddressSanitizer and UndefinedBehaviorSanitizer (gcc), and checks results
 * that follow from the definitions alone (A = I, A = all-ones, the adjoint
 * identity, generator determinism and range).  Exit status 0 = all passed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_matvec(int64_t m, int64_t n, const double* A, const double* x, double* y);
void oracle_matvec_t(int64_t m, int64_t n, const double* A, const double* w, double* z);
void oracle_ata_x(int64_t m, int64_t n, const double* A, const double* x, double* t, double* y);
void oracle_bicg(int64_t m, int64_t n, const double* A, const double* p, const double* r, double* q, double* s);
void oracle_axpby_mv(int64_t m, int64_t n, double alpha, const double* A, double beta, const double* B,
                     const double* x, double* y);
double oracle_reduce_sum(int64_t n, const double* x);
void oracle_vector_add(int64_t n, const double* a, const double* b, double* c);
void oracle_gemver(int64_t m, int64_t n, double alpha, double beta, const double* A, const double* u1,
                   const double* v1, const double* u2, const double* v2, const double* y, const double* z,
                   double* Ahat, double* x, double* w);
void mep_dg_bits(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, uint64_t* out);
void mep_dg_uniform_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out);
void mep_dg_uniform_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out);
void mep_dg_normal_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out);
void mep_dg_normal_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out);
void mep_dg_ternary_f32(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, float* out);
void mep_dg_ternary_f64(uint64_t seed, uint64_t array_id, uint64_t first, int64_t count, double* out);

static int failures = 0;
#define CHECK(c, ...) do { if (!(c)) { fprintf(stderr, __VA_ARGS__); fputc('\n', stderr); ++failures; } } while (0)

static double* arr(int64_t n) { return (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double)); }

static void shape(int64_t m, int64_t n, uint64_t seed)
{
    double *A = arr(m * n), *B = arr(m * n), *x = arr(n), *w = arr(m), *u1 = arr(m), *u2 = arr(m);
    double *v1 = arr(n), *v2 = arr(n), *z = arr(n), *yv = arr(m);
    double *ym = arr(m), *zt = arr(n), *t = arr(m), *ya = arr(n), *q = arr(m), *s = arr(n), *g = arr(m);
    double *Ahat = arr(m * n), *xg = arr(n), *wg = arr(m);
    mep_dg_uniform_f64(seed, 0, 0, m * n, A);
    mep_dg_normal_f64(seed, 1, 0, m * n, B);
    mep_dg_uniform_f64(seed, 2, 0, n, x);
    mep_dg_uniform_f64(seed, 3, 0, m, w);
    mep_dg_uniform_f64(seed, 4, 0, m, u1);
    mep_dg_uniform_f64(seed, 5, 0, m, u2);
    mep_dg_uniform_f64(seed, 6, 0, n, v1);
    mep_dg_uniform_f64(seed, 7, 0, n, v2);
    mep_dg_uniform_f64(seed, 8, 0, n, z);
    mep_dg_uniform_f64(seed, 9, 0, m, yv);

    oracle_matvec(m, n, A, x, ym);
    oracle_matvec_t(m, n, A, w, zt);
    oracle_ata_x(m, n, A, x, t, ya);
    oracle_bicg(m, n, A, x, w, q, s);
    oracle_axpby_mv(m, n, 1.5, A, 1.2, B, x, g);
    oracle_gemver(m, n, 1.5, 1.2, A, u1, v1, u2, v2, yv, z, Ahat, xg, wg);
    double sum = oracle_reduce_sum(m, w);
    double* c = arr(m);
    oracle_vector_add(m, w, u1, c);

    /* adjoint identity w.(Ax) = (A^T w).x, within a loose bound */
    double l = 0, r = 0, scale = 0;
    for (int64_t i = 0; i < m; ++i) l += w[i] * ym[i];
    for (int64_t j = 0; j < n; ++j) r += zt[j] * x[j];
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) scale += fabs(w[i] * A[i * n + j] * x[j]);
    CHECK(fabs(l - r) <= 1e-12 * (scale + 1), "adjoint %lldx%lld: %g vs %g", (long long)m, (long long)n, l, r);
    /* BICG equals the two separate products bit for bit; ATAX's t is A x */
    for (int64_t i = 0; i < m; ++i) CHECK(q[i] == ym[i] && t[i] == ym[i], "bicg/ata q or t row %lld", (long long)i);
    for (int64_t j = 0; j < n; ++j) CHECK(s[j] == zt[j], "bicg s col %lld", (long long)j);
    double sref = 0;
    for (int64_t i = 0; i < m; ++i) {
        sref += w[i];
        CHECK(c[i] == w[i] + u1[i], "vector add %lld", (long long)i);
    }
    CHECK(fabs(sum - sref) <= 1e-12 * (double)m, "sum");

    /* A = I (m x n, ones on the diagonal): A x = x (padded), A^T w = w (padded) */
    for (int64_t i = 0; i < m * n; ++i) A[i] = 0.0;
    for (int64_t i = 0; i < m && i < n; ++i) A[i * n + i] = 1.0;
    oracle_matvec(m, n, A, x, ym);
    for (int64_t i = 0; i < m; ++i) CHECK(ym[i] == (i < n ? x[i] : 0.0), "identity matvec %lld", (long long)i);
    oracle_matvec_t(m, n, A, w, zt);
    for (int64_t j = 0; j < n; ++j) CHECK(zt[j] == (j < m ? w[j] : 0.0), "identity matvec_t %lld", (long long)j);

    free(A); free(B); free(x); free(w); free(u1); free(u2); free(v1); free(v2); free(z); free(yv);
    free(ym); free(zt); free(t); free(ya); free(q); free(s); free(g); free(Ahat); free(xg); free(wg); free(c);
}

static void generator(void)
{
    const int64_t n = 1001;
    uint64_t* b1 = (uint64_t*)malloc(n * sizeof(uint64_t));
    uint64_t* b2 = (uint64_t*)malloc(n * sizeof(uint64_t));
    mep_dg_bits(7, 3, 0, n, b1);
    mep_dg_bits(7, 3, 10, n - 10, b2);
    for (int64_t k = 0; k + 10 < n; ++k) CHECK(b1[k + 10] == b2[k], "counter form at %lld", (long long)k);
    float* f = (float*)malloc(n * sizeof(float));
    double* d = arr(n);
    mep_dg_uniform_f32(1, 0, 0, n, f);
    for (int64_t k = 0; k < n; ++k) CHECK(f[k] >= -1.0f && f[k] < 1.0f, "uniform f32 range");
    mep_dg_uniform_f64(1, 0, 0, n, d);
    for (int64_t k = 0; k < n; ++k) CHECK(d[k] >= -1.0 && d[k] < 1.0, "uniform f64 range");
    mep_dg_normal_f32(1, 0, 0, n, f);
    mep_dg_normal_f64(1, 0, 0, n, d);
    for (int64_t k = 0; k < n; ++k) CHECK(isfinite(f[k]) && isfinite(d[k]), "normal finite");
    mep_dg_ternary_f32(1, 0, 0, n, f);
    mep_dg_ternary_f64(1, 0, 0, n, d);
    for (int64_t k = 0; k < n; ++k) CHECK((f[k] == -1 || f[k] == 0 || f[k] == 1) && (d[k] == -1 || d[k] == 0 || d[k] == 1), "ternary");
    mep_dg_uniform_f64(1, 0, 0, 0, d);  /* empty draw writes nothing */
    /* a draw from counter 10 on equals the tail of the draw from 0 */
    double* d2 = arr(n);
    mep_dg_uniform_f64(1, 0, 0, n, d);
    mep_dg_uniform_f64(1, 0, 10, n - 10, d2);
    for (int64_t k = 0; k + 10 < n; ++k) CHECK(d[k + 10] == d2[k], "uniform from counter 10 at %lld", (long long)k);
    mep_dg_normal_f32(1, 0, 0, n, f);
    float* f2 = (float*)malloc(n * sizeof(float));
    mep_dg_normal_f32(1, 0, 10, n - 10, f2);
    for (int64_t k = 0; k + 10 < n; ++k) CHECK(f[k + 10] == f2[k], "normal from counter 10 at %lld", (long long)k);
    free(d2); free(f2);
    free(b1); free(b2); free(f); free(d);
}

int main(void)
{
    const int64_t shapes[][2] = {{1, 1}, {1, 9}, {9, 1}, {3, 5}, {17, 33}, {64, 64}, {65, 7}};
    for (size_t k = 0; k < sizeof shapes / sizeof shapes[0]; ++k)
        shape(shapes[k][0], shapes[k][1], 100 + k);
    generator();
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("sanitized oracle and generator: all checks passed\n");
    return 0;
}
