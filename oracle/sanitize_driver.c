/*
 * sanitize_driver.c -- runs every function of the oracle on small seeded
 * inputs in one process, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_oracle_sanitized.py compiles it
 * together with gpic_oracle.c).  TEST INFRASTRUCTURE, like the oracle.
 *
 * Buffers are allocated to exactly the sizes each function documents, so
 * an access past them, a use after free, a leak or undefined arithmetic in
 * the oracle ends the run with a sanitizer report.  The checks here are
 * only the invariants that need no second implementation (rows of W sum
 * to 1, v stays a probability vector, the uniform vector stops after two
 * updates, k-means labels are contiguous and in range, the kNN graph is
 * symmetric without self loops); the values themselves are pinned by the
 * Python pin suite.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int32_t orc_num_threads(void);
void orc_affinity_cosine_rows(const float *X, int64_t n, int32_t d, int64_t row0,
                              int64_t nrows, double *out);
void orc_affinity_rows(const float *X, int64_t n, int32_t d, double sigma, int64_t row0,
                       int64_t nrows, double *out);
void orc_degree_rows(const float *X, int64_t n, int32_t d, double sigma, const int64_t *rows,
                     int64_t nrows, double *deg);
int64_t orc_degree_normalize(double *A, int64_t n, double *degree, double *v0);
int64_t orc_degree_normalize_csr(const int64_t *row_ptr, const int32_t *col, const double *a,
                                 int64_t n, double *w, double *degree, double *v0);
int64_t orc_degree_onthefly(const float *X, int64_t n, int32_t d, double sigma,
                            double *degree, double *v0);
int32_t orc_power_iterate_dense(const double *W, int64_t n, int32_t mode, int32_t max_iter,
                                double eps, double *v, double *delta, double *stats,
                                int32_t *converged);
int32_t orc_power_iterate_csr(const int64_t *row_ptr, const int32_t *col, const double *w,
                              int64_t n, int32_t mode, int32_t max_iter, double eps,
                              double *v, double *delta, double *stats, int32_t *converged);
int32_t orc_power_iterate_onthefly(const float *X, int64_t n, int32_t d, double sigma,
                                   const double *degree, int32_t mode, int32_t max_iter,
                                   double eps, double *v, double *delta, double *stats,
                                   int32_t *converged);
void orc_matvec_onthefly_rows(const float *X, int64_t n, int32_t d, double sigma,
                              const double *degree, const double *v, const int64_t *rows,
                              int64_t nrows, double *y);
int32_t orc_kmeans1d(const double *v, int64_t n, int32_t k, int32_t method, int32_t *labels,
                     double *centroids, int32_t *k_eff, double *cost_out);
int64_t orc_knn_graph(const float *X, int64_t n, int32_t d, int32_t k, double sigma,
                      int64_t *row_ptr, int32_t *col, float *val);
int32_t orc_knn_rows(const float *X, int64_t n, int32_t d, int32_t k, double sigma,
                     const int64_t *rows, int64_t m, int64_t *nbr, double *d2, float *w);

static int failures = 0;

#define EXPECT(cond, ...)                                                      \
    do {                                                                       \
        if (!(cond)) {                                                         \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);               \
            fprintf(stderr, __VA_ARGS__);                                      \
            fprintf(stderr, "\n");                                             \
            ++failures;                                                        \
        }                                                                      \
    } while (0)

/* xorshift64*: deterministic inputs without the C library's rand() */
static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform01(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 2685821657736338717ull) >> 11) * 0x1.0p-53;
}

static void *xmalloc(size_t bytes)
{
    void *p = malloc(bytes ? bytes : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

/* n points in d dimensions around k centres, float32 */
static float *points(int64_t n, int32_t d, int32_t k, double spread)
{
    float *X = xmalloc((size_t)(n * d) * sizeof(float));
    for (int64_t i = 0; i < n; ++i)
        for (int32_t c = 0; c < d; ++c)
            X[i * d + c] = (float)(spread * (double)(i % k) + uniform01() - 0.5);
    return X;
}

static double l1(const double *x, int64_t n)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i)
        s += fabs(x[i]);
    return s;
}

static void run_dense(int64_t n, int32_t d)
{
    float *X = points(n, d, 3, 4.0);
    const double sigma = 1.25;
    double *A = xmalloc((size_t)(n * n) * sizeof(double));
    orc_affinity_rows(X, n, d, sigma, 0, n, A);
    double *deg = xmalloc((size_t)n * sizeof(double));
    double *v0 = xmalloc((size_t)n * sizeof(double));
    const int64_t nz = orc_degree_normalize(A, n, deg, v0);
    EXPECT(nz == 0, "dense n=%lld: %lld zero-degree rows", (long long)n, (long long)nz);
    for (int64_t i = 0; i < n; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j)
            s += A[i * n + j];
        EXPECT(fabs(s - 1.0) < 1e-12, "row %lld of W sums to %.17g", (long long)i, s);
    }
    EXPECT(fabs(l1(v0, n) - 1.0) < 1e-12, "v0 does not sum to 1");

    /* degrees of a few rows recomputed on the fly */
    int64_t rows[3] = {0, n / 2, n - 1};
    double dr[3];
    orc_degree_rows(X, n, d, sigma, rows, 3, dr);
    for (int r = 0; r < 3; ++r)
        EXPECT(fabs(dr[r] - deg[rows[r]]) <= 1e-12 * deg[rows[r]], "degree_rows");

    double *v = xmalloc((size_t)n * sizeof(double));
    double *delta = xmalloc((size_t)n * sizeof(double));
    double *stats = xmalloc(40 * sizeof(double));
    int32_t conv = 0;
    memcpy(v, v0, (size_t)n * sizeof(double));
    memcpy(delta, v0, (size_t)n * sizeof(double));
    int32_t it = orc_power_iterate_dense(A, n, 0, 40, 0.0, v, delta, stats, &conv);
    EXPECT(it == 40 && !conv, "dense fixed: %d updates", it);
    EXPECT(fabs(l1(v, n) - 1.0) < 1e-12, "v after 40 updates does not sum to 1");

    /* the uniform vector is a fixed point: two updates in converge mode */
    for (int64_t i = 0; i < n; ++i)
        v[i] = delta[i] = 1.0 / (double)n;
    it = orc_power_iterate_dense(A, n, 1, 40, 1e-5 / (double)n, v, delta, stats, &conv);
    EXPECT(it == 2 && conv, "uniform start: %d updates, converged %d", it, conv);

    /* the on-the-fly operator over the same points */
    double *degf = xmalloc((size_t)n * sizeof(double));
    double *v0f = xmalloc((size_t)n * sizeof(double));
    EXPECT(orc_degree_onthefly(X, n, d, sigma, degf, v0f) == 0, "on-the-fly zero rows");
    for (int64_t i = 0; i < n; ++i)
        EXPECT(fabs(degf[i] - deg[i]) <= 1e-12 * deg[i], "on-the-fly degree %lld",
               (long long)i);
    memcpy(v, v0f, (size_t)n * sizeof(double));
    memcpy(delta, v0f, (size_t)n * sizeof(double));
    it = orc_power_iterate_onthefly(X, n, d, sigma, degf, 0, 5, 0.0, v, delta, stats, &conv);
    EXPECT(it == 5, "on-the-fly fixed: %d updates", it);
    double y[3];
    orc_matvec_onthefly_rows(X, n, d, sigma, degf, v, rows, 3, y);
    for (int r = 0; r < 3; ++r)
        EXPECT(isfinite(y[r]) && y[r] >= 0.0, "on-the-fly product row");

    /* cosine rows */
    orc_affinity_cosine_rows(X, n, d, 1, n - 1, A);
    for (int64_t i = 0; i < (n - 1) * n; ++i)
        EXPECT(A[i] >= 0.0 && A[i] <= 1.0, "cosine entry out of [0, 1]");

    /* k-means on the iterate, both methods, several k */
    int32_t *lab = xmalloc((size_t)n * sizeof(int32_t));
    for (int32_t k = 1; k <= 4; ++k)
        for (int32_t method = 0; method <= 1; ++method) {
            double cent[4];
            int32_t ke = 0;
            double cost = 0.0;
            EXPECT(orc_kmeans1d(v, n, k, method, lab, cent, &ke, &cost) == 0, "kmeans");
            EXPECT(ke >= 1 && ke <= k && cost >= 0.0, "kmeans k_eff %d cost %g", ke, cost);
            for (int64_t i = 0; i < n; ++i)
                EXPECT(lab[i] >= 0 && lab[i] < ke, "label out of range");
            for (int32_t c = 1; c < ke; ++c)
                EXPECT(cent[c - 1] < cent[c], "centroids not ascending");
        }
    free(lab);
    free(degf);
    free(v0f);
    free(stats);
    free(delta);
    free(v);
    free(v0);
    free(deg);
    free(A);
    free(X);
}

static void run_sparse(int64_t n, int32_t d, int32_t k)
{
    float *X = points(n, d, 4, 6.0);
    int64_t *rp = xmalloc((size_t)(n + 1) * sizeof(int64_t));
    int32_t *col = xmalloc((size_t)(2 * n * k) * sizeof(int32_t));
    float *val = xmalloc((size_t)(2 * n * k) * sizeof(float));
    const int64_t nnz = orc_knn_graph(X, n, d, k, 1.0, rp, col, val);
    EXPECT(nnz >= n * k && nnz <= 2 * n * k, "knn nnz %lld", (long long)nnz);
    EXPECT(rp[0] == 0 && rp[n] == nnz, "row_ptr ends");
    for (int64_t i = 0; i < n; ++i) {
        EXPECT(rp[i + 1] - rp[i] >= k, "row %lld has fewer than k entries", (long long)i);
        for (int64_t p = rp[i]; p < rp[i + 1]; ++p) {
            const int32_t j = col[p];
            EXPECT(j >= 0 && j < n && j != i, "bad column");
            EXPECT(p == rp[i] || col[p - 1] < j, "row not sorted");
            int found = 0;                       /* union symmetry: (j, i) stored too */
            for (int64_t q = rp[j]; q < rp[j + 1]; ++q)
                found |= (col[q] == (int32_t)i && val[q] == val[p]);
            EXPECT(found, "edge (%lld, %d) without its mirror", (long long)i, j);
        }
    }
    {                                            /* the neighbour lists alone */
        const int64_t rows[3] = {0, n / 2, n - 1};
        int64_t *nb = xmalloc((size_t)(3 * k) * sizeof(int64_t));
        double *d2 = xmalloc((size_t)(3 * k) * sizeof(double));
        float *wk = xmalloc((size_t)(3 * k) * sizeof(float));
        EXPECT(orc_knn_rows(X, n, d, k, 1.0, rows, 3, nb, d2, wk) == 0, "knn rows");
        for (int t = 0; t < 3; ++t)
            for (int32_t s = 0; s < k; ++s) {
                int found = 0;                   /* each neighbour is in the row */
                for (int64_t q = rp[rows[t]]; q < rp[rows[t] + 1]; ++q)
                    found |= (col[q] == (int32_t)nb[t * k + s] && val[q] == wk[t * k + s]);
                EXPECT(found, "neighbour %d of row %lld missing", s, (long long)rows[t]);
                EXPECT(s == 0 || d2[t * k + s - 1] <= d2[t * k + s], "neighbours not ordered");
            }
        const int64_t bad[1] = {n};
        EXPECT(orc_knn_rows(X, n, d, k, 1.0, bad, 1, nb, d2, wk) == -1, "row out of range");
        free(wk);
        free(d2);
        free(nb);
    }
    double *a = xmalloc((size_t)nnz * sizeof(double));
    double *w = xmalloc((size_t)nnz * sizeof(double));
    for (int64_t p = 0; p < nnz; ++p)
        a[p] = (double)val[p];
    double *deg = xmalloc((size_t)n * sizeof(double));
    double *v = xmalloc((size_t)n * sizeof(double));
    double *delta = xmalloc((size_t)n * sizeof(double));
    double stats[30];
    int32_t conv = 0;
    EXPECT(orc_degree_normalize_csr(rp, col, a, n, w, deg, v) == 0, "csr zero rows");
    memcpy(delta, v, (size_t)n * sizeof(double));
    const int32_t it = orc_power_iterate_csr(rp, col, w, n, 1, 30, 1e-5 / (double)n, v, delta,
                                             stats, &conv);
    EXPECT(it >= 1 && it <= 30, "csr updates %d", it);
    EXPECT(fabs(l1(v, n) - 1.0) < 1e-12, "csr v does not sum to 1");
    free(delta);
    free(v);
    free(deg);
    free(w);
    free(a);
    free(val);
    free(col);
    free(rp);
    free(X);
}

int main(void)
{
    const int32_t threads = orc_num_threads();
    EXPECT(threads >= 1, "thread count %d", threads);
    run_dense(2, 1);
    run_dense(7, 2);
    run_dense(64, 3);
    run_dense(301, 17);
    run_sparse(40, 2, 3);
    run_sparse(257, 8, 8);
    /* k-means edge cases: duplicates (5 distinct values, -0 equal to 0), k above that */
    const double dup[9] = {3.0, -0.0, 0.0, 3.0, 1e-300, -40.0, 7.0, 3.0, 7.0};
    int32_t lab[9];
    double cent[9];
    for (int32_t k = 1; k <= 9; ++k)
        for (int32_t method = 0; method <= 1; ++method) {
            int32_t ke = 0;
            double cost = 0.0;
            EXPECT(orc_kmeans1d(dup, 9, k, method, lab, cent, &ke, &cost) == 0, "kmeans dup");
            EXPECT(ke == (k < 5 ? k : 5), "distinct values: k_eff %d for k %d", ke, k);
        }
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("sanitized oracle run: all checks passed (%d threads)\n", threads);
    return 0;
}
