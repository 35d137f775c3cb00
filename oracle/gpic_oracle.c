/*
 * gpic_oracle.c -- the oracle for Power Iteration Clustering (PIC) as the
 * GPIC paper (arXiv 1604.02700) states it.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check and
 * the benchmark's CPU-baseline leg load this library.  The GPU library never
 * links, includes or calls it, and this file includes nothing of the GPU
 * library: the two share no code.
 *
 * Everything is plain float64 C, written for a reader to check against the
 * paper by eye.  OpenMP only splits independent rows between threads; every
 * row's sum runs sequentially in ascending column order on one thread, and
 * every cross-row reduction (sum of degrees, the L1 norm, the max of the stop
 * statistic) runs serially in ascending row order, so results are bitwise
 * independent of the thread count.
 *
 * What each function follows:
 *   orc_affinity_rows      affinity matrix A of the graph G (section
 *                          "Spectral Cluster"); Gaussian kernel with a zero
 *                          diagonal, the reading taken because the paper
 *                          never writes its kernel down.
 *   orc_affinity_cosine_rows  the cosine similarity of Experiment I (Table 2
 *                          caption), shifted to (1 + cos) / 2 so that A stays
 *                          non-negative, zero diagonal.
 *   orc_degree_normalize   d_ii = sum_j a_ij and W = D^-1 A ("Spectral
 *                          Cluster"); v0 = D / sum(D) (Algorithm 2, the
 *                          Reduction and Norm steps before the loop).
 *   orc_power_iterate_*    the update equation of section "PIC: an
 *                          overview" (W v scaled to unit L1 norm) with the
 *                          acceleration stop of Algorithm 1 (velocity
 *                          |v_new - v| per entry, the first velocity
 *                          compared against v_0; stop once no entry's
 *                          velocity changes by more than eps).
 *   orc_knn_graph          the sparse affinity graph the CSR path takes as
 *                          input: exact k nearest neighbours, union
 *                          symmetrised, Gaussian weights (not in the paper;
 *                          the input of its method in graph form).
 *   orc_knn_rows           the same neighbour lists and weights for listed
 *                          points only.
 *   orc_kmeans1d           "k-means of v" (Algorithm 1, last step), read as
 *                          the exact minimum within-cluster sum of squares
 *                          partition of the scalars v_i (plain O(k n^2)
 *                          dynamic programme, or the same programme with the
 *                          divide-and-conquer argmin search for large n).
 *
 * Pins: every function is checked by the CPU tests against invariants,
 * closed forms, library routines or brute force (row sums, uniform and
 * block-diagonal fixed points, the eigendecomposition closed form, a
 * hand-derived two-node trace, scipy's distance routine, exhaustive
 * partition search).  No function here is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int32_t orc_num_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------ */
/* Affinity                                                            */
/* ------------------------------------------------------------------ */

/* a_ij = exp(-||x_i - x_j||^2 / (2 sigma^2)) for i != j, a_ii = 0.
 * The squared distance is summed from the coordinate differences (not from
 * norms and dot products), every coordinate promoted exactly to float64. */
static double gauss_affinity(const float *X, int32_t d, int64_t i, int64_t j,
                             double two_sigma2)
{
    if (i == j)
        return 0.0;
    const float *xi = X + i * (int64_t)d;
    const float *xj = X + j * (int64_t)d;
    double dist2 = 0.0;
    for (int32_t c = 0; c < d; ++c) {
        double diff = (double)xi[c] - (double)xj[c];
        dist2 += diff * diff;
    }
    return exp(-dist2 / two_sigma2);
}

/* Cosine similarity, read as a_ij = (1 + cos(x_i, x_j)) / 2 for i != j and
 * a_ii = 0, cos = x_i . x_j / (||x_i|| ||x_j||), taken as 0 when either
 * point is the origin.  The shift keeps A >= 0 (cosine alone is negative
 * for points more than a right angle apart, and W = D^-1 A needs A >= 0). */
static double cosine_affinity(const float *X, int32_t d, int64_t i, int64_t j)
{
    if (i == j)
        return 0.0;
    const float *xi = X + i * (int64_t)d;
    const float *xj = X + j * (int64_t)d;
    double dot = 0.0, ni = 0.0, nj = 0.0;
    for (int32_t c = 0; c < d; ++c) {
        const double a = (double)xi[c], b = (double)xj[c];
        dot += a * b;
        ni += a * a;
        nj += b * b;
    }
    if (ni == 0.0 || nj == 0.0)
        return 0.5;
    return 0.5 * (1.0 + dot / (sqrt(ni) * sqrt(nj)));
}

/* Rows row0 .. row0+nrows-1 of the cosine A, written to out[r * n + j]. */
void orc_affinity_cosine_rows(const float *X, int64_t n, int32_t d, int64_t row0,
                              int64_t nrows, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nrows; ++r)
        for (int64_t j = 0; j < n; ++j)
            out[r * n + j] = cosine_affinity(X, d, row0 + r, j);
}

/* Rows row0 .. row0+nrows-1 of A, written to out[r * n + j]. */
void orc_affinity_rows(const float *X, int64_t n, int32_t d, double sigma,
                       int64_t row0, int64_t nrows, double *out)
{
    const double two_sigma2 = 2.0 * sigma * sigma;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nrows; ++r)
        for (int64_t j = 0; j < n; ++j)
            out[r * n + j] = gauss_affinity(X, d, row0 + r, j, two_sigma2);
}

/* Degrees of the listed rows, d_i = sum_j a_ij, with A recomputed. */
void orc_degree_rows(const float *X, int64_t n, int32_t d, double sigma,
                     const int64_t *rows, int64_t nrows, double *deg)
{
    const double two_sigma2 = 2.0 * sigma * sigma;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nrows; ++r) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j)
            s += gauss_affinity(X, d, rows[r], j, two_sigma2);
        deg[r] = s;
    }
}

/* ------------------------------------------------------------------ */
/* Degree, W = D^-1 A and v0 = D / sum(D)                               */
/* ------------------------------------------------------------------ */

/* v0_i = d_i / sum_j d_j; returns the number of zero-degree rows, or -1
 * when the degrees sum to zero (v0 undefined). */
static int64_t start_vector(const double *degree, int64_t n, double *v0)
{
    double total = 0.0;
    int64_t nzero = 0;
    for (int64_t i = 0; i < n; ++i) {
        total += degree[i];
        if (degree[i] == 0.0)
            ++nzero;
    }
    if (!(total > 0.0) || !isfinite(total))
        return -1;
    for (int64_t i = 0; i < n; ++i)
        v0[i] = degree[i] / total;
    return nzero;
}

/* Dense: A (n x n, row-major) is overwritten by W.  A zero-degree row stays
 * a zero row.  Returns the zero-row count, or -1 if sum(D) is not positive. */
int64_t orc_degree_normalize(double *A, int64_t n, double *degree, double *v0)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j)
            s += A[i * n + j];
        degree[i] = s;
        for (int64_t j = 0; j < n; ++j)
            A[i * n + j] = (s == 0.0) ? 0.0 : A[i * n + j] / s;
    }
    return start_vector(degree, n, v0);
}

/* CSR: w = D^-1 a over the stored entries (columns ascending per row). */
int64_t orc_degree_normalize_csr(const int64_t *row_ptr, const int32_t *col,
                                 const double *a, int64_t n, double *w,
                                 double *degree, double *v0)
{
    (void)col;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double s = 0.0;
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
            s += a[p];
        degree[i] = s;
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
            w[p] = (s == 0.0) ? 0.0 : a[p] / s;
    }
    return start_vector(degree, n, v0);
}

/* Degrees of every row with A recomputed (the on-the-fly operator). */
int64_t orc_degree_onthefly(const float *X, int64_t n, int32_t d, double sigma,
                            double *degree, double *v0)
{
    const double two_sigma2 = 2.0 * sigma * sigma;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j)
            s += gauss_affinity(X, d, i, j, two_sigma2);
        degree[i] = s;
    }
    return start_vector(degree, n, v0);
}

/* ------------------------------------------------------------------ */
/* The operator y = W v in its three storage forms                      */
/* ------------------------------------------------------------------ */

enum { OP_DENSE = 0, OP_CSR = 1, OP_ONTHEFLY = 2 };

typedef struct {
    int kind;
    int64_t n;
    /* dense */
    const double *W;
    /* csr */
    const int64_t *row_ptr;
    const int32_t *col;
    const double *w;
    /* on the fly: W_ij = a_ij / d_i with a_ij recomputed from X */
    const float *X;
    int32_t d;
    double sigma;
    const double *degree;
} orc_op;

static double op_row(const orc_op *op, int64_t i, const double *v)
{
    double y = 0.0;
    switch (op->kind) {
    case OP_DENSE:
        for (int64_t j = 0; j < op->n; ++j)
            y += op->W[i * op->n + j] * v[j];
        break;
    case OP_CSR:
        for (int64_t p = op->row_ptr[i]; p < op->row_ptr[i + 1]; ++p)
            y += op->w[p] * v[op->col[p]];
        break;
    default: {
        const double two_sigma2 = 2.0 * op->sigma * op->sigma;
        const double di = op->degree[i];
        if (di == 0.0)
            return 0.0;
        for (int64_t j = 0; j < op->n; ++j)
            y += (gauss_affinity(op->X, op->d, i, j, two_sigma2) / di) * v[j];
    }
    }
    return y;
}

static void op_apply(const orc_op *op, const double *v, double *y)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t i = 0; i < op->n; ++i)
        y[i] = op_row(op, i, v);
}

/* ------------------------------------------------------------------ */
/* Power iteration with the acceleration stop (section "PIC: an         */
/* overview", update equation; stopping rule of Algorithm 1)            */
/* ------------------------------------------------------------------ */

/* Every update applies the operator, y = W v, scales y by its L1 norm
 * tau = sum_i |y_i| to give the next iterate, and measures the velocity
 * of each coordinate as the absolute change of v.  Its statistic is the
 * largest absolute change of that velocity between consecutive updates;
 * the velocity the first update compares against is whatever delta holds
 * on entry (v_0 itself by the paper's convention, set by the caller).
 * mode 0 runs exactly max_iter updates and records the statistic; mode 1
 * stops after the first update whose statistic is <= eps.  v and delta
 * carry the state in and out (the newest iterate and velocity), so a run
 * can be resumed.  stats[t] receives the statistic of update t.  Returns
 * the number of operator applications performed, or -1 when the L1 norm
 * is zero or not finite. */
static int32_t power_iterate(const orc_op *op, int32_t mode, int32_t max_iter,
                             double eps, double *v, double *delta,
                             double *stats, int32_t *converged)
{
    const int64_t n = op->n;
    double *y = (double *)malloc((size_t)n * sizeof(double));
    *converged = 0;
    int32_t done = max_iter;
    for (int32_t t = 0; t < max_iter; ++t) {
        op_apply(op, v, y);
        double tau = 0.0;
        for (int64_t i = 0; i < n; ++i)
            tau += fabs(y[i]);
        if (!(tau > 0.0) || !isfinite(tau)) {
            done = -1;
            break;
        }
        double s = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            const double v_new = y[i] / tau;
            const double vel = fabs(v_new - v[i]);
            const double change = fabs(vel - delta[i]);
            if (change > s)
                s = change;
            v[i] = v_new;
            delta[i] = vel;
        }
        if (stats)
            stats[t] = s;
        if (mode == 1 && s <= eps) {
            *converged = 1;
            done = t + 1;
            break;
        }
    }
    free(y);
    return done;
}

int32_t orc_power_iterate_dense(const double *W, int64_t n, int32_t mode,
                                int32_t max_iter, double eps, double *v,
                                double *delta, double *stats,
                                int32_t *converged)
{
    orc_op op = {0};
    op.kind = OP_DENSE;
    op.n = n;
    op.W = W;
    return power_iterate(&op, mode, max_iter, eps, v, delta, stats, converged);
}

int32_t orc_power_iterate_csr(const int64_t *row_ptr, const int32_t *col,
                              const double *w, int64_t n, int32_t mode,
                              int32_t max_iter, double eps, double *v,
                              double *delta, double *stats, int32_t *converged)
{
    orc_op op = {0};
    op.kind = OP_CSR;
    op.n = n;
    op.row_ptr = row_ptr;
    op.col = col;
    op.w = w;
    return power_iterate(&op, mode, max_iter, eps, v, delta, stats, converged);
}

int32_t orc_power_iterate_onthefly(const float *X, int64_t n, int32_t d,
                                   double sigma, const double *degree,
                                   int32_t mode, int32_t max_iter, double eps,
                                   double *v, double *delta, double *stats,
                                   int32_t *converged)
{
    orc_op op = {0};
    op.kind = OP_ONTHEFLY;
    op.n = n;
    op.X = X;
    op.d = d;
    op.sigma = sigma;
    op.degree = degree;
    return power_iterate(&op, mode, max_iter, eps, v, delta, stats, converged);
}

/* One product y_i = (W v)_i for the listed rows only, W recomputed. */
void orc_matvec_onthefly_rows(const float *X, int64_t n, int32_t d,
                              double sigma, const double *degree,
                              const double *v, const int64_t *rows,
                              int64_t nrows, double *y)
{
    orc_op op = {0};
    op.kind = OP_ONTHEFLY;
    op.n = n;
    op.X = X;
    op.d = d;
    op.sigma = sigma;
    op.degree = degree;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nrows; ++r)
        y[r] = op_row(&op, rows[r], v);
}

/* ------------------------------------------------------------------ */
/* Exact 1-D k-means                                                    */
/* ------------------------------------------------------------------ */

typedef struct {
    double value;
    int64_t index;
} keyed;

static int cmp_keyed(const void *a, const void *b)
{
    const keyed *x = (const keyed *)a, *y = (const keyed *)b;
    if (x->value < y->value) return -1;
    if (x->value > y->value) return 1;
    return (x->index < y->index) ? -1 : (x->index > y->index);
}

typedef struct {
    int64_t n;
    const double *S1; /* S1[p] = sum_{q<p} u_q   (length n+1) */
    const double *S2; /* S2[p] = sum_{q<p} u_q^2 (length n+1) */
} prefix_t;

/* Within-cluster sum of squares of sorted positions j..i (inclusive),
 * from the prefix sums of the centred values; clamped at zero. */
static double seg_cost(const prefix_t *P, int64_t j, int64_t i)
{
    double m = (double)(i - j + 1);
    double s1 = P->S1[i + 1] - P->S1[j];
    double s2 = P->S2[i + 1] - P->S2[j];
    double c = s2 - s1 * s1 / m;
    return c > 0.0 ? c : 0.0;
}

/* Leftmost argmin over allowed split points j in [lo, hi] of
 * prev[j-1] + cost(j, i); j must start a run of equal values. */
static void best_split(const prefix_t *P, const unsigned char *run_start,
                       const double *prev, int64_t i, int64_t lo, int64_t hi,
                       double *best, int64_t *arg)
{
    double b = INFINITY;
    int64_t a = -1;
    for (int64_t j = lo; j <= hi; ++j) {
        if (!run_start[j])
            continue;
        double c = prev[j - 1] + seg_cost(P, j, i);
        if (c < b) {
            b = c;
            a = j;
        }
    }
    *best = b;
    *arg = a;
}

/* divide and conquer over rows lo..hi whose leftmost argmins lie in
 * [olo, ohi] (monotone optimal split points, see the quadrangle inequality
 * of the within-cluster sum of squares in 1-D) */
static void dc_layer(const prefix_t *P, const unsigned char *run_start,
                     const double *prev, double *cur, int64_t *opt,
                     int64_t lo, int64_t hi, int64_t olo, int64_t ohi)
{
    while (lo <= hi) {
        int64_t mid = lo + (hi - lo) / 2;
        int64_t a_lo = olo < 1 ? 1 : olo;
        int64_t a_hi = ohi < mid ? ohi : mid;
        double b;
        int64_t a;
        best_split(P, run_start, prev, mid, a_lo, a_hi, &b, &a);
        cur[mid] = b;
        opt[mid] = (a < 0) ? a_lo : a;
        /* left half recursively, right half in this loop */
        if (lo <= mid - 1)
            dc_layer(P, run_start, prev, cur, opt, lo, mid - 1, olo, opt[mid]);
        lo = mid + 1;
        olo = opt[mid];
    }
}

/* method 0: plain O(k n^2) programme; method 1: divide-and-conquer search.
 * labels[i] in 0..k_eff-1 by ascending centroid; centroids[c] is the mean
 * of cluster c; *cost_out the total within-cluster sum of squares, both
 * computed directly from the members.  Returns 0, or -1 on bad input. */
int32_t orc_kmeans1d(const double *v, int64_t n, int32_t k, int32_t method,
                     int32_t *labels, double *centroids, int32_t *k_eff,
                     double *cost_out)
{
    if (n < 1 || k < 1)
        return -1;
    keyed *kv = (keyed *)malloc((size_t)n * sizeof(keyed));
    for (int64_t i = 0; i < n; ++i) {
        kv[i].value = v[i];
        kv[i].index = i;
    }
    qsort(kv, (size_t)n, sizeof(keyed), cmp_keyed);

    unsigned char *run_start = (unsigned char *)malloc((size_t)n);
    int64_t distinct = 0;
    for (int64_t p = 0; p < n; ++p) {
        run_start[p] = (p == 0 || kv[p].value != kv[p - 1].value);
        distinct += run_start[p];
    }
    int32_t ke = (int64_t)k < distinct ? k : (int32_t)distinct;

    double mean = 0.0;
    for (int64_t p = 0; p < n; ++p)
        mean += kv[p].value;
    mean /= (double)n;
    double *S1 = (double *)malloc((size_t)(n + 1) * sizeof(double));
    double *S2 = (double *)malloc((size_t)(n + 1) * sizeof(double));
    S1[0] = S2[0] = 0.0;
    for (int64_t p = 0; p < n; ++p) {
        double u = kv[p].value - mean;
        S1[p + 1] = S1[p] + u;
        S2[p + 1] = S2[p] + u * u;
    }
    prefix_t P = {n, S1, S2};

    /* D[c][i]: best cost of sorted positions 0..i in c+1 clusters */
    double *prev = (double *)malloc((size_t)n * sizeof(double));
    double *cur = (double *)malloc((size_t)n * sizeof(double));
    int64_t *opt = (int64_t *)malloc((size_t)ke * (size_t)n * sizeof(int64_t));
    for (int64_t i = 0; i < n; ++i) {
        prev[i] = seg_cost(&P, 0, i);
        opt[i] = 0;
    }
    for (int32_t c = 1; c < ke; ++c) {
        int64_t *oc = opt + (int64_t)c * n;
        if (method == 0) {
#pragma omp parallel for schedule(dynamic, 64)
            for (int64_t i = 0; i < n; ++i) {
                double b;
                int64_t a;
                best_split(&P, run_start, prev, i, 1, i, &b, &a);
                cur[i] = b;
                oc[i] = (a < 0) ? 1 : a;
            }
        } else {
            dc_layer(&P, run_start, prev, cur, oc, 0, n - 1, 1, n - 1);
        }
        double *tmp = prev;
        prev = cur;
        cur = tmp;
    }

    /* backtrack from the last position */
    int64_t *first = (int64_t *)malloc((size_t)ke * sizeof(int64_t));
    int64_t i = n - 1;
    for (int32_t c = ke - 1; c >= 0; --c) {
        int64_t j = opt[(int64_t)c * n + i];
        first[c] = j;
        i = j - 1;
    }
    int32_t status = (i == -1 && first[0] == 0) ? 0 : -1;

    double total = 0.0;
    for (int32_t c = 0; c < ke && status == 0; ++c) {
        int64_t b = first[c], e = (c + 1 < ke) ? first[c + 1] - 1 : n - 1;
        double s = 0.0;
        for (int64_t p = b; p <= e; ++p)
            s += kv[p].value;
        double mu = s / (double)(e - b + 1);
        centroids[c] = mu;
        for (int64_t p = b; p <= e; ++p) {
            labels[kv[p].index] = c;
            total += (kv[p].value - mu) * (kv[p].value - mu);
        }
    }
    *k_eff = ke;
    if (cost_out)
        *cost_out = total;

    free(first);
    free(opt);
    free(cur);
    free(prev);
    free(S2);
    free(S1);
    free(run_start);
    free(kv);
    return status;
}

/* ------------------------------------------------------------------ */
/* kNN input graph                                                     */
/* ------------------------------------------------------------------ */

typedef struct {
    int64_t row, col;
} edge_t;

static int cmp_edge(const void *a, const void *b)
{
    const edge_t *x = (const edge_t *)a, *y = (const edge_t *)b;
    if (x->row != y->row)
        return x->row < y->row ? -1 : 1;
    if (x->col != y->col)
        return x->col < y->col ? -1 : 1;
    return 0;
}

static double sq_dist(const float *X, int32_t d, int64_t i, int64_t j)
{
    double s = 0.0;
    for (int32_t c = 0; c < d; ++c) {
        double diff = (double)X[i * d + c] - (double)X[j * d + c];
        s += diff * diff;
    }
    return s;
}

/* N(i): the k points j != i with the smallest (||x_i - x_j||^2, j), in that
 * order (squared distance summed over coordinates in order; ties to the
 * smaller index), into bj[0..k) with their squared distances in bd. */
static void knn_of(const float *X, int64_t n, int32_t d, int32_t k, int64_t i, double *bd,
                   int64_t *bj)
{
    int32_t m = 0;                               /* kept so far, sorted by (dist, j) */
    for (int64_t j = 0; j < n; ++j) {
        if (j == i)
            continue;
        double dj = sq_dist(X, d, i, j);
        if (m == k && !(dj < bd[k - 1]))
            continue;                            /* j > kept indices: ties lose */
        int32_t p = (m < k) ? m++ : k - 1;
        while (p > 0 && dj < bd[p - 1]) {
            bd[p] = bd[p - 1];
            bj[p] = bj[p - 1];
            --p;
        }
        bd[p] = dj;
        bj[p] = j;
    }
}

/* Exact k-nearest-neighbour graph: N(i) as in knn_of; edge {i, j} if j in
 * N(i) or i in N(j); weight exp(-||x_i - x_j||^2 / (2 sigma^2)) in float64,
 * rounded once to float32; rows sorted by column.  row_ptr [n+1]; col and
 * val hold up to 2 n k entries.  Returns nnz, or -1 if k is not in
 * [1, n-1]. */
int64_t orc_knn_graph(const float *X, int64_t n, int32_t d, int32_t k, double sigma,
                      int64_t *row_ptr, int32_t *col, float *val)
{
    if (k < 1 || (int64_t)k > n - 1)
        return -1;
    edge_t *e = (edge_t *)malloc(sizeof(edge_t) * 2 * (size_t)n * (size_t)k);
#pragma omp parallel
    {
        double *bd = (double *)malloc(sizeof(double) * (size_t)k);
        int64_t *bj = (int64_t *)malloc(sizeof(int64_t) * (size_t)k);
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            knn_of(X, n, d, k, i, bd, bj);
            for (int32_t t = 0; t < k; ++t) {
                e[(2 * i) * (int64_t)k + 2 * t].row = i;
                e[(2 * i) * (int64_t)k + 2 * t].col = bj[t];
                e[(2 * i) * (int64_t)k + 2 * t + 1].row = bj[t];
                e[(2 * i) * (int64_t)k + 2 * t + 1].col = i;
            }
        }
        free(bj);
        free(bd);
    }
    const int64_t m2 = 2 * n * (int64_t)k;
    qsort(e, (size_t)m2, sizeof(edge_t), cmp_edge);
    const double two_sigma2 = 2.0 * sigma * sigma;
    int64_t nnz = 0;
    for (int64_t i = 0; i <= n; ++i)
        row_ptr[i] = 0;
    for (int64_t t = 0; t < m2; ++t) {
        if (t > 0 && e[t].row == e[t - 1].row && e[t].col == e[t - 1].col)
            continue;
        col[nnz] = (int32_t)e[t].col;
        val[nnz] = (float)exp(-sq_dist(X, d, e[t].row, e[t].col) / two_sigma2);
        row_ptr[e[t].row + 1]++;
        ++nnz;
    }
    for (int64_t i = 0; i < n; ++i)
        row_ptr[i + 1] += row_ptr[i];
    free(e);
    return nnz;
}

/* N(i) of the listed points alone (the graph's neighbour lists one by one,
 * for sampled checks of graphs too large to build here): for row t,
 * nbr[t k + s] = the s-th nearest of point rows[t] as in knn_of, d2 its
 * squared distance and w its weight exp(-d2 / (2 sigma^2)) rounded once to
 * float32.  Returns 0, or -1 if k is not in [1, n-1] or a row is out of
 * range. */
int32_t orc_knn_rows(const float *X, int64_t n, int32_t d, int32_t k, double sigma,
                     const int64_t *rows, int64_t m, int64_t *nbr, double *d2, float *w)
{
    if (k < 1 || (int64_t)k > n - 1)
        return -1;
    for (int64_t t = 0; t < m; ++t)
        if (rows[t] < 0 || rows[t] >= n)
            return -1;
    const double two_sigma2 = 2.0 * sigma * sigma;
#pragma omp parallel for schedule(dynamic)
    for (int64_t t = 0; t < m; ++t) {
        knn_of(X, n, d, k, rows[t], d2 + t * k, nbr + t * k);
        for (int32_t s = 0; s < k; ++s)
            w[t * k + s] = (float)exp(-d2[t * k + s] / two_sigma2);
    }
    return 0;
}
