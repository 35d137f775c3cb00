/*
 * gpic.h -- C ABI of libgpic, Power Iteration Clustering (PIC) on one
 * AMD Instinct MI355X (gfx950), following the GPIC paper (arXiv 1604.02700).
 *
 * The library covers the data-parallel hot path of the method:
 *   1. the affinity matrix A of the data graph (section "Spectral Cluster";
 *      the AffinityMatrix step of Algorithm 2),
 *   2. the degrees d_ii = sum_j a_ij, W = D^-1 A and v0 = D / sum(D)
 *      ("Spectral Cluster"; the RowSum, NormMat, Reduction and Norm steps
 *      of Algorithm 2),
 *   3. the power iteration v_{t+1} = W v_t / ||W v_t||_1 (update equation of
 *      section "Power Iteration Clustering: An Overview") with the
 *      acceleration stop of Algorithm 1 -- delta_0 = v_0,
 *      delta_{t+1} = |v_{t+1} - v_t|, stop when |delta_{t+1} - delta_t| <= eps
 *      in every entry -- over three storages of W: a dense matrix, an
 *      on-the-fly (fused) recomputation from the points, and a CSR graph,
 *   4. the final k-means of the one-dimensional embedding v (last step of
 *      Algorithms 1 and 2), computed exactly.
 *
 * Conventions (all entry points):
 *   - Pointers are DEVICE pointers owned by the caller unless marked "host".
 *     The library never allocates or frees device memory; scratch space comes
 *     from the caller through (ws, ws_bytes), sized by gpic_workspace_bytes.
 *     Workspace must be 256-byte aligned.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls are asynchronous unless stated otherwise.
 *   - Every call returns a gpic_status; no C++ exception crosses the ABI.
 *     Arguments are validated on the host before any launch.  On an error
 *     the outputs are unspecified; gpic_last_error() gives the text
 *     (thread-local).
 *   - Layouts: points X are float32 [n x d] row-major (4-byte aligned);
 *     dense A / W are float32 [n x lda] row-major, only the first n columns
 *     of each row are read or written, lda % 4 == 0, base 16-byte aligned.
 *     Vectors v, delta, degree, v0 are float64 [n], 16-byte aligned.
 *     CSR graphs: row_ptr int64 [n+1], col int32 [nnz], val float32 [nnz].
 *     gpic_degree_normalize_csr and gpic_power_iterate_csr check the
 *     structure on the device before any kernel indexes through it (row_ptr
 *     nondecreasing from 0 to nnz, every column in [0, n); otherwise
 *     GPIC_ERR_INVALID_ARG, a check that synchronises the stream);
 *     gpic_matvec_csr, which takes no workspace, relies on a graph one of
 *     those calls has accepted.
 *   - Floating point: stored matrices and points are float32; every
 *     accumulation and all iteration state (v, delta, the L1 norm, the stop
 *     statistic, degrees) are float64.  Reductions are deterministic (fixed
 *     order, no floating-point atomics): two runs give identical bits.
 */
#ifndef GPIC_H
#define GPIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GPIC_ABI_VERSION 1

typedef enum gpic_status {
    GPIC_OK = 0,
    GPIC_ERR_INVALID_ARG = 1, /* null pointer, bad size, bad alignment, ... */
    GPIC_ERR_WORKSPACE = 2,   /* ws_bytes smaller than gpic_workspace_bytes */
    GPIC_ERR_HIP = 3,         /* a HIP launch or runtime call failed        */
    GPIC_ERR_NUMERIC = 4,     /* ||W v||_1 or sum(D) zero or not finite     */
    GPIC_ERR_UNSUPPORTED = 5  /* valid request this build does not handle   */
} gpic_status;

/* Operation codes for gpic_workspace_bytes. */
enum {
    GPIC_OP_AFFINITY = 0,
    GPIC_OP_DEGREE_NORMALIZE = 1,
    GPIC_OP_DEGREE_NORMALIZE_CSR = 2,
    GPIC_OP_DEGREE_FUSED = 3,
    GPIC_OP_PI_DENSE = 4,
    GPIC_OP_PI_FUSED = 5,
    GPIC_OP_PI_CSR = 6,
    GPIC_OP_KMEANS1D = 7,
    GPIC_OP_AFFINITY_NORMALIZED = 8,
    GPIC_OP_MATVEC_FUSED = 9,
    GPIC_OP_AFFINITY_COSINE = 10,
    GPIC_OP_AFFINITY_COSINE_NORMALIZED = 11,
    GPIC_OP_KNN_GRAPH = 12,
    GPIC_OP_AFFINITY_SYM = 13,
    GPIC_OP_MATVEC_SYM = 14,
    GPIC_OP_PI_SYM = 15,
    GPIC_OP_PI_DENSE_HOST = 16
};

/* Power-iteration modes. */
enum {
    GPIC_MODE_FIXED = 0,   /* exactly max_iter updates; the statistic is recorded */
    GPIC_MODE_CONVERGE = 1 /* stop at the first update whose statistic <= eps */
};

typedef struct gpic_pi_params {
    int32_t mode;        /* GPIC_MODE_FIXED or GPIC_MODE_CONVERGE                  */
    int32_t max_iter;    /* T in FIXED mode, the cap in CONVERGE mode (>= 0)       */
    double eps;          /* stop precision (>= 0); the paper uses 1e-5 / n         */
    int32_t check_every; /* CONVERGE: the host reads the stop state every this
                            many updates (0 = default 16); results do not depend
                            on it, only the number of empty launches after a stop */
    int32_t reserved;    /* must be 0                                              */
    double *stats_host;  /* host, nullable: receives the statistic
                            s_t = max_i |delta_{t+1,i} - delta_{t,i}| of every
                            update performed (room for max_iter values)            */
} gpic_pi_params;

typedef struct gpic_pi_result {
    int32_t iterations;  /* matrix-vector products performed                       */
    int32_t converged;   /* 1 if the stop test held, else 0 (not an error)         */
    double last_stat;    /* statistic of the last update (0 if none)               */
} gpic_pi_result;

/* ---------------------------------------------------------------- helpers */

int32_t gpic_abi_version(void);
const char *gpic_status_string(gpic_status s);
/* Text of the last error raised on the calling thread ("" if none). */
const char *gpic_last_error(void);
/* Workspace bytes an operation needs for n rows, nnz stored entries (CSR)
 * and k clusters (k-means); arguments an operation does not use are
 * ignored.  0 means the operation needs none.  Returns 0 for an unknown op
 * or negative sizes. */
size_t gpic_workspace_bytes(int32_t op, int64_t n, int64_t nnz, int32_t k);

/* ------------------------------------------------------- 1. affinity (A) */

/* Dense Gaussian affinity, the reading taken for the affinity of section
 * "Spectral Cluster" (the paper does not write its kernel down):
 *   A_ij = exp(-||x_i - x_j||^2 / (2 sigma^2)) for i != j,  A_ii = 0.
 * X: float32 [n x d]; A: float32 [n x lda], written in columns 0..n-1 only.
 * d < 16 or d > 128 uses direct coordinate differences; 16 <= d <= 128
 * forms c * squared distance on the fp32 matrix cores from augmented points
 * [x_j, |x_j|^2, 1] . [-2c x_i, c, c |x_i|^2] (c = log2(e) / (2 sigma^2),
 * clamped at 0).  degree (nullable) receives d_i = sum_j A_ij of the stored
 * float32 values, accumulated in float64 in a fixed order.
 * ws: gpic_workspace_bytes(GPIC_OP_AFFINITY, n, 0, 0) bytes (squared norms
 * and per-chunk row sums).
 * Errors: INVALID_ARG for null X/A, n < 2, d < 1, sigma <= 0 or not finite,
 * lda < n, lda % 4 != 0, misaligned pointers.  Asynchronous. */
gpic_status gpic_affinity(const float *X, int64_t n, int32_t d, float sigma,
                          float *A, int64_t lda, double *degree, void *ws,
                          size_t ws_bytes, void *stream);

/* Steps 1 and 2 in one call, A never stored: a first sweep forms the
 * degrees d_i = sum_{j != i} A_ij of the float32 affinities (as
 * gpic_affinity's row sums), then v0 = D / sum D and the zero-degree count,
 * and a second sweep recomputes A and writes W_ij = A_ij * r_i with
 * r_i = float32(1 / d_i) into W [n x ldw].  Bit for bit the
 * same W, degree and v0 as gpic_affinity followed by gpic_degree_normalize
 * with degree_given = 1, with 4 n^2 bytes of HBM traffic instead of 12 n^2.
 * Same argument rules as those two calls; synchronises the stream (sum(D)
 * check).  ws: gpic_workspace_bytes(GPIC_OP_AFFINITY_NORMALIZED, n, 0, 0). */
gpic_status gpic_affinity_normalized(const float *X, int64_t n, int32_t d,
                                     float sigma, float *W, int64_t ldw,
                                     double *degree, double *v0,
                                     int64_t *n_zero_rows, void *ws,
                                     size_t ws_bytes, void *stream);

/* Dense cosine affinity, the similarity of the paper's Experiment I (Table
 * 2 caption), shifted so that A stays non-negative (W = D^-1 A needs it):
 *   A_ij = max(0, (1 + cos(x_i, x_j)) / 2) for i != j,  A_ii = 0,
 *   cos(x_i, x_j) = x_i . x_j / (||x_i|| ||x_j||), taken as 0 when either
 *   point is the origin (so the origin has A = 1/2 against every point).
 * The dot product is a float32 sum over the raw coordinates, scaled by the
 * reciprocal norms (float64, rounded once).  X, A, lda, degree as in
 * gpic_affinity.  ws: gpic_workspace_bytes(GPIC_OP_AFFINITY_COSINE, n, 0, 0)
 * bytes (reciprocal norms).  Errors: INVALID_ARG for null X/A, n < 2,
 * d < 1, lda < n, lda % 4 != 0, misaligned pointers.  Asynchronous. */
gpic_status gpic_affinity_cosine(const float *X, int64_t n, int32_t d, float *A,
                                 int64_t lda, double *degree, void *ws,
                                 size_t ws_bytes, void *stream);

/* gpic_affinity_normalized for the cosine affinity: a degree sweep, v0 and
 * the zero-degree count, then W_ij = A_ij * float32(1 / d_i) written
 * directly.  Synchronises the stream (sum(D) check).
 * ws: gpic_workspace_bytes(GPIC_OP_AFFINITY_COSINE_NORMALIZED, n, 0, 0). */
gpic_status gpic_affinity_cosine_normalized(const float *X, int64_t n, int32_t d,
                                            float *W, int64_t ldw, double *degree,
                                            double *v0, int64_t *n_zero_rows,
                                            void *ws, size_t ws_bytes, void *stream);

/* The sparse affinity graph the CSR path takes as input (the paper's
 * affinity of section "Spectral Cluster" restricted to nearest
 * neighbours): N(i) = the k points j != i with the smallest
 * (||x_i - x_j||^2, j), ties to the smaller index; edge {i, j} when j is in
 * N(i) or i in N(j); weight exp(-||x_i - x_j||^2 / (2 sigma^2)) in float64
 * (squared distance summed over coordinates in order), rounded once to
 * float32; rows sorted by column.  Exact (float32 distances only narrow
 * the candidates; the selection uses float64 distances).
 * X: float32 [n x d], d <= 16; 1 <= k <= min(64, n - 1); 2 n k < 2^32.
 * Outputs (device, caller-allocated): row_ptr int64 [n+1]; col int32 and
 * val float32 with room for 2 n k entries; *nnz (host) = row_ptr[n].
 * Synchronises the stream.  ws: gpic_workspace_bytes(GPIC_OP_KNN_GRAPH, n,
 * 0, k) bytes (about 8 KiB per point: a 2,048-slot candidate list per row).
 * Errors: INVALID_ARG for null or misaligned pointers, n < 2, d < 1, k out
 * of range, sigma <= 0; UNSUPPORTED for d > 16. */
gpic_status gpic_knn_graph(const float *X, int64_t n, int32_t d, int32_t k,
                           float sigma, int64_t *row_ptr, int32_t *col, float *val,
                           int64_t *nnz, void *ws, size_t ws_bytes, void *stream);

/* The same graph with its nodes numbered in the Morton order of the points
 * (their quantised centred coordinates, the order the builder sorts them
 * by): node p is point perm[p] (perm: int32 [n], device, written), rows
 * and columns use node numbers, rows sorted by node number, weights from
 * the points as above.  The affinity graph is the same whatever the
 * numbering (section "Spectral Cluster"); this one keeps graph neighbours
 * at nearby numbers, so the CSR product's gathers of v stay in cache.  A
 * result v over the nodes maps back to the points as v_point[perm[p]] =
 * v_node[p].  Arguments, workspace and errors as gpic_knn_graph, plus
 * INVALID_ARG for a null or misaligned perm. */
gpic_status gpic_knn_graph_local(const float *X, int64_t n, int32_t d, int32_t k,
                                 float sigma, int64_t *row_ptr, int32_t *col, float *val,
                                 int64_t *nnz, int32_t *perm, void *ws, size_t ws_bytes,
                                 void *stream);

/* Symmetric storage ("packed upper tiles") of the affinity: A is symmetric
 * (section "Spectral Cluster"), so only its upper block triangle is kept and
 * the power iteration applies W v = D^-1 (A v), streaming 2 n^2 bytes per
 * product instead of the 4 n^2 of a dense W.  Layout: the indices are cut
 * into nb = ceil(n / 256) blocks of 256; tile (I, J), I <= J, is a float32
 * [256 x 256] row-major array holding A[256 I + r][256 J + c], and the
 * tiles are stored one after the other in the order (0,0), (0,1), ..,
 * (0,nb-1), (1,1), .., (nb-1,nb-1).  Diagonal tiles hold the whole block
 * (zero diagonal).  Entries outside [0, n)^2 are never written and may hold
 * anything: the product loads whole tile rows but replaces them by 0.
 * 2 <= n <= 2^24 for every symmetric entry point (INVALID_ARG otherwise).
 * gpic_sym_bytes(n): bytes of that storage (0 for n out of range). */
size_t gpic_sym_bytes(int64_t n);

/* Affinity A into the symmetric storage As (gpic_sym_bytes(n) bytes,
 * 16-byte aligned, caller-allocated), with the degrees d_i = sum_j A_ij
 * (float64 row sums of the stored symmetric A, taken by the symmetric
 * product with v = 1, so the rows of D^-1 A sum to 1 up to float64
 * rounding), v0 = d / sum(d) and the zero-degree row count (as
 * gpic_affinity_normalized; GPIC_ERR_NUMERIC when sum(D) is zero or not
 * finite, a check that synchronises the stream).  Stored entries are the
 * upper ones: A_ij as computed for row i, for block(i) <= block(j), used
 * for A_ji as well.  ws: gpic_workspace_bytes(GPIC_OP_AFFINITY_SYM, n, 0, 0). */
gpic_status gpic_affinity_sym(const float *X, int64_t n, int32_t d, float sigma,
                              float *As, double *degree, double *v0,
                              int64_t *n_zero_rows, void *ws, size_t ws_bytes,
                              void *stream);

/* --------------------------------- 2. degrees, W = D^-1 A, v0 = D / sum D */

/* Dense, in place: A becomes W (row i times r_i = float32(1 / d_i)).  If degree_given
 * is non-zero, degree holds d (e.g. written by gpic_affinity) and is read;
 * otherwise it is computed here from A and written.  v0_i = d_i / sum_j d_j.
 * A zero-degree row stays a zero row, gets v0_i = 0 and is counted in
 * *n_zero_rows (device int64, nullable).  If sum(D) is zero or not finite,
 * v0 is left unwritten and the call returns GPIC_ERR_NUMERIC (this check
 * synchronises the stream).  ws: gpic_workspace_bytes(GPIC_OP_DEGREE_NORMALIZE, n, 0, 0). */
gpic_status gpic_degree_normalize(float *A, int64_t n, int64_t lda,
                                  double *degree, int32_t degree_given,
                                  double *v0, int64_t *n_zero_rows, void *ws,
                                  size_t ws_bytes, void *stream);

/* CSR, in place over val (rows sorted or not; entries summed in storage
 * order).  Same outputs and errors as the dense version.
 * ws: gpic_workspace_bytes(GPIC_OP_DEGREE_NORMALIZE_CSR, n, nnz, 0). */
gpic_status gpic_degree_normalize_csr(const int64_t *row_ptr,
                                      const int32_t *col, float *val,
                                      int64_t n, int64_t nnz, double *degree,
                                      double *v0, int64_t *n_zero_rows,
                                      void *ws, size_t ws_bytes, void *stream);

/* Fused (W never stored): d_i = sum_{j != i} A_ij with A recomputed from the
 * points as in gpic_affinity, and v0 = D / sum D.  Nothing of size n^2 is
 * written.  For 16 <= d <= 128 and n <= 2^19 the fused operator evaluates
 * each pair {i, j} once (A = A^T, section "Spectral Cluster") and uses that
 * one float32 value for both A_ij and A_ji; the degrees are the row sums of
 * that same symmetric A (so W's rows sum to 1 up to float64 rounding), and
 * may differ from gpic_affinity's row sums in the last float32 bits of
 * individual entries.  ws: gpic_workspace_bytes(GPIC_OP_DEGREE_FUSED, n, 0, 0)
 * (for n <= 2^19 it includes about n^2 / 64 bytes of column partial sums). */
gpic_status gpic_degree_fused(const float *X, int64_t n, int32_t d,
                              float sigma, double *degree, double *v0,
                              int64_t *n_zero_rows, void *ws, size_t ws_bytes,
                              void *stream);

/* ------------------------------------------ 3. the operator y = W v alone */

/* One product y = W v over dense float32 W [n x ldw] (Multiply step of
 * Algorithm 2), accumulated in float64.  No normalisation.  Asynchronous. */
gpic_status gpic_matvec_dense(const float *W, int64_t n, int64_t ldw,
                              const double *v, double *y, void *stream);

/* One product y_i = (sum_j A_ij v_j) / d_i over the symmetric storage As
 * (see gpic_sym_bytes; y_i = 0 for d_i = 0), accumulated in float64 in a
 * fixed order.  ws: gpic_workspace_bytes(GPIC_OP_MATVEC_SYM, n, 0, 0)
 * (the per-tile partial sums, nb^2 * 256 float64).  Asynchronous. */
gpic_status gpic_matvec_sym(const float *As, int64_t n, const double *degree,
                            const double *v, double *y, void *ws, size_t ws_bytes,
                            void *stream);

/* One product over a CSR W, rows in storage order, accumulated in float64.
 * The structure is not checked here (see the layout notes at the top).
 * Asynchronous. */
gpic_status gpic_matvec_csr(const int64_t *row_ptr, const int32_t *col,
                            const float *val, int64_t n, int64_t nnz,
                            const double *v, double *y, void *stream);

/* One product y_i = (sum_{j != i} A_ij v_j) / d_i with A recomputed from X
 * (the fused operator; W = D^-1 A is never stored).  A zero-degree row gives
 * y_i = 0.  For 16 <= d <= 128 and n <= 2^19 each pair is evaluated once
 * (see gpic_degree_fused): the rows of 256-point groups give their row sums
 * and, beyond their own group, column sums to later groups, added per row
 * in a fixed order by a second launch.
 * ws: gpic_workspace_bytes(GPIC_OP_MATVEC_FUSED, n, 0, 0).  Asynchronous. */
gpic_status gpic_matvec_fused(const float *X, int64_t n, int32_t d,
                              float sigma, const double *degree,
                              const double *v, double *y, void *ws,
                              size_t ws_bytes, void *stream);

/* ------------------------------------------------- 3+4. power iteration */

/* Algorithm 1's loop over dense W.  v (in: v_t, usually v0; out: the newest
 * iterate) and delta (in: delta_t; out: the newest velocity) carry the whole
 * state, so a run can be resumed; delta == NULL means delta_0 = v_0 (kept
 * in the workspace).  Each update: y = W v, tau = sum_i |y_i|,
 * v <- y / tau, delta' = |v_new - v_old|, s_t = max_i |delta' - delta|.
 * Synchronises the stream at the end (and every check_every updates in
 * CONVERGE mode); *res (host) receives the counts.  GPIC_ERR_NUMERIC if
 * tau is zero or not finite; reaching max_iter without the stop is not an
 * error (converged = 0).  ws: gpic_workspace_bytes(GPIC_OP_PI_DENSE, n, 0, 0). */
gpic_status gpic_power_iterate_dense(const float *W, int64_t n, int64_t ldw,
                                     const gpic_pi_params *params, double *v,
                                     double *delta, void *ws, size_t ws_bytes,
                                     gpic_pi_result *res, void *stream);

/* For callers that cannot allocate device memory (tight serving loops,
 * harnesses that forbid hipMalloc): gpic_power_iterate_dense with its
 * scratch (control words, statistic ring, per-workgroup |y| partials, y and,
 * when delta is null, delta) in a static device array of
 * GPIC_NOALLOC_SCRATCH_BYTES that the library owns, one per GPU, held until
 * the process ends, instead of a caller workspace.  Same arguments, results
 * (bitwise: the same kernels) and errors as gpic_power_iterate_dense, minus
 * ws; allocates nothing (no hipMalloc/hipFree, no library allocation).
 * n <= GPIC_NOALLOC_MAX_N, else GPIC_ERR_WORKSPACE before any launch.  The
 * scratch is re-initialised on the device by every call, but it is shared:
 * calls that overlap on one GPU (several streams or threads at once) race
 * and must be serialised by the caller. */
#define GPIC_NOALLOC_SCRATCH_BYTES (8u << 20)
#define GPIC_NOALLOC_MAX_N 465536
gpic_status gpic_power_iterate_dense_noalloc(const float *W, int64_t n, int64_t ldw,
                                             const gpic_pi_params *params, double *v,
                                             double *delta, gpic_pi_result *res,
                                             void *stream);

/* Out-of-core: the same loop over a dense W that stays in HOST memory
 * (W_host: host pointer, float32 [n x ldw] row-major, ldw >= n; allocate it
 * pinned, e.g. with hipHostMalloc, so that copies overlap the products).
 * For a W larger than the device memory: section "Our Approach GPIC"
 * divides the data into chunks copied to the device one after another;
 * on 288 GB of HBM every workload here fits, so this path serves larger n.  Every update streams
 * W to the device in panels of P rows through two staging buffers in ws
 * (copy of panel k on an internal copy stream, product of panel k-1 on
 * `stream`); results are bitwise those of gpic_power_iterate_dense.  P is
 * the largest multiple of 4 whose two buffers (P rows of n floats rounded
 * up to 4) fit in ws after the power-iteration state:
 * gpic_workspace_bytes(GPIC_OP_PI_DENSE_HOST, n, 0, 0) gives two 64 MiB
 * panels; a smaller ws (at least two 4-row panels) gives smaller panels,
 * a larger one larger panels.  In CONVERGE mode check_every = 0 means 1
 * here (an update queued past the stop costs a full pass of W over PCIe).
 * Creates and destroys one stream and four events per call; synchronises
 * at the end.  Errors: as gpic_power_iterate_dense; WORKSPACE when ws holds
 * no two 4-row panels. */
gpic_status gpic_power_iterate_dense_host(const float *W_host, int64_t n, int64_t ldw,
                                          const gpic_pi_params *params, double *v,
                                          double *delta, void *ws, size_t ws_bytes,
                                          gpic_pi_result *res, void *stream);

/* The same loop over the symmetric storage As with the degrees d (both
 * from gpic_affinity_sym): each update's product is y = D^-1 (A v).
 * ws: gpic_workspace_bytes(GPIC_OP_PI_SYM, n, 0, 0). */
gpic_status gpic_power_iterate_sym(const float *As, int64_t n, const double *degree,
                                   const gpic_pi_params *params, double *v,
                                   double *delta, void *ws, size_t ws_bytes,
                                   gpic_pi_result *res, void *stream);

/* The same loop with the fused operator (A recomputed every update from X,
 * sigma, and the degrees from gpic_degree_fused).
 * ws: gpic_workspace_bytes(GPIC_OP_PI_FUSED, n, 0, 0). */
gpic_status gpic_power_iterate_fused(const float *X, int64_t n, int32_t d,
                                     float sigma, const double *degree,
                                     const gpic_pi_params *params, double *v,
                                     double *delta, void *ws, size_t ws_bytes,
                                     gpic_pi_result *res, void *stream);

/* The same loop over a CSR W (values already normalised by
 * gpic_degree_normalize_csr).  ws: gpic_workspace_bytes(GPIC_OP_PI_CSR, n, nnz, 0).
 * For 2^18 < n <= 2^23 the workspace also holds a column-blocked copy of W
 * (about 8 bytes per stored entry plus per-block row offsets and sums),
 * made once per call and used when every row's columns are ascending, at
 * least a quarter of the entries lie more than 2^17 columns from the
 * diagonal and each block of 2^18 columns holds fewer than 2^30 entries;
 * the iterates then differ from the row-wise product's only in the order
 * of the float64 sums.  Building the copy synchronises the stream once
 * more. */
gpic_status gpic_power_iterate_csr(const int64_t *row_ptr, const int32_t *col,
                                   const float *val, int64_t n, int64_t nnz,
                                   const gpic_pi_params *params, double *v,
                                   double *delta, void *ws, size_t ws_bytes,
                                   gpic_pi_result *res, void *stream);

/* ------------------------------------------------------- 5. 1-D k-means */

/* "k-means of v" read as the exact minimum within-cluster sum of squares
 * partition of the n scalars v_i into k clusters (the paper leaves the
 * variant open).  Equal values are never split: with fewer than k distinct
 * values, *k_eff (host) < k.  labels (int32 [n]) are 0..k_eff-1 by
 * ascending centroid; centroids (float64 [k]) get the k_eff cluster means;
 * *cost (host, nullable) the total within-cluster sum of squares.  Split
 * ties go to the smallest sorted position.  Synchronises the stream.
 * Errors: INVALID_ARG for n < 1, n > 2^30, k < 1, k > n, null pointers;
 * values must be finite.  ws: gpic_workspace_bytes(GPIC_OP_KMEANS1D, n, 0, k). */
gpic_status gpic_kmeans1d(const double *v, int64_t n, int32_t k,
                          int32_t *labels, double *centroids, int32_t *k_eff,
                          double *cost, void *ws, size_t ws_bytes,
                          void *stream);

/* ------------------------------------------- 6. bandwidth reference */

/* Length of the sink gpic_read_stream writes. */
#define GPIC_READ_STREAM_SINK 1536

/* Reads the n floats of x (device, 16-byte aligned, n a positive multiple
 * of 4) once with 16-byte non-temporal loads over GPIC_READ_STREAM_SINK
 * workgroups, each writing the float64 sum of what it read to sink (device,
 * float64 [GPIC_READ_STREAM_SINK], 16-byte aligned).  Not a step of the
 * method: the plain read stream the dense product (a pure HBM read of W) is
 * compared with, timed on the same buffer.  Asynchronous. */
gpic_status gpic_read_stream(const float *x, int64_t n, double *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GPIC_H */
