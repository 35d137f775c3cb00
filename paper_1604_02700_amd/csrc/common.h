// Internal helpers shared by the libgpic HIP translation units (not part of
// the C ABI).  Written for gfx950: 64-lane wavefronts, float64 shuffles
// through two 32-bit lane exchanges, no floating-point atomics anywhere.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gpic {

constexpr int kWave = 64;

// ---------------------------------------------------------------- errors
// Records the text of the last error on the calling thread.
void set_error(const char *fmt, ...);

// ------------------------------------------------------ wave reductions
// Butterfly reductions: lane l combines with lane l ^ o.  Because a + b and
// b + a round identically, every lane ends with bit-identical results and
// the result does not depend on scheduling.
__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        x += __shfl_xor(x, o, kWave);
    return x;
}

__device__ __forceinline__ double wave_max(double x)
{
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        x = fmax(x, __shfl_xor(x, o, kWave));
    return x;
}

// Sum over groups of `width` consecutive lanes (width a power of two <= 64).
template <int width>
__device__ __forceinline__ double group_sum(double x)
{
#pragma unroll
    for (int o = width / 2; o > 0; o >>= 1)
        x += __shfl_xor(x, o, kWave);
    return x;
}

// Block sum for a block of NT threads; result valid in every thread.
// `scratch` must hold NT / 64 doubles.  Order: wave butterflies, then the
// wave partials in ascending wave order.
template <int NT>
__device__ __forceinline__ double block_sum(double x, double *scratch)
{
    constexpr int nw = NT / kWave;
    x = wave_sum(x);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0)
        scratch[w] = x;
    __syncthreads();
    double t = 0.0;
#pragma unroll
    for (int i = 0; i < nw; ++i)
        t += scratch[i];
    __syncthreads();
    return t;
}

template <int NT>
__device__ __forceinline__ double block_max(double x, double *scratch)
{
    constexpr int nw = NT / kWave;
    x = wave_max(x);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x % kWave) == 0)
        scratch[w] = x;
    __syncthreads();
    double t = scratch[0];
#pragma unroll
    for (int i = 1; i < nw; ++i)
        t = fmax(t, scratch[i]);
    __syncthreads();
    return t;
}

// ---------------------------------------------------- power-iteration state
// Device-side stop control shared by the product, reduction and update
// kernels of one update t.  The statistic of update t lives in
// stat_ring[t % ring]; the product kernel of update t clears that slot
// (block 0) and every kernel of update t is skipped when the statistic of
// update t-1 already satisfied the stop test, or a numeric error was
// flagged.  Skipped updates leave their slot at 0, so the chain of skips
// continues to the end of the launched batch.
struct StopCtl {
    const double *prev_stat; // slot of update t-1, or nullptr (no test)
    double *cur_stat;        // slot of update t
    double eps;              // stop precision (< 0 in FIXED mode: never)
    int *err;                // numeric error flag (tau zero / not finite)
};

__device__ __forceinline__ bool stop_reached(const StopCtl &c)
{
    if (*c.err != 0)
        return true;
    return c.prev_stat != nullptr && *c.prev_stat <= c.eps;
}

// --------------------------------------------------------------- launchers
// Host-side launch wrappers implemented in the kernel translation units.
// Each returns hipSuccess or the launch error.
const char *last_error_text();

// affinity.hip -- ws: affinity_ws(n) bytes (squared norms and per-chunk row
// sums); needed for 16 <= d <= 128, ignored otherwise
size_t affinity_ws(int64_t n);
hipError_t launch_affinity(const float *X, int64_t n, int d, float c_log2,
                           float *A, int64_t lda, double *degree, void *ws,
                           hipStream_t s);
hipError_t launch_affinity_w(const float *X, int64_t n, int d, float c_log2,
                             float *W, int64_t ldw, const double *degree,
                             void *ws, hipStream_t s);
hipError_t launch_fused_degree(const float *X, int64_t n, int d, float c_log2,
                               double *degree, void *ws, hipStream_t s);
// Augmented operands for the matrix-core engine, once for a run of
// products that pass operands_ready = true (no-op below 16 or above 128
// dimensions).
hipError_t launch_fused_prepare(const float *X, int64_t n, int d, float c_log2,
                                void *ws, hipStream_t s);
// ws: fused_ws(n) bytes
hipError_t launch_fused_apply(const float *X, int64_t n, int d, float c_log2,
                              const double *v, const double *degree, double *y,
                              double *partial, StopCtl ctl, bool use_ctl,
                              void *ws, hipStream_t s, bool operands_ready = false);
// number of |y| partial sums the fused product writes
int64_t fused_blocks(int64_t n, int d);
// the fused product's ws: affinity_ws(n) bytes, then (n <= 2^19, where the
// product takes each pair once) the column partial sums
size_t fused_ws(int64_t n);
// the degrees of the fused operator's A (ws: fused_ws(n) bytes): where the
// product takes each pair once, the same sweep with v = 1, else the
// row-sum sweep of launch_fused_degree
hipError_t launch_fused_operator_degree(const float *X, int64_t n, int d, float c_log2,
                                       double *degree, void *ws, hipStream_t s);
// A into the packed upper tiles of the symmetric storage (sym.hip);
// ws: affinity_ws(n) bytes
hipError_t launch_affinity_sym(const float *X, int64_t n, int d, float c_log2,
                               float *As, void *ws, hipStream_t s);
// cosine affinity (1 + cos) / 2, zero diagonal -- ws: cosine_ws(n) bytes
// (reciprocal norms)
size_t cosine_ws(int64_t n);
hipError_t launch_affinity_cosine(const float *X, int64_t n, int d, float *A,
                                  int64_t lda, double *degree, void *ws, hipStream_t s);
hipError_t launch_cosine_degree(const float *X, int64_t n, int d, double *degree,
                                void *ws, hipStream_t s);
hipError_t launch_cosine_w(const float *X, int64_t n, int d, float *W, int64_t ldw,
                           const double *degree, void *ws, hipStream_t s);

// normalize.hip
hipError_t launch_dense_degree(const float *A, int64_t n, int64_t lda,
                               double *degree, hipStream_t s);
hipError_t launch_dense_scale(float *A, int64_t n, int64_t lda,
                              const double *degree, hipStream_t s);
hipError_t launch_csr_degree_scale(const int64_t *row_ptr, float *val,
                                   int64_t n, double *degree, hipStream_t s);
size_t start_vector_ws(int64_t n);
// Sum of degrees, zero-row count and v0 = d / sum(d); synchronises the
// stream and reports a zero / non-finite sum through *bad_host.
hipError_t launch_start_vector(const double *degree, int64_t n, double *v0,
                               int64_t *n_zero, void *ws, hipStream_t s,
                               int *bad_host);
// Structural check of a CSR graph; synchronises, *bad_host = 1 if invalid.
hipError_t launch_csr_check(const int64_t *row_ptr, const int32_t *col,
                            int64_t n, int64_t nnz, int *flag, hipStream_t s,
                            int *bad_host);

// power.hip
int64_t gemv_blocks(int64_t n);
int64_t spmv_blocks(int64_t n);
hipError_t launch_gemv(const float *W, int64_t n, int64_t ldw, const double *v,
                       double *y, double *partial, StopCtl ctl, bool use_ctl,
                       hipStream_t s);
// the same over a panel of m rows (n columns): y[0..m), partial[0..m/4)
hipError_t launch_gemv_panel(const float *W, int64_t m, int64_t n, int64_t ldw,
                             const double *v, double *y, double *partial, StopCtl ctl,
                             bool use_ctl, hipStream_t s);
// One launch per update of the dense loop for n <= a small bound (launch u:
// iteration u - 1's tau and update of the workgroup's rows, then iteration
// u's product with v formed on the fly; same values as the two-launch loop)
bool gemv_pipe_applies(int64_t n);
hipError_t launch_gemv_pipe(const float *W, int64_t n, int64_t ldw, double *v, double *delta,
                            const double *y_prev, const double *part_prev, double *y_cur,
                            double *part_cur, bool update, bool product, double *zero_slot,
                            StopCtl ctl, hipStream_t s);
// CSR product: up to 64 entries per row on average, the staged product
// (tiles of 256 rows, entries staged in LDS by all lanes, a thread per row
// summing in entry order), else 16 lanes per row; spmv_partials(n, nnz)
// |y| partial sums either way
bool spmv_staged(int64_t n, int64_t nnz);
int64_t spmv_partials(int64_t n, int64_t nnz);
hipError_t launch_spmv(const int64_t *row_ptr, const int32_t *col,
                       const float *val, int64_t n, int64_t nnz, const double *v,
                       double *y, double *partial, StopCtl ctl, bool use_ctl,
                       hipStream_t s);
// tau and the update in one launch (every workgroup forms tau itself in
// one fixed order, so all hold the same bits)
hipError_t launch_tau_update(const double *partial, int64_t nb, double *tau,
                             const double *y, double *v, double *delta, int64_t n,
                             StopCtl ctl, hipStream_t s);
hipError_t launch_init_state(double *ring, int64_t ring_len, int *err,
                             const double *v, double *delta, int64_t n,
                             bool copy_delta, hipStream_t s);

// sym.hip -- y = D^-1 (A v) over the packed upper tiles of a symmetric A:
// blocks of 256 indices (sym_blocks), storage bytes, the per-product
// partial sums (sym_part_bytes, caller scratch); two launches, the second
// writing one |y| partial per block of 256 rows when partial != nullptr;
// v == nullptr stands for v = 1 and degree == nullptr for no division
// (then y holds the row sums A v)
int64_t sym_blocks(int64_t n);
size_t sym_storage_bytes(int64_t n);
size_t sym_part_bytes(int64_t n);
hipError_t launch_sym_gemv(const float *As, int64_t n, const double *degree,
                           const double *v, double *y, double *part, double *partial,
                           StopCtl ctl, bool use_ctl, hipStream_t s);

// spmv_blocked.hip -- column-blocked copy of a CSR W for the product
struct CsrBlocked {
    int64_t n, nb;     // rows, column blocks
    int lanes;         // lanes per row in the product (1, 2, 4, 8 or 16)
    int64_t *base;     // [nb + 1] first entry of each block in colb / valb
    int32_t *rpb;      // [nb][n + 1] row offsets relative to base[b]
    int32_t *colb;     // [nnz]
    float *valb;       // [nnz]
    double *ypart;     // [nb][n] per-block row sums
};
// true when n spans 2 .. 32 column blocks of 2^18 columns
bool csr_blocked_applies(int64_t n);
// workspace bytes for the copy (0 when it does not apply)
size_t csr_blocked_ws(int64_t n, int64_t nnz);
// number of |y| partial sums the blocked product writes
int64_t csr_blocked_partials(int64_t n);
// Builds the copy in ws; synchronises.  *usable_host = 0 (nothing built)
// when a row's columns are not ascending, fewer than a quarter of the
// entries lie more than 2^17 columns from the diagonal, or a block holds
// >= 2^30 entries.
hipError_t build_csr_blocked(const int64_t *row_ptr, const int32_t *col,
                             const float *val, int64_t n, int64_t nnz, void *ws,
                             CsrBlocked *out, hipStream_t s, int *usable_host);
// Product (two launches): per-block row sums, then y and |y| partials.
hipError_t launch_spmv_blocked(const CsrBlocked &B, const double *v, double *y,
                               double *partial, StopCtl ctl, hipStream_t s);

// sort.hip -- stable LSD radix sort of n < 2^32 uint64 keys on their low
// `bits` bits (a multiple of 8), with an optional int32 payload (idxA and
// idxB null for keys alone).  The sorted arrays end in keyA / idxA (the
// pointers are swapped per pass).  hist: radix_hist_bytes(n) bytes, hsum:
// radix_hsum_bytes(n) bytes.
size_t radix_hist_bytes(int64_t n);
size_t radix_hsum_bytes(int64_t n);
// in-place exclusive scan of m uint32 values (total < 2^32); sums:
// scan_sums_bytes(m) bytes
size_t scan_sums_bytes(int64_t m);
hipError_t exclusive_scan_u32(uint32_t *a, int64_t m, uint32_t *sums, hipStream_t s);
hipError_t radix_sort_u64(uint64_t *&keyA, int32_t *&idxA, uint64_t *&keyB, int32_t *&idxB,
                          int64_t n, int bits, uint32_t *hist, uint32_t *hsum,
                          hipStream_t s);

// knn.hip -- exact kNN graph (d <= 16, k <= 64, 2 n k < 2^32); synchronises.
// *status_host = 1 when the candidate bounds failed to converge (nothing
// written).  row_ptr [n+1]; col and val hold up to 2 n k entries.  With
// perm_out (int32 [n], device) the nodes are numbered in the Morton order
// of the points: node p is point perm_out[p].
size_t knn_graph_ws(int64_t n, int32_t k);
hipError_t run_knn_graph(const float *X, int64_t n, int d, int k, float sigma,
                         int64_t *row_ptr, int32_t *col, float *val, int64_t *nnz_host,
                         int *status_host, void *ws, hipStream_t s,
                         int32_t *perm_out = nullptr);

// stream.hip -- read-bandwidth reference (not a step of the method):
// kReadStreamBlocks workgroups read n floats (n % 4 == 0, 16-byte aligned)
// once and write one float64 sum each to sink.
constexpr int kReadStreamBlocks = 1536;
hipError_t launch_read_stream(const float *x, int64_t n, double *sink, hipStream_t s);

// kmeans.hip
size_t kmeans_ws(int64_t n, int32_t k);
// Runs the whole exact 1-D k-means; synchronises the stream.
hipError_t run_kmeans1d(const double *v, int64_t n, int32_t k, int32_t *labels,
                        double *centroids, int32_t *k_eff, double *cost,
                        void *ws, hipStream_t s);

} // namespace gpic
