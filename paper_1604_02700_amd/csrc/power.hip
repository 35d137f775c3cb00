// Power-iteration kernels for gfx950: the CSR product y = W v (the dense
// product is in gemv.hip),
// the L1 norm tau = sum_i |y_i|, and the update
//   v_{t+1} = y / tau,  delta_{t+1} = |v_{t+1} - v_t|,
//   s_t = max_i |delta_{t+1,i} - delta_{t,i}|
// of Algorithm 1 (update equation of section "Power Iteration Clustering:
// An Overview"; the Multiply, Reduction and Norm steps of Algorithm 2's loop
// and its stop test).
//
// One update is two launches on the caller's stream: the product (writes y
// and per-block partial sums of |y_i|), then tau and the update in one
// launch (every workgroup sums the partials itself in one fixed order, so
// all hold the same tau; block maxima of the statistic are combined with an
// integer atomic max on the bit pattern of the non-negative float64, which
// is order-free and therefore deterministic).  Up to 2,048 rows of a dense
// W they share one launch with the next product (update.hip).
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kSpmvLanes = 16;      // lanes per CSR row
constexpr int kSpmvRows = 32;       // rows per workgroup of the CSR product
constexpr int kSpmvUnroll = 4;      // independent gathers in flight per lane
constexpr int kStagedRows = 256;    // rows per tile of the staged CSR product
constexpr int kStageK = 24;         // entries per thread per round of the staged product
constexpr int kStage = kStageK * kThreads;   // entries staged in LDS per round (48 KB)
constexpr int64_t kStagedMaxAvg = 64;   // mean entries per row up to which it is used
constexpr int kXcds = 8;            // workgroups go round-robin to the 8 XCDs

// CSR product: 16 lanes per row, lane l summing entries l, l + 16, ... of
// its row in that order, then a 16-lane butterfly.  The workgroup's row
// pointers are staged in LDS first, and each lane issues kSpmvUnroll column
// loads and then kSpmvUnroll gathers of v before using any of them, so
// several gathers are in flight per lane (the order of the sum is unchanged).
__global__ __launch_bounds__(kThreads) void spmv_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, int64_t n, const double *__restrict__ v,
    double *__restrict__ y, double *__restrict__ partial, StopCtl ctl,
    int use_ctl)
{
    __shared__ double red[kThreads / kWave];
    __shared__ int64_t rp[kSpmvRows + 1];
    if (use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int64_t base = (int64_t)blockIdx.x * kSpmvRows;
    for (int t = threadIdx.x; t <= kSpmvRows; t += kThreads)
        rp[t] = row_ptr[base + t < n ? base + t : n];
    __syncthreads();
    const int sl = threadIdx.x % kSpmvLanes;
    const int grp = threadIdx.x / kSpmvLanes;
    constexpr int groups = kThreads / kSpmvLanes;
    double part = 0.0;
    for (int pass = 0; pass < kSpmvRows / groups; ++pass) {
        const int li = pass * groups + grp;
        const int64_t i = base + li;
        double s = 0.0;
        if (i < n) {
            const int64_t b = rp[li], e = rp[li + 1];
            for (int64_t p0 = b + sl; p0 < e; p0 += kSpmvLanes * kSpmvUnroll) {
                int32_t c[kSpmvUnroll];
                float w[kSpmvUnroll];
                double x[kSpmvUnroll];
#pragma unroll
                for (int u = 0; u < kSpmvUnroll; ++u) {
                    const int64_t p = p0 + (int64_t)u * kSpmvLanes;
                    c[u] = p < e ? col[p] : -1;
                    w[u] = p < e ? val[p] : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < kSpmvUnroll; ++u)
                    x[u] = c[u] >= 0 ? v[c[u]] : 0.0;
#pragma unroll
                for (int u = 0; u < kSpmvUnroll; ++u)
                    if (c[u] >= 0)
                        s = fma((double)w[u], x[u], s);
            }
        }
        s = group_sum<kSpmvLanes>(s);
        if (i < n && sl == 0) {
            y[i] = s;
            part += fabs(s);
        }
    }
    const double t = block_sum<kThreads>(part, red);
    if (threadIdx.x == 0 && partial != nullptr)
        partial[blockIdx.x] = t;
}

// CSR product for short rows (a kNN graph holds about 45 entries per row):
// with 16 lanes per row, most lanes of a gather instruction sit idle while
// the wave finishes its longest row.  Here a workgroup owns a tile of 256
// consecutive rows and walks the tile's entries in storage order in rounds
// of kStage: every thread loads kStageK columns and weights (coalesced, all
// in flight at once), gathers v at those columns (all in flight), and
// stages the float64 products w_p v[col_p] in LDS; after a barrier a thread
// per row adds its row's products in entry order -- the oracle's own
// arithmetic, a product rounded then added -- carrying its sum across
// rounds.  The next round's columns and weights are loaded while the
// current round's rows are summed.  Tiles are numbered XCD-major: the
// workgroups one XCD runs hold a contiguous eighth of the rows, so with a
// numbering that keeps graph neighbours close, the v entries an XCD
// gathers stay in its L2.
__global__ __launch_bounds__(kThreads) void spmv_staged_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, int64_t n, int64_t tiles, int64_t per_xcd,
    const double *__restrict__ v, double *__restrict__ y, double *__restrict__ partial,
    StopCtl ctl, int use_ctl)
{
    __shared__ int64_t rp[kStagedRows + 1];
    __shared__ double ps[kStage];
    __shared__ double red[kThreads / kWave];
    if (use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int64_t tile = (int64_t)(blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (tile >= tiles)
        return;                                      // uniform over the workgroup
    const int64_t row0 = tile * kStagedRows;
    for (int t = threadIdx.x; t <= kStagedRows; t += kThreads)
        rp[t] = row_ptr[row0 + t < n ? row0 + t : n];
    __syncthreads();
    const int64_t e0 = rp[0], e1 = rp[kStagedRows];
    const int li = threadIdx.x;
    const int64_t i = row0 + li;
    const int64_t rs = rp[li], re = rp[li + 1];      // this thread's row (empty past n)
    int32_t c[kStageK];
    float w[kStageK];
    auto load = [&](int64_t r0) {
#pragma unroll
        for (int u = 0; u < kStageK; ++u) {
            const int64_t p = r0 + threadIdx.x + (int64_t)u * kThreads;
            c[u] = p < e1 ? col[p] : -1;
            w[u] = p < e1 ? val[p] : 0.0f;
        }
    };
    double s = 0.0;
    load(e0);
    for (int64_t r0 = e0; r0 < e1; r0 += kStage) {
        double x[kStageK];
#pragma unroll
        for (int u = 0; u < kStageK; ++u)
            x[u] = c[u] >= 0 ? v[c[u]] : 0.0;
#pragma unroll
        for (int u = 0; u < kStageK; ++u)
            ps[threadIdx.x + u * kThreads] = (double)w[u] * x[u];   // 0 past the tile
        __syncthreads();
        if (r0 + kStage < e1)
            load(r0 + kStage);                       // in flight during the sums
        const int64_t r1 = (r0 + kStage < e1) ? r0 + kStage : e1;
        // the row's slice of this round, clamped in 64 bits before it is
        // narrowed: a row outside the round gets the empty slice (rows may
        // lie far from the round in a tile of more than 2^31 entries)
        const int64_t lo = (rs > r0) ? rs : r0;
        const int64_t hi = (re < r1) ? re : r1;
        const int a = (hi > lo) ? (int)(lo - r0) : 0;
        const int z = (hi > lo) ? (int)(hi - r0) : 0;
        int p = a;
        for (; p + 4 <= z; p += 4) {
            double q[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                q[u] = ps[p + u];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                s = s + q[u];
        }
        for (; p < z; ++p)
            s = s + ps[p];
        __syncthreads();                             // before the next round's stage
    }
    double yabs = 0.0;
    if (i < n) {
        y[i] = s;
        yabs = fabs(s);
    }
    const double t = block_sum<kThreads>(yabs, red);
    if (threadIdx.x == 0 && partial != nullptr)
        partial[tile] = t;
}

// Lane t of a 1,024-thread workgroup: the sum of partial[t], partial[t +
// 1024], ... in that order, eight loads in flight at a time.
__device__ __forceinline__ double lane_partial_sum(const double *__restrict__ partial,
                                                   int64_t nb)
{
    double s = 0.0;
    int64_t b = threadIdx.x;
    for (; b + 7 * 1024 < nb; b += 8 * 1024) {
        double x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            x[u] = partial[b + u * 1024];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            s += x[u];
    }
    for (; b < nb; b += 1024)
        s += partial[b];
    return s;
}

// tau and the update in one launch: every workgroup forms tau from the
// partials in the same fixed order (lane t of 1,024 sums partial[t],
// partial[t + 1024], ... in that order, then the block sum: the same bits
// everywhere), then updates its rows: v <- y / tau, delta <- |v_new -
// v_old|, statistic = max |delta_new - delta|, kUpdateRows rows per thread
// per step with their loads in flight (the maximum is order-free).  Each
// workgroup adds its maximum to the statistic with one same-address
// atomic, and those serialise (about 12 ns each), so at most kUpdateBlocks
// workgroups: at n = 2M an update grid of 2,048 workgroups of 256 threads
// cost 292 us per update of the CSR loop, 256 of 1,024 threads 278
// (128-512 workgroups, 2-16 rows per step: 278-334), and tau in the same
// launch instead of a one-workgroup launch of its own 275.
constexpr int kUpdateRows = 4;              // rows per thread per step
constexpr int64_t kUpdateBlocks = 256;
__global__ __launch_bounds__(1024) void tau_update_kernel(
    const double *__restrict__ partial, int64_t nb, double *__restrict__ tau,
    const double *__restrict__ y, double *__restrict__ v, double *__restrict__ delta,
    int64_t n, StopCtl ctl)
{
    __shared__ double red[1024 / kWave];
    if (stop_reached(ctl))
        return;
    const double t = block_sum<1024>(lane_partial_sum(partial, nb), red);
    const bool bad = !(t > 0.0) || !isfinite(t);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        *tau = t;
        if (bad)
            *ctl.err = 1;
    }
    if (bad)
        return;                                     // uniform: t is the same everywhere
    double m = 0.0;
    const int64_t stride = (int64_t)gridDim.x * 1024;
    constexpr int U = kUpdateRows;
    for (int64_t i0 = (int64_t)blockIdx.x * 1024 + threadIdx.x; i0 < n; i0 += U * stride) {
        double yy[U], vv[U], dd[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + u * stride;
            yy[u] = i < n ? y[i] : 0.0;
            vv[u] = i < n ? v[i] : 0.0;
            dd[u] = i < n ? delta[i] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + u * stride;
            if (i < n) {
                const double vn = yy[u] / t;
                const double dn = fabs(vn - vv[u]);
                m = fmax(m, fabs(dn - dd[u]));
                v[i] = vn;
                delta[i] = dn;
            }
        }
    }
    m = block_max<1024>(m, red);
    if (threadIdx.x == 0)
        atomicMax(reinterpret_cast<unsigned long long *>(ctl.cur_stat),
                  (unsigned long long)__double_as_longlong(m));
}

__global__ __launch_bounds__(kThreads) void init_state_kernel(
    double *__restrict__ ring, int64_t ring_len, int *__restrict__ err,
    const double *__restrict__ v, double *__restrict__ delta, int64_t n,
    int copy_delta)
{
    const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    if (t0 == 0)
        *err = 0;
    for (int64_t i = t0; i < ring_len; i += stride)
        ring[i] = 0.0;
    if (copy_delta)
        for (int64_t i = t0; i < n; i += stride)
            delta[i] = v[i];
}

unsigned grid_for(int64_t n, int64_t cap)
{
    int64_t b = (n + kThreads - 1) / kThreads;
    if (b > cap)
        b = cap;
    if (b < 1)
        b = 1;
    return (unsigned)b;
}

} // namespace

int64_t spmv_blocks(int64_t n) { return (n + kSpmvRows - 1) / kSpmvRows; }

bool spmv_staged(int64_t n, int64_t nnz) { return nnz <= kStagedMaxAvg * n; }

int64_t spmv_partials(int64_t n, int64_t nnz)
{
    return spmv_staged(n, nnz) ? (n + kStagedRows - 1) / kStagedRows : spmv_blocks(n);
}

hipError_t launch_spmv(const int64_t *row_ptr, const int32_t *col,
                       const float *val, int64_t n, int64_t nnz, const double *v,
                       double *y, double *partial, StopCtl ctl, bool use_ctl,
                       hipStream_t s)
{
    if (spmv_staged(n, nnz)) {
        const int64_t tiles = (n + kStagedRows - 1) / kStagedRows;
        const int64_t per = (tiles + kXcds - 1) / kXcds;
        hipLaunchKernelGGL(spmv_staged_kernel, dim3((unsigned)(per * kXcds)), dim3(kThreads),
                           0, s, row_ptr, col, val, n, tiles, per, v, y, partial, ctl,
                           use_ctl ? 1 : 0);
    } else {
        hipLaunchKernelGGL(spmv_kernel, dim3((unsigned)spmv_blocks(n)),
                           dim3(kThreads), 0, s, row_ptr, col, val, n, v, y, partial,
                           ctl, use_ctl ? 1 : 0);
    }
    return hipGetLastError();
}

hipError_t launch_tau_update(const double *partial, int64_t nb, double *tau,
                             const double *y, double *v, double *delta, int64_t n,
                             StopCtl ctl, hipStream_t s)
{
    int64_t b = (n + 1023) / 1024;
    b = b < 1 ? 1 : (b > kUpdateBlocks ? kUpdateBlocks : b);
    hipLaunchKernelGGL(tau_update_kernel, dim3((unsigned)b), dim3(1024), 0, s, partial, nb, tau,
                       y, v, delta, n, ctl);
    return hipGetLastError();
}

hipError_t launch_init_state(double *ring, int64_t ring_len, int *err,
                             const double *v, double *delta, int64_t n,
                             bool copy_delta, hipStream_t s)
{
    const int64_t m = copy_delta ? (n > ring_len ? n : ring_len) : ring_len;
    hipLaunchKernelGGL(init_state_kernel, dim3(grid_for(m, 2048)), dim3(kThreads),
                       0, s, ring, ring_len, err, v, delta, n,
                       copy_delta ? 1 : 0);
    return hipGetLastError();
}

} // namespace gpic
