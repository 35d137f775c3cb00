// Power-iteration kernels for gfx950: the CSR product y = W v (the dense
// product is in gemv.hip),
// the L1 norm tau = sum_i |y_i|, and the update
//   v_{t+1} = y / tau,  delta_{t+1} = |v_{t+1} - v_t|,
//   s_t = max_i |delta_{t+1,i} - delta_{t,i}|
// of Algorithm 1 (update equation of section "Power Iteration Clustering:
// An Overview"; the Multiply, Reduction and Norm steps of Algorithm 2's loop
// and its stop test).
//
// One update is three launches on the caller's stream: product (writes y and
// per-block partial sums of |y_i|), tau (one workgroup sums the partials in
// ascending block order), update (grid-wide; block maxima of the statistic
// are combined with an integer atomic max on the bit pattern of the
// non-negative float64, which is order-free and therefore deterministic).
// Up to 16,384 rows, tau and the update share one launch, in which every
// workgroup forms tau itself in the same order (so the same bits).
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kSpmvLanes = 16;      // lanes per CSR row
constexpr int kSpmvRows = 32;       // rows per workgroup of the CSR product
constexpr int kSpmvUnroll = 4;      // independent gathers in flight per lane
constexpr int64_t kTauUpdateMaxN = 16384;   // one launch for tau and the update

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

// tau = sum of the block partials, by one workgroup in a fixed order.
__global__ __launch_bounds__(1024) void reduce_tau_kernel(
    const double *__restrict__ partial, int64_t nb, double *__restrict__ tau,
    StopCtl ctl)
{
    __shared__ double red[1024 / kWave];
    if (stop_reached(ctl))
        return;
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < nb; b += 1024)
        s += partial[b];
    const double t = block_sum<1024>(s, red);
    if (threadIdx.x == 0) {
        *tau = t;
        if (!(t > 0.0) || !isfinite(t))
            *ctl.err = 1;
    }
}

// v <- y / tau, delta <- |v_new - v_old|, statistic = max |delta_new - delta|.
__global__ __launch_bounds__(kThreads) void update_kernel(
    const double *__restrict__ y, const double *__restrict__ tau,
    double *__restrict__ v, double *__restrict__ delta, int64_t n, StopCtl ctl)
{
    __shared__ double red[kThreads / kWave];
    if (stop_reached(ctl))
        return;
    const double t = *tau;
    double s = 0.0;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += stride) {
        const double vn = y[i] / t;
        const double dn = fabs(vn - v[i]);
        s = fmax(s, fabs(dn - delta[i]));
        v[i] = vn;
        delta[i] = dn;
    }
    const double m = block_max<kThreads>(s, red);
    if (threadIdx.x == 0)
        atomicMax(reinterpret_cast<unsigned long long *>(ctl.cur_stat),
                  (unsigned long long)__double_as_longlong(m));
}

// Both steps in one launch for small n: every workgroup forms tau from the
// partials exactly as reduce_tau_kernel does (same order, so the same
// bits), then updates its rows.
__global__ __launch_bounds__(1024) void tau_update_kernel(
    const double *__restrict__ partial, int64_t nb, double *__restrict__ tau,
    const double *__restrict__ y, double *__restrict__ v, double *__restrict__ delta,
    int64_t n, StopCtl ctl)
{
    __shared__ double red[1024 / kWave];
    if (stop_reached(ctl))
        return;
    double s = 0.0;
    for (int64_t b = threadIdx.x; b < nb; b += 1024)
        s += partial[b];
    const double t = block_sum<1024>(s, red);
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
    for (int64_t i = (int64_t)blockIdx.x * 1024 + threadIdx.x; i < n; i += stride) {
        const double vn = y[i] / t;
        const double dn = fabs(vn - v[i]);
        m = fmax(m, fabs(dn - delta[i]));
        v[i] = vn;
        delta[i] = dn;
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

hipError_t launch_spmv(const int64_t *row_ptr, const int32_t *col,
                       const float *val, int64_t n, const double *v, double *y,
                       double *partial, StopCtl ctl, bool use_ctl, hipStream_t s)
{
    hipLaunchKernelGGL(spmv_kernel, dim3((unsigned)spmv_blocks(n)),
                       dim3(kThreads), 0, s, row_ptr, col, val, n, v, y, partial,
                       ctl, use_ctl ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_reduce_tau(const double *partial, int64_t nb, double *tau,
                             StopCtl ctl, hipStream_t s)
{
    hipLaunchKernelGGL(reduce_tau_kernel, dim3(1), dim3(1024), 0, s, partial, nb,
                       tau, ctl);
    return hipGetLastError();
}

bool tau_update_fused(int64_t n) { return n <= kTauUpdateMaxN; }

hipError_t launch_tau_update(const double *partial, int64_t nb, double *tau,
                             const double *y, double *v, double *delta, int64_t n,
                             StopCtl ctl, hipStream_t s)
{
    hipLaunchKernelGGL(tau_update_kernel, dim3((unsigned)((n + 1023) / 1024)), dim3(1024),
                       0, s, partial, nb, tau, y, v, delta, n, ctl);
    return hipGetLastError();
}

hipError_t launch_update(const double *y, const double *tau, double *v,
                         double *delta, int64_t n, StopCtl ctl, hipStream_t s)
{
    hipLaunchKernelGGL(update_kernel, dim3(grid_for(n, 2048)), dim3(kThreads), 0,
                       s, y, tau, v, delta, n, ctl);
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
