// Dense product y = W v for gfx950 (the Multiply step of Algorithm 2's
// loop; W v of the update equation of section "Power Iteration Clustering:
// An Overview").  W is float32 [n x ldw] row-major, v and y float64; each
// workgroup also writes the sum of |y_i| over its rows for the L1 norm.
// This is the dominant kernel of the dense path: it streams 4 n^2 bytes of
// W per product and is bound by HBM reads.
#include "common.h"

namespace gpic {
namespace {

constexpr int kGemvRows = 4;        // rows per workgroup of the dense product
constexpr int kGemvThreads = 512;   // threads per workgroup of the dense product

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Dense product over m rows of n columns (m = n for a whole W; m < n for a
// row panel of it).  A workgroup owns kGemvRows consecutive rows; every thread
// takes 16-byte column groups c, c + NT, ... and keeps one float64
// accumulator per row, so each 32-byte slice of v it loads is reused across
// all rows of the block.  W is streamed exactly once per product, so its
// loads are non-temporal (they do not displace v, which every workgroup
// re-reads, from the caches).  Each thread keeps the W loads of its next two
// column groups in flight while it multiplies the current one (at n = 50,000:
// 1,457 us per product, against 1,510 us with each group's loads issued in its
// own iteration; same summation order, same bits).  Rows past m are clamped
// for loading and never written.
template <int R, int NT>
__global__ __launch_bounds__(NT) void gemv_kernel(
    const float *__restrict__ W, int64_t m, int64_t n, int64_t ldw,
    const double *__restrict__ v, double *__restrict__ y,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    __shared__ double red[R][NT / kWave];
    if (use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int64_t row0 = (int64_t)blockIdx.x * R;
    const floatx4 *rp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = (row0 + r < m) ? row0 + r : m - 1;
        rp[r] = reinterpret_cast<const floatx4 *>(W + i * ldw);
    }
    double acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.0;

    const int64_t n4 = n >> 2;
    const double2 *v2 = reinterpret_cast<const double2 *>(v);
    floatx4 wn[R], wm[R];
    if ((int64_t)threadIdx.x < n4) {
#pragma unroll
        for (int r = 0; r < R; ++r)
            wn[r] = __builtin_nontemporal_load(rp[r] + threadIdx.x);
    }
    if ((int64_t)threadIdx.x + NT < n4) {
#pragma unroll
        for (int r = 0; r < R; ++r)
            wm[r] = __builtin_nontemporal_load(rp[r] + threadIdx.x + NT);
    }
#pragma unroll 1
    for (int64_t c = threadIdx.x; c < n4; c += NT) {
        floatx4 w[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            w[r] = wn[r];
            wn[r] = wm[r];
        }
        if (c + 2 * NT < n4) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                wm[r] = __builtin_nontemporal_load(rp[r] + c + 2 * NT);
        }
        const double2 va = v2[2 * c];
        const double2 vb = v2[2 * c + 1];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            acc[r] = fma((double)w[r].x, va.x, acc[r]);
            acc[r] = fma((double)w[r].y, va.y, acc[r]);
            acc[r] = fma((double)w[r].z, vb.x, acc[r]);
            acc[r] = fma((double)w[r].w, vb.y, acc[r]);
        }
    }
    const int64_t tail = n - (n4 << 2);
    if (threadIdx.x < tail) {
        const int64_t j = (n4 << 2) + threadIdx.x;
        const double vj = v[j];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float *row = reinterpret_cast<const float *>(rp[r]);
            acc[r] = fma((double)row[j], vj, acc[r]);
        }
    }
    const int wave = threadIdx.x / kWave;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const double t = wave_sum(acc[r]);
        if ((threadIdx.x % kWave) == 0)
            red[r][wave] = t;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double part = 0.0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            double t = 0.0;
#pragma unroll
            for (int w = 0; w < NT / kWave; ++w)
                t += red[r][w];
            if (row0 + r < m) {
                y[row0 + r] = t;
                part += fabs(t);
            }
        }
        if (partial != nullptr)
            partial[blockIdx.x] = part;
    }
}

} // namespace

int64_t gemv_blocks(int64_t n) { return (n + kGemvRows - 1) / kGemvRows; }

hipError_t launch_gemv(const float *W, int64_t n, int64_t ldw, const double *v,
                       double *y, double *partial, StopCtl ctl, bool use_ctl,
                       hipStream_t s)
{
    return launch_gemv_panel(W, n, n, ldw, v, y, partial, ctl, use_ctl, s);
}

hipError_t launch_gemv_panel(const float *W, int64_t m, int64_t n, int64_t ldw,
                             const double *v, double *y, double *partial, StopCtl ctl,
                             bool use_ctl, hipStream_t s)
{
    hipLaunchKernelGGL((gemv_kernel<kGemvRows, kGemvThreads>),
                       dim3((unsigned)gemv_blocks(m)), dim3(kGemvThreads), 0, s, W,
                       m, n, ldw, v, y, partial, ctl, use_ctl ? 1 : 0);
    return hipGetLastError();
}

} // namespace gpic
