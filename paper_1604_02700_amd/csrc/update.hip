// One launch per update of the dense loop for small n (the Multiply,
// Reduction and Norm steps of Algorithm 2's loop and its stop test, with
// the update equation of section "Power Iteration Clustering: An
// Overview"): launch u of a run does iteration u - 1's tau and update and
// iteration u's product y = W v.  Its product takes gemv_kernel's rows and
// threads (4 rows per 512-thread workgroup) and its multiply-adds and
// reductions in the same order, so its y and its gemv_blocks(n) |y|
// partials are the two-launch loop's (up to 2,048 columns a thread has one
// column group, so there are no loads to run ahead).
#include "common.h"

namespace gpic {
namespace {

constexpr int kPipeRows = 4;            // rows per workgroup, as gemv_kernel
constexpr int kPipeThreads = 512;       // threads per workgroup, as gemv_kernel
constexpr int64_t kPipeMaxN = 2048;     // one launch per update up to this n

typedef float floatx4 __attribute__((ext_vector_type(4)));

// One launch per update for small n, where launches dominate.  Launch u of
// the loop forms, when `update` is set, iteration u - 1's tau from the
// previous launch's partials (every workgroup alone, in the order and with
// the reductions of tau_update_kernel: 1,024 summing lanes, thread t
// playing lanes t and t + 512), and for the workgroup's own rows
// v <- y_prev / tau, delta <- |v_new - v_old| and the statistic (integer
// atomic max); then, when `product` is set, iteration u's product
// y_cur = W v with v taken as y_prev / tau on the fly (the values the update
// stores), and its |y| partials.  Every value is the two-launch loop's, bit
// for bit; the last launch of a run only updates.  `zero_slot` is the
// statistic slot the next launch fills.
template <int R, int NT>
__global__ __launch_bounds__(NT) void gemv_pipe_kernel(
    const float *__restrict__ W, int64_t n, int64_t ldw, double *__restrict__ v,
    double *__restrict__ delta, const double *__restrict__ y_prev,
    const double *__restrict__ part_prev, int64_t nb, double *__restrict__ y_cur,
    double *__restrict__ part_cur, int update, int product, double *__restrict__ zero_slot,
    StopCtl ctl)
{
    static_assert(NT == 512, "two summing lanes per thread");
    __shared__ double red[R][NT / kWave];
    __shared__ double tred[2 * NT / kWave];
    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    if (zero_slot != nullptr && blockIdx.x == 0 && tid == 0)
        *zero_slot = 0.0;
    if (stop_reached(ctl))
        return;
    const int64_t row0 = (int64_t)blockIdx.x * R;
    double tau = 1.0;
    if (update) {
        double sa = 0.0, sb = 0.0;
        for (int64_t b = tid; b < nb; b += 2 * NT)
            sa += part_prev[b];
        for (int64_t b = tid + NT; b < nb; b += 2 * NT)
            sb += part_prev[b];
        sa = wave_sum(sa);
        sb = wave_sum(sb);
        if (lane == 0) {
            tred[wave] = sa;
            tred[NT / kWave + wave] = sb;
        }
        __syncthreads();
        double t = 0.0;
#pragma unroll
        for (int i = 0; i < 2 * NT / kWave; ++i)
            t += tred[i];
        if (!(t > 0.0) || !isfinite(t)) {
            if (blockIdx.x == 0 && tid == 0)
                *ctl.err = 1;
            return;                                  // uniform: t is the same everywhere
        }
        tau = t;
        double m = 0.0;
        if (tid < R && row0 + tid < n) {
            const int64_t i = row0 + tid;
            const double vn = y_prev[i] / t;
            const double dn = fabs(vn - v[i]);
            m = fabs(dn - delta[i]);
            v[i] = vn;
            delta[i] = dn;
        }
        if (wave == 0) {
            m = wave_max(m);
            if (tid == 0)
                atomicMax(reinterpret_cast<unsigned long long *>(ctl.cur_stat),
                          (unsigned long long)__double_as_longlong(m));
        }
    }
    if (!product)
        return;
    const floatx4 *rp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = (row0 + r < n) ? row0 + r : n - 1;
        rp[r] = reinterpret_cast<const floatx4 *>(W + i * ldw);
    }
    double acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.0;
    const int64_t n4 = n >> 2;
    const double2 *x2 = reinterpret_cast<const double2 *>(update ? y_prev : v);
#pragma unroll 1
    for (int64_t c = tid; c < n4; c += NT) {
        floatx4 w[R];
#pragma unroll
        for (int r = 0; r < R; ++r)
            w[r] = __builtin_nontemporal_load(rp[r] + c);
        double2 va = x2[2 * c];
        double2 vb = x2[2 * c + 1];
        if (update) {
            va.x = va.x / tau;
            va.y = va.y / tau;
            vb.x = vb.x / tau;
            vb.y = vb.y / tau;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            acc[r] = fma((double)w[r].x, va.x, acc[r]);
            acc[r] = fma((double)w[r].y, va.y, acc[r]);
            acc[r] = fma((double)w[r].z, vb.x, acc[r]);
            acc[r] = fma((double)w[r].w, vb.y, acc[r]);
        }
    }
    const int64_t tail = n - (n4 << 2);
    if (tid < tail) {
        const int64_t j = (n4 << 2) + tid;
        const double vj = update ? y_prev[j] / tau : v[j];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float *row = reinterpret_cast<const float *>(rp[r]);
            acc[r] = fma((double)row[j], vj, acc[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const double t = wave_sum(acc[r]);
        if (lane == 0)
            red[r][wave] = t;
    }
    __syncthreads();
    if (tid == 0) {
        double part = 0.0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            double t = 0.0;
#pragma unroll
            for (int w = 0; w < NT / kWave; ++w)
                t += red[r][w];
            if (row0 + r < n) {
                y_cur[row0 + r] = t;
                part += fabs(t);
            }
        }
        part_cur[blockIdx.x] = part;
    }
}

} // namespace

bool gemv_pipe_applies(int64_t n) { return n <= kPipeMaxN; }

hipError_t launch_gemv_pipe(const float *W, int64_t n, int64_t ldw, double *v, double *delta,
                            const double *y_prev, const double *part_prev, double *y_cur,
                            double *part_cur, bool update, bool product, double *zero_slot,
                            StopCtl ctl, hipStream_t s)
{
    hipLaunchKernelGGL((gemv_pipe_kernel<kPipeRows, kPipeThreads>), dim3((unsigned)gemv_blocks(n)),
                       dim3(kPipeThreads), 0, s, W, n, ldw, v, delta, y_prev, part_prev,
                       gemv_blocks(n), y_cur, part_cur, update ? 1 : 0, product ? 1 : 0,
                       zero_slot, ctl);
    return hipGetLastError();
}

} // namespace gpic
