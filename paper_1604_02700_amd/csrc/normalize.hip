// Degrees, row normalisation and the start vector for gfx950.
//
// d_ii = sum_j a_ij and W = D^-1 A (section "Spectral Cluster"; the RowSum
// and NormMat steps of Algorithm 2); v0 = D / sum(D) (its Reduction and Norm
// steps before the loop).  All sums are float64 in a fixed order: within a
// row by lane-strided partial sums and a butterfly, across rows by per-block
// partials reduced in ascending block order by a single workgroup.
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;

// One workgroup per row; float4 loads along the row.
__global__ __launch_bounds__(kThreads) void dense_degree_kernel(
    const float *__restrict__ A, int64_t n, int64_t lda, double *__restrict__ degree)
{
    __shared__ double red[kThreads / kWave];
    const int64_t i = blockIdx.x;
    const float *row = A + i * lda;
    const int64_t n4 = n >> 2;
    double s = 0.0;
    for (int64_t c = threadIdx.x; c < n4; c += kThreads) {
        const float4 w = reinterpret_cast<const float4 *>(row)[c];
        s += (double)w.x;
        s += (double)w.y;
        s += (double)w.z;
        s += (double)w.w;
    }
    const int64_t tail = n - (n4 << 2);
    if (threadIdx.x < tail)
        s += (double)row[(n4 << 2) + threadIdx.x];
    const double t = block_sum<kThreads>(s, red);
    if (threadIdx.x == 0)
        degree[i] = t;
}

// W_ij = A_ij * r_i in place with r_i = float32(1 / d_i) (the float64
// reciprocal rounded once); a zero-degree row is written as zeros.
__global__ __launch_bounds__(kThreads) void dense_scale_kernel(
    float *__restrict__ A, int64_t n, int64_t lda, const double *__restrict__ degree)
{
    const int64_t i = blockIdx.x;
    float *row = A + i * lda;
    const double di = degree[i];
    const float r = (di == 0.0) ? 0.0f : (float)(1.0 / di);
    const int64_t n4 = n >> 2;
    for (int64_t c = threadIdx.x; c < n4; c += kThreads) {
        float4 w = reinterpret_cast<float4 *>(row)[c];
        w.x *= r;
        w.y *= r;
        w.z *= r;
        w.w *= r;
        reinterpret_cast<float4 *>(row)[c] = w;
    }
    const int64_t tail = n - (n4 << 2);
    if (threadIdx.x < tail) {
        float *p = row + (n4 << 2) + threadIdx.x;
        *p *= r;
    }
}

// CSR: 16 lanes per row; lane-strided sums, a 16-lane butterfly, then the
// row is scaled in place by float32(1 / d_i).
constexpr int kCsrLanes = 16;

__global__ __launch_bounds__(kThreads) void csr_degree_scale_kernel(
    const int64_t *__restrict__ row_ptr, float *__restrict__ val, int64_t n,
    double *__restrict__ degree)
{
    const int64_t i = (int64_t)blockIdx.x * (kThreads / kCsrLanes) +
                      threadIdx.x / kCsrLanes;
    const int sl = threadIdx.x % kCsrLanes;
    const bool live = i < n;
    const int64_t b = live ? row_ptr[i] : 0, e = live ? row_ptr[i + 1] : 0;
    double s = 0.0;
    for (int64_t p = b + sl; p < e; p += kCsrLanes)
        s += (double)val[p];
    s = group_sum<kCsrLanes>(s);
    if (!live)
        return;
    if (sl == 0)
        degree[i] = s;
    const float r = (s == 0.0) ? 0.0f : (float)(1.0 / s);
    for (int64_t p = b + sl; p < e; p += kCsrLanes)
        val[p] *= r;
}

// ---- start vector: per-block partial sums and zero counts, a single-group
// ---- reduction, then v0 = d / sum(d).
constexpr int kChunk = 4096;

struct StartWs {
    double total;
    int64_t nzero;
    int bad;
    int pad;
};

__global__ __launch_bounds__(kThreads) void degree_partials_kernel(
    const double *__restrict__ degree, int64_t n, double *__restrict__ psum,
    int64_t *__restrict__ pzero)
{
    __shared__ double red[kThreads / kWave];
    const int64_t b = (int64_t)blockIdx.x * kChunk;
    const int64_t e = (b + kChunk < n) ? b + kChunk : n;
    double s = 0.0, z = 0.0;
    for (int64_t i = b + threadIdx.x; i < e; i += kThreads) {
        const double x = degree[i];
        s += x;
        z += (x == 0.0) ? 1.0 : 0.0;
    }
    const double ts = block_sum<kThreads>(s, red);
    const double tz = block_sum<kThreads>(z, red);
    if (threadIdx.x == 0) {
        psum[blockIdx.x] = ts;
        pzero[blockIdx.x] = (int64_t)tz;
    }
}

__global__ __launch_bounds__(1024) void degree_total_kernel(
    const double *__restrict__ psum, const int64_t *__restrict__ pzero,
    int64_t nb, StartWs *__restrict__ st, int64_t *__restrict__ n_zero)
{
    __shared__ double red[1024 / kWave];
    double s = 0.0, z = 0.0;
    for (int64_t b = threadIdx.x; b < nb; b += 1024) {
        s += psum[b];
        z += (double)pzero[b];
    }
    const double ts = block_sum<1024>(s, red);
    const double tz = block_sum<1024>(z, red);
    if (threadIdx.x == 0) {
        st->total = ts;
        st->nzero = (int64_t)tz;
        st->bad = !(ts > 0.0) || !isfinite(ts);
        if (n_zero != nullptr)
            *n_zero = (int64_t)tz;
    }
}

__global__ __launch_bounds__(kThreads) void start_vector_kernel(
    const double *__restrict__ degree, int64_t n, const StartWs *__restrict__ st,
    double *__restrict__ v0)
{
    if (st->bad)
        return;
    const double total = st->total;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n)
        v0[i] = degree[i] / total;
}

// row_ptr[0] == 0, row_ptr[n] == nnz, row_ptr non-decreasing, every column
// in [0, n).  Any violation sets *flag.
__global__ __launch_bounds__(kThreads) void csr_check_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    int64_t n, int64_t nnz, int *__restrict__ flag)
{
    const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    bool bad = false;
    if (t0 == 0)
        bad = row_ptr[0] != 0 || row_ptr[n] != nnz;
    for (int64_t i = t0; i < n; i += stride)
        bad = bad || row_ptr[i + 1] < row_ptr[i];
    for (int64_t p = t0; p < nnz; p += stride) {
        const int32_t c = col[p];
        bad = bad || c < 0 || (int64_t)c >= n;
    }
    if (bad)
        *flag = 1;
}

__global__ void clear_flag_kernel(int *flag) { *flag = 0; }

} // namespace

hipError_t launch_csr_check(const int64_t *row_ptr, const int32_t *col,
                            int64_t n, int64_t nnz, int *flag, hipStream_t s,
                            int *bad_host)
{
    hipLaunchKernelGGL(clear_flag_kernel, dim3(1), dim3(1), 0, s, flag);
    const int64_t m = (n > nnz) ? n : nnz;
    int64_t b = (m + kThreads - 1) / kThreads;
    if (b > 4096)
        b = 4096;
    if (b < 1)
        b = 1;
    hipLaunchKernelGGL(csr_check_kernel, dim3((unsigned)b), dim3(kThreads), 0, s,
                       row_ptr, col, n, nnz, flag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    int bad = 0;
    e = hipMemcpyAsync(&bad, flag, sizeof(int), hipMemcpyDeviceToHost, s);
    if (e != hipSuccess)
        return e;
    e = hipStreamSynchronize(s);
    if (e != hipSuccess)
        return e;
    *bad_host = bad;
    return hipSuccess;
}

hipError_t launch_dense_degree(const float *A, int64_t n, int64_t lda,
                               double *degree, hipStream_t s)
{
    hipLaunchKernelGGL(dense_degree_kernel, dim3((unsigned)n), dim3(kThreads), 0,
                       s, A, n, lda, degree);
    return hipGetLastError();
}

hipError_t launch_dense_scale(float *A, int64_t n, int64_t lda,
                              const double *degree, hipStream_t s)
{
    hipLaunchKernelGGL(dense_scale_kernel, dim3((unsigned)n), dim3(kThreads), 0,
                       s, A, n, lda, degree);
    return hipGetLastError();
}

hipError_t launch_csr_degree_scale(const int64_t *row_ptr, float *val,
                                   int64_t n, double *degree, hipStream_t s)
{
    const int64_t rows_per = kThreads / kCsrLanes;
    hipLaunchKernelGGL(csr_degree_scale_kernel,
                       dim3((unsigned)((n + rows_per - 1) / rows_per)),
                       dim3(kThreads), 0, s, row_ptr, val, n, degree);
    return hipGetLastError();
}

static int64_t start_blocks(int64_t n) { return (n + kChunk - 1) / kChunk; }

size_t start_vector_ws(int64_t n)
{
    const int64_t nb = start_blocks(n);
    return 256 + (size_t)nb * 16 + 512;
}

// ws layout: [StartWs (256 B)][psum nb doubles][pzero nb int64]
hipError_t launch_start_vector(const double *degree, int64_t n, double *v0,
                               int64_t *n_zero, void *ws, hipStream_t s,
                               int *bad_host)
{
    const int64_t nb = start_blocks(n);
    char *base = static_cast<char *>(ws);
    StartWs *st = reinterpret_cast<StartWs *>(base);
    double *psum = reinterpret_cast<double *>(base + 256);
    int64_t *pzero = reinterpret_cast<int64_t *>(base + 256 + nb * 8);
    hipLaunchKernelGGL(degree_partials_kernel, dim3((unsigned)nb), dim3(kThreads),
                       0, s, degree, n, psum, pzero);
    hipLaunchKernelGGL(degree_total_kernel, dim3(1), dim3(1024), 0, s, psum,
                       pzero, nb, st, n_zero);
    hipLaunchKernelGGL(start_vector_kernel,
                       dim3((unsigned)((n + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, degree, n, st, v0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    int bad = 0;
    e = hipMemcpyAsync(&bad, &st->bad, sizeof(int), hipMemcpyDeviceToHost, s);
    if (e != hipSuccess)
        return e;
    e = hipStreamSynchronize(s);
    if (e != hipSuccess)
        return e;
    *bad_host = bad;
    return hipSuccess;
}

} // namespace gpic
