// Read-bandwidth reference for the dense product: a plain stream of 16-byte
// non-temporal loads over a buffer, summed so that no load can be dropped.
// It is not a step of the method; the benchmark times it on the same buffer
// as W to report the product's rate against the read ceiling this device
// reaches in the same run.
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;

typedef float floatx4 __attribute__((ext_vector_type(4)));

// A fixed grid walks the buffer in strides of the whole grid, four strides
// per iteration; each workgroup writes the float64 sum of its loads.  The
// compiler issues this loop's loads two at a time, which reads at 7.10 TB/s
// on an idle MI355X; the same loop written with its four loads issued at
// once (then four adds) read at 6.76-6.79 TB/s.
__global__ __launch_bounds__(kThreads) void read_stream_kernel(
    const floatx4 *__restrict__ x, int64_t n4, double *__restrict__ sink)
{
    __shared__ double red[kThreads / kWave];
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    floatx4 acc[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
        acc[u] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    for (; i + 3 * stride < n4; i += 4 * stride) {
        floatx4 a[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            a[u] = __builtin_nontemporal_load(x + i + u * stride);
#pragma unroll
        for (int u = 0; u < 4; ++u)
            acc[u] += a[u];
    }
    for (; i < n4; i += stride)
        acc[0] += x[i];
    const floatx4 t = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    const double s = block_sum<kThreads>((double)t.x + t.y + t.z + t.w, red);
    if (threadIdx.x == 0)
        sink[blockIdx.x] = s;
}

} // namespace

hipError_t launch_read_stream(const float *x, int64_t n, double *sink, hipStream_t s)
{
    hipLaunchKernelGGL(read_stream_kernel, dim3(kReadStreamBlocks), dim3(kThreads), 0, s,
                       reinterpret_cast<const floatx4 *>(x), n >> 2, sink);
    return hipGetLastError();
}

} // namespace gpic
