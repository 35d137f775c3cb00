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

// A fixed grid walks the buffer in strides of the whole grid, four loads in
// flight per thread; each workgroup writes the float64 sum of its loads.
__global__ __launch_bounds__(kThreads) void read_stream_kernel(
    const floatx4 *__restrict__ x, int64_t n4, double *__restrict__ sink)
{
    __shared__ double red[kThreads / kWave];
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    floatx4 s0 = {0.0f, 0.0f, 0.0f, 0.0f}, s1 = s0, s2 = s0, s3 = s0;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        const floatx4 a = __builtin_nontemporal_load(x + i);
        const floatx4 b = __builtin_nontemporal_load(x + i + stride);
        const floatx4 c = __builtin_nontemporal_load(x + i + 2 * stride);
        const floatx4 d = __builtin_nontemporal_load(x + i + 3 * stride);
        s0 += a;
        s1 += b;
        s2 += c;
        s3 += d;
    }
    for (; i < n4; i += stride)
        s0 += __builtin_nontemporal_load(x + i);
    const floatx4 t = (s0 + s1) + (s2 + s3);
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
