// Stable LSD radix sort of uint64 keys with an optional int32 payload, for
// gfx950: 8-bit digits; per pass a histogram per tile of 4,096 keys, an
// exclusive scan of the digit-major counts (three launches when they are
// many), and a stable scatter that ranks keys inside each wave with ballots
// over the digit bits.  Up to 4,096 keys are sorted instead by one
// workgroup in LDS (a bitonic network over (key, input position), the same
// order).  Shared by the 1-D k-means (sorting v) and the kNN graph builder
// (sorting edges).
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;   // elements per sort / scan tile
constexpr int kRadix = 256;

__host__ __device__ inline int64_t tiles(int64_t n) { return (n + kTile - 1) / kTile; }

// hist[digit * ntiles + tile]
__global__ __launch_bounds__(kThreads) void radix_hist_kernel(
    const uint64_t *__restrict__ key, int64_t n, int shift,
    uint32_t *__restrict__ hist)
{
    __shared__ uint32_t h[kRadix];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kTile;
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = base + it * kThreads + threadIdx.x;
        if (i < n)
            atomicAdd(&h[(key[i] >> shift) & 0xff], 1u);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * gridDim.x + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan of m uint32 counts, in place, in three launches: each
// workgroup sums kTile counts, one workgroup scans those sums, and each
// workgroup rescans its counts from its offset.
__global__ __launch_bounds__(kThreads) void scan_sums_kernel(const uint32_t *__restrict__ a,
                                                             int64_t m,
                                                             uint32_t *__restrict__ bsum)
{
    __shared__ uint32_t red[kThreads / kWave];
    const int64_t b0 = (int64_t)blockIdx.x * kTile;
    uint32_t t = 0;
    for (int k = threadIdx.x; k < kTile; k += kThreads)
        if (b0 + k < m)
            t += a[b0 + k];
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        t += __shfl_xor(t, o, kWave);
    if ((threadIdx.x % kWave) == 0)
        red[threadIdx.x / kWave] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t u = 0;
        for (int w = 0; w < kThreads / kWave; ++w)
            u += red[w];
        bsum[blockIdx.x] = u;
    }
}

// One workgroup of 1024: exclusive scan of m counts (the block sums, or a
// short count array directly), in place.
__global__ __launch_bounds__(1024) void scan_bsums_kernel(uint32_t *__restrict__ a,
                                                          int64_t m)
{
    __shared__ uint32_t s[1024];
    const int64_t per = (m + 1023) / 1024;
    const int64_t b = threadIdx.x * per;
    const int64_t e = (b + per < m) ? b + per : m;
    uint32_t tot = 0;
    for (int64_t i = b; i < e; ++i)
        tot += a[i];
    s[threadIdx.x] = tot;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
        const uint32_t x = (threadIdx.x >= (unsigned)o) ? s[threadIdx.x - o] : 0u;
        __syncthreads();
        s[threadIdx.x] += x;
        __syncthreads();
    }
    uint32_t run = s[threadIdx.x] - tot;
    for (int64_t i = b; i < e; ++i) {
        const uint32_t x = a[i];
        a[i] = run;
        run += x;
    }
}

// Each thread owns kItems consecutive counts of its workgroup's tile.
__global__ __launch_bounds__(kThreads) void scan_apply_kernel(uint32_t *__restrict__ a,
                                                              int64_t m,
                                                              const uint32_t *__restrict__ boff)
{
    __shared__ uint32_t part[kThreads];
    const int64_t x0 = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    uint32_t t = 0;
    for (int k = 0; k < kItems; ++k)
        if (x0 + k < m)
            t += a[x0 + k];
    part[threadIdx.x] = t;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
        const uint32_t x = (threadIdx.x >= (unsigned)o) ? part[threadIdx.x - o] : 0u;
        __syncthreads();
        part[threadIdx.x] += x;
        __syncthreads();
    }
    uint32_t run = boff[blockIdx.x] + part[threadIdx.x] - t;
    for (int k = 0; k < kItems; ++k)
        if (x0 + k < m) {
            const uint32_t x = a[x0 + k];
            a[x0 + k] = run;
            run += x;
        }
}

// Stable scatter of one tile.  Element order inside a tile is
// (item, thread); for every item the 256 elements are ranked inside their
// wave with ballots over the 8 digit bits, and across waves with per-wave
// digit counts in LDS.
__global__ __launch_bounds__(kThreads) void radix_scatter_kernel(
    const uint64_t *__restrict__ kin, const int32_t *__restrict__ iin,
    uint64_t *__restrict__ kout, int32_t *__restrict__ iout, int64_t n,
    int shift, const uint32_t *__restrict__ offs)
{
    constexpr int nw = kThreads / kWave;
    __shared__ uint32_t base[kRadix];
    __shared__ uint32_t wc[nw][kRadix];
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    base[threadIdx.x] = offs[(int64_t)threadIdx.x * gridDim.x + blockIdx.x];
    for (int w = 0; w < nw; ++w)
        wc[w][threadIdx.x] = 0;
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t tb = (int64_t)blockIdx.x * kTile;
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = tb + it * kThreads + threadIdx.x;
        const bool live = i < n;
        uint64_t k = 0;
        int32_t ix = 0;
        int dg = 0;
        if (live) {
            k = kin[i];
            ix = iin ? iin[i] : 0;
            dg = (int)((k >> shift) & 0xff);
        }
        uint64_t peers = __ballot(live);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
            const uint64_t bb = __ballot((dg >> bit) & 1);
            peers &= ((dg >> bit) & 1) ? bb : ~bb;
        }
        const uint32_t rank = (uint32_t)__popcll(peers & lt);
        const uint32_t cnt = (uint32_t)__popcll(peers);
        const bool leader = live && (peers & lt) == 0;
        if (leader)
            wc[wave][dg] = cnt;
        __syncthreads();
        if (live) {
            uint32_t pos = base[dg] + rank;
            for (int w = 0; w < wave; ++w)
                pos += wc[w][dg];
            kout[pos] = k;
            if (iout)
                iout[pos] = ix;
        }
        __syncthreads();
        uint32_t add = 0;
        for (int w = 0; w < nw; ++w) {
            add += wc[w][threadIdx.x];
            wc[w][threadIdx.x] = 0;
        }
        base[threadIdx.x] += add;
        __syncthreads();
    }
}

// Up to kSmallSort keys: one workgroup sorts (low `bits` of the key, input
// position) pairs with a bitonic network in LDS, so equal keys keep their
// input order exactly as the radix passes do; one launch instead of three
// per 8-bit pass.  P is n rounded up to a power of two; the padding sorts
// last.
constexpr int kSmallSort = 4096;
constexpr int kSmallThreads = 1024;

__global__ __launch_bounds__(kSmallThreads) void small_sort_kernel(
    const uint64_t *__restrict__ key, const int32_t *__restrict__ idx,
    uint64_t *__restrict__ okey, int32_t *__restrict__ oidx, int n, int P, uint64_t mask)
{
    __shared__ uint64_t k[kSmallSort];
    __shared__ int32_t pos[kSmallSort];
    for (int i = threadIdx.x; i < P; i += kSmallThreads) {
        k[i] = (i < n) ? (key[i] & mask) : ~0ull;
        pos[i] = i;
    }
    __syncthreads();
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = threadIdx.x; t < P / 2; t += kSmallThreads) {
                const int lo = 2 * t - (t & (stride - 1));
                const int hi = lo + stride;
                const bool up = (lo & size) == 0;
                const uint64_t a = k[lo], b = k[hi];
                const int32_t pa = pos[lo], pb = pos[hi];
                const bool gt = (a > b) || (a == b && pa > pb);
                if (gt == up) {
                    k[lo] = b;
                    k[hi] = a;
                    pos[lo] = pb;
                    pos[hi] = pa;
                }
            }
            __syncthreads();
        }
    }
    for (int i = threadIdx.x; i < n; i += kSmallThreads) {
        okey[i] = key[pos[i]];
        if (oidx != nullptr && idx != nullptr)
            oidx[i] = idx[pos[i]];
    }
}

} // namespace

size_t radix_hist_bytes(int64_t n) { return (size_t)kRadix * tiles(n) * 4; }
size_t scan_sums_bytes(int64_t m) { return (size_t)tiles(m) * 4 + 4; }

hipError_t exclusive_scan_u32(uint32_t *a, int64_t m, uint32_t *sums, hipStream_t s)
{
    if (m <= 16 * kTile) {
        hipLaunchKernelGGL(scan_bsums_kernel, dim3(1), dim3(1024), 0, s, a, m);
    } else {
        const unsigned hb = (unsigned)tiles(m);
        hipLaunchKernelGGL(scan_sums_kernel, dim3(hb), dim3(kThreads), 0, s, a, m, sums);
        hipLaunchKernelGGL(scan_bsums_kernel, dim3(1), dim3(1024), 0, s, sums, (int64_t)hb);
        hipLaunchKernelGGL(scan_apply_kernel, dim3(hb), dim3(kThreads), 0, s, a, m, sums);
    }
    return hipGetLastError();
}
size_t radix_hsum_bytes(int64_t n) { return (size_t)tiles(kRadix * tiles(n)) * 4 + 4; }

hipError_t radix_sort_u64(uint64_t *&keyA, int32_t *&idxA, uint64_t *&keyB, int32_t *&idxB,
                          int64_t n, int bits, uint32_t *hist, uint32_t *hsum,
                          hipStream_t s)
{
    if (n <= 0)
        return hipSuccess;
    if (n <= kSmallSort) {
        int P = 1;
        while (P < n)
            P <<= 1;
        const uint64_t mask = (bits >= 64) ? ~0ull : ((1ull << bits) - 1);
        hipLaunchKernelGGL(small_sort_kernel, dim3(1), dim3(kSmallThreads), 0, s, keyA,
                           idxA, keyB, idxB, (int)n, P, mask);
        uint64_t *tk = keyA; keyA = keyB; keyB = tk;
        int32_t *ti = idxA; idxA = idxB; idxB = ti;
        return hipGetLastError();
    }
    const int64_t nt = tiles(n);
    for (int shift = 0; shift < bits; shift += 8) {
        hipLaunchKernelGGL(radix_hist_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s,
                           keyA, n, shift, hist);
        exclusive_scan_u32(hist, (int64_t)kRadix * nt, hsum, s);
        hipLaunchKernelGGL(radix_scatter_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s,
                           keyA, idxA, keyB, idxB, n, shift, hist);
        uint64_t *tk = keyA; keyA = keyB; keyB = tk;
        int32_t *ti = idxA; idxA = idxB; idxB = ti;
    }
    return hipGetLastError();
}

} // namespace gpic
