// Column-blocked CSR product y = W v for gfx950 (the Multiply step of
// Algorithm 2's loop over a sparse W).
//
// A row-wise CSR product gathers v[col] at random when the node numbering
// has no locality; once the float64 vector is larger than an XCD's 4 MB
// L2, each 8-byte gather brings in a whole cache line from HBM or the
// Infinity Cache.  Here the power iteration first copies W, once, into
// column blocks of 2^18 columns (2 MB of v each): block b holds, for every
// row, the row's entries with column in [b 2^18, (b+1) 2^18), in CSR form.
// One launch then walks (block, row tile) pairs block-major, so the
// workgroups in flight on every XCD gather from one 2 MB slice of v, and
// writes per-block row sums; a second launch adds them in block order.
// When rows hold few entries per block (one lane per row would do), the
// tile's entries are gathered by all lanes in storage order and staged in
// LDS before a thread per row adds them (spmv_blocked_staged_kernel).
//
// The copy needs every row's columns in ascending order (checked on the
// device), at most 32 blocks (n <= 2^23) and fewer than 2^30 entries in
// each block (their positions are int32), and it is made only when at
// least a quarter of the entries lie more than 2^17 columns from the
// diagonal (a numbering with locality already suits the row-wise kernel,
// which is used otherwise).  Results differ from the row-wise kernel only in the order of
// the float64 sums (deterministic either way).
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kColShift = 18;            // 2^18 columns per block
constexpr int64_t kMaxBlocks = 32;
constexpr int kLanes = 16;               // lanes per row in the copy
constexpr int kUnroll = 4;               // gathers in flight per lane
constexpr int kScanTile = 4096;          // elements per scan tile (16 per thread)
constexpr int64_t kFar = (int64_t)1 << 17;   // "far" from the diagonal
// entries per block below which the block's int32 positions, and the
// products' position arithmetic past them, stay in range
constexpr int64_t kMaxBlockEntries = (int64_t)1 << 30;

int64_t al(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Whether the copy is worth making, before any per-block work: the order
// check (flags[0]: a row's columns not ascending) and the number of
// entries more than 2^17 columns from the diagonal (far[0], an integer
// sum: a row-wise product is cache friendly when few entries are far).
// kLanes lanes per row read its columns coalesced; grid-stride over rows,
// one count per workgroup into part[], added up by far_total_kernel (no
// same-address atomics: they serialise).
constexpr int kScanBlocks = 8192;
__global__ __launch_bounds__(kThreads) void far_scan_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, int64_t n,
    int *__restrict__ flags, unsigned long long *__restrict__ part)
{
    __shared__ unsigned long long red[kThreads / kWave];
    const int sl = threadIdx.x % kLanes;
    constexpr int rows_per_block = kThreads / kLanes;
    unsigned long long nfar = 0;
    bool unsorted = false;
    for (int64_t i = (int64_t)blockIdx.x * rows_per_block + threadIdx.x / kLanes; i < n;
         i += (int64_t)gridDim.x * rows_per_block) {
        const int64_t b = row_ptr[i], e = row_ptr[i + 1];
        for (int64_t p = b + sl; p < e; p += kLanes) {
            const int64_t c = col[p];
            nfar += (c - i > kFar || i - c > kFar) ? 1u : 0u;
            unsorted = unsorted || (p > b && col[p - 1] > c);
        }
    }
    if (unsorted)
        flags[0] = 1;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        nfar += __shfl_xor(nfar, o, kWave);
    if ((threadIdx.x % kWave) == 0)
        red[threadIdx.x / kWave] = nfar;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long t = 0;
        for (int w = 0; w < kThreads / kWave; ++w)
            t += red[w];
        part[blockIdx.x] = t;
    }
}

// far[0] = the sum of the m workgroup counts (one workgroup).
__global__ __launch_bounds__(kThreads) void far_total_kernel(
    const unsigned long long *__restrict__ part, int m, unsigned long long *__restrict__ far)
{
    __shared__ unsigned long long red[kThreads / kWave];
    unsigned long long t = 0;
    for (int b = threadIdx.x; b < m; b += kThreads)
        t += part[b];
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        t += __shfl_xor(t, o, kWave);
    if ((threadIdx.x % kWave) == 0)
        red[threadIdx.x / kWave] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long u = 0;
        for (int w = 0; w < kThreads / kWave; ++w)
            u += red[w];
        far[0] = u;
    }
}

// First entry of column block b in row [s0, e) (rows ascending): the
// first q with col[q] >= b 2^18, e for b = nb.
__device__ __forceinline__ int64_t block_start(const int32_t *__restrict__ col, int64_t s0,
                                               int64_t e, int b, int nb)
{
    if (b >= nb)
        return e;
    const int32_t lim = (int32_t)((int64_t)b << kColShift);
    int64_t lo = s0, hi = e;
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (col[mid] < lim)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

// kLanes lanes per row: the row's block starts (a binary search each,
// b = lane, lane + kLanes, ...) into LDS, bnd[g][b] for b = 0 .. nb.
constexpr int kRowsPerBlock = kThreads / kLanes;
__device__ __forceinline__ void row_block_starts(const int32_t *__restrict__ col, int64_t s0,
                                                 int64_t e, bool live, int nb, int sl,
                                                 int64_t *bnd)
{
    for (int b = sl; b <= nb; b += kLanes)
        bnd[b] = live ? block_start(col, s0, e, b, nb) : 0;
}

// Per row: entries per column block (counts[b * n + i]) once the copy is
// to be made (rows ascending), from the row's block starts; flags[0] when a
// row segment alone reaches the block limit (repeated columns).
__global__ __launch_bounds__(kThreads) void block_count_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col, int64_t n,
    int nb, int32_t *__restrict__ counts, int *__restrict__ flags)
{
    __shared__ int64_t bnd[kRowsPerBlock][kMaxBlocks + 1];
    const int g = threadIdx.x / kLanes, sl = threadIdx.x % kLanes;
    const int64_t i = (int64_t)blockIdx.x * kRowsPerBlock + g;
    const bool live = i < n;
    const int64_t s0 = live ? row_ptr[i] : 0, e = live ? row_ptr[i + 1] : 0;
    row_block_starts(col, s0, e, live, nb, sl, bnd[g]);
    __syncthreads();
    if (!live)
        return;
    bool huge = false;
    for (int b = sl; b < nb; b += kLanes) {
        const int64_t c = bnd[g][b + 1] - bnd[g][b];
        huge = huge || c >= kMaxBlockEntries;     // repeated columns
        counts[(int64_t)b * n + i] = (int32_t)(c < kMaxBlockEntries ? c : 0);
    }
    if (huge)
        flags[0] = 1;
}

// Exclusive scan of counts (block-major) into int64 offsets: tile sums,
// a one-workgroup scan of the tile sums, then each tile rescanned.
__global__ __launch_bounds__(kThreads) void scan_tile_sums_kernel(
    const int32_t *__restrict__ counts, int64_t m, int64_t *__restrict__ tsum)
{
    __shared__ int64_t red[kThreads / kWave];
    const int64_t t0 = (int64_t)blockIdx.x * kScanTile;
    int64_t s = 0;
    for (int k = threadIdx.x; k < kScanTile; k += kThreads) {
        const int64_t x = t0 + k;
        if (x < m)
            s += counts[x];
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        s += __shfl_xor(s, o, kWave);
    if ((threadIdx.x % kWave) == 0)
        red[threadIdx.x / kWave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < kThreads / kWave; ++w)
            t += red[w];
        tsum[blockIdx.x] = t;
    }
}

__global__ __launch_bounds__(1024) void scan_tile_offsets_kernel(int64_t *__restrict__ tsum,
                                                                 int64_t ntiles)
{
    // one workgroup: exclusive scan in place, in chunks of 1024
    __shared__ int64_t buf[1024];
    int64_t carry = 0;
    for (int64_t c0 = 0; c0 < ntiles; c0 += 1024) {
        const int64_t x = c0 + threadIdx.x;
        const int64_t v = (x < ntiles) ? tsum[x] : 0;
        buf[threadIdx.x] = v;
        __syncthreads();
        for (int o = 1; o < 1024; o <<= 1) {
            const int64_t add = (threadIdx.x >= (unsigned)o) ? buf[threadIdx.x - o] : 0;
            __syncthreads();
            buf[threadIdx.x] += add;
            __syncthreads();
        }
        if (x < ntiles)
            tsum[x] = carry + buf[threadIdx.x] - v;
        const int64_t total = buf[1023];
        __syncthreads();
        carry += total;
    }
}

__global__ __launch_bounds__(kThreads) void scan_apply_kernel(
    const int32_t *__restrict__ counts, int64_t m, const int64_t *__restrict__ toff,
    int64_t *__restrict__ offs)
{
    // the tile goes through LDS both ways, so that the loads of counts and
    // the stores of offsets are coalesced; thread t scans its kItems
    // consecutive counts (rows padded by one slot against bank conflicts)
    constexpr int per = kScanTile / kThreads;
    constexpr int pitch = per + 1;
    __shared__ int32_t cin[kThreads * pitch];
    __shared__ int64_t out[kThreads * pitch];
    __shared__ int64_t part[kThreads];
    const int64_t b0 = (int64_t)blockIdx.x * kScanTile;
    for (int e = threadIdx.x; e < kScanTile; e += kThreads)
        cin[(e / per) * pitch + e % per] = (b0 + e < m) ? counts[b0 + e] : 0;
    __syncthreads();
    int64_t s = 0;
    for (int k = 0; k < per; ++k)
        s += cin[threadIdx.x * pitch + k];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
        const int64_t add = (threadIdx.x >= (unsigned)o) ? part[threadIdx.x - o] : 0;
        __syncthreads();
        part[threadIdx.x] += add;
        __syncthreads();
    }
    int64_t run = toff[blockIdx.x] + part[threadIdx.x] - s;
    for (int k = 0; k < per; ++k) {
        out[threadIdx.x * pitch + k] = run;
        run += cin[threadIdx.x * pitch + k];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kScanTile; e += kThreads)
        if (b0 + e < m)
            offs[b0 + e] = out[(e / per) * pitch + e % per];
}

// Scatter every row's entries into its blocks: kLanes lanes per row; entry
// p of block b goes to offs[b][i] + (p - the row's first entry of block b).
__global__ __launch_bounds__(kThreads) void block_scatter_kernel(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, int64_t n, int nb, const int64_t *__restrict__ offs,
    int32_t *__restrict__ colb, float *__restrict__ valb)
{
    __shared__ int64_t bnd[kRowsPerBlock][kMaxBlocks + 1];
    const int g = threadIdx.x / kLanes, sl = threadIdx.x % kLanes;
    const int64_t i = (int64_t)blockIdx.x * kRowsPerBlock + g;
    const bool live = i < n;
    const int64_t s0 = live ? row_ptr[i] : 0, e = live ? row_ptr[i + 1] : 0;
    row_block_starts(col, s0, e, live, nb, sl, bnd[g]);
    __syncthreads();
    if (!live)
        return;
    for (int64_t p = s0 + sl; p < e; p += kLanes) {
        const int32_t c = col[p];
        const int b = c >> kColShift;
        const int64_t dst = offs[(int64_t)b * n + i] + (p - bnd[g][b]);
        colb[dst] = c;
        valb[dst] = val[p];
    }
}

// base[b] = first entry of block b; rpb[b][i] = offs[b][i] - base[b],
// rpb[b][n] = entries in block b.  Flags a block of 2^30 entries or more.
__global__ __launch_bounds__(kThreads) void block_rows_kernel(
    const int64_t *__restrict__ offs, int64_t n, int nb, int64_t nnz,
    int64_t *__restrict__ base, int32_t *__restrict__ rpb, int *__restrict__ flags)
{
    const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t b = t / (n + 1);
    const int64_t i = t % (n + 1);
    if (b >= nb)
        return;
    const int64_t b0 = offs[b * n];
    const int64_t b1 = (b + 1 < nb) ? offs[(b + 1) * n] : nnz;
    if (i == 0) {
        base[b] = b0;
        if (b + 1 == nb)
            base[nb] = nnz;
        if (b1 - b0 >= kMaxBlockEntries)
            flags[0] = 1;
    }
    const int64_t o = (i < n) ? offs[b * n + i] : b1;
    rpb[b * (n + 1) + i] = (int32_t)(o - b0);
}

__global__ void clear_flags_kernel(int *flags, unsigned long long *far)
{
    flags[0] = 0;
    far[0] = 0ull;
}

// The product, block-major over (block, row tile): per-block row sums.
// LANES lanes per row (a row holds few entries per block), 256 / LANES
// rows per workgroup; lane l sums entries l, l + LANES, ... of its segment
// in that order with four gathers in flight, then a LANES-lane butterfly.
template <int LANES>
__global__ __launch_bounds__(kThreads) void spmv_blocked_kernel(
    const int64_t *__restrict__ base, const int32_t *__restrict__ rpb,
    const int32_t *__restrict__ colb, const float *__restrict__ valb, int64_t n,
    int64_t tiles, const double *__restrict__ v, double *__restrict__ ypart, StopCtl ctl)
{
    constexpr int R = kThreads / LANES;
    __shared__ int32_t rp[R + 1];
    if (blockIdx.x == 0 && threadIdx.x == 0)
        *ctl.cur_stat = 0.0;
    if (stop_reached(ctl))
        return;
    const int64_t b = blockIdx.x / tiles;
    const int64_t row0 = (blockIdx.x % tiles) * R;
    const int32_t *rb = rpb + b * (n + 1);
    for (int t = threadIdx.x; t <= R; t += kThreads)
        rp[t] = rb[row0 + t < n ? row0 + t : n];
    __syncthreads();
    const int32_t *cb = colb + base[b];
    const float *vb = valb + base[b];
    const int sl = threadIdx.x % LANES;
    const int li = threadIdx.x / LANES;
    const int64_t i = row0 + li;
    double s = 0.0;
    if (i < n) {
        const int32_t e = rp[li + 1];
        for (int32_t p0 = rp[li] + sl; p0 < e; p0 += LANES * kUnroll) {
            int32_t c[kUnroll];
            float w[kUnroll];
            double x[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int32_t p = p0 + u * LANES;
                c[u] = p < e ? cb[p] : -1;
                w[u] = p < e ? vb[p] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                x[u] = c[u] >= 0 ? v[c[u]] : 0.0;
#pragma unroll
            for (int u = 0; u < kUnroll; ++u)
                if (c[u] >= 0)
                    s = fma((double)w[u], x[u], s);
        }
    }
    if (LANES > 1)
        s = group_sum<LANES>(s);
    if (i < n && sl == 0)
        ypart[b * n + i] = s;
}

// The product for one lane per row, staged: a row holds few entries per
// block (about 5.6 for a 32-NN graph), so a lane per row leaves most lanes
// of a gather instruction idle while the wave finishes its longest row.
// Here the 256 threads first walk the tile's entries in storage order
// (every lane busy: coalesced column and value loads, then the gathers,
// kUnroll in flight per thread) and stage w and v[col] in LDS; after a
// barrier a thread per row adds its entries in entry order with the same
// multiply-adds as the lane-per-row kernel, so the sums are bitwise the
// same.  Tiles with more entries than the stage go round by round.
constexpr int kStage = 2048;             // staged entries per round

__global__ __launch_bounds__(kThreads) void spmv_blocked_staged_kernel(
    const int64_t *__restrict__ base, const int32_t *__restrict__ rpb,
    const int32_t *__restrict__ colb, const float *__restrict__ valb, int64_t n,
    int64_t tiles, const double *__restrict__ v, double *__restrict__ ypart, StopCtl ctl)
{
    constexpr int R = kThreads;                  // rows per tile
    __shared__ int32_t rp[R + 1];
    __shared__ double xs[kStage];
    __shared__ float ws[kStage];
    if (blockIdx.x == 0 && threadIdx.x == 0)
        *ctl.cur_stat = 0.0;
    if (stop_reached(ctl))
        return;
    const int64_t b = blockIdx.x / tiles;
    const int64_t row0 = (blockIdx.x % tiles) * R;
    const int32_t *rb = rpb + b * (n + 1);
    for (int t = threadIdx.x; t <= R; t += kThreads)
        rp[t] = rb[row0 + t < n ? row0 + t : n];
    __syncthreads();
    const int32_t *cb = colb + base[b];
    const float *vb = valb + base[b];
    const int32_t e0 = rp[0], e1 = rp[R];
    const int li = threadIdx.x;
    const int64_t i = row0 + li;
    const int32_t rs = rp[li], re = rp[li + 1];  // this thread's row (empty past n)
    double s = 0.0;
    for (int32_t r0 = e0; r0 < e1; r0 += kStage) {
        const int32_t r1 = (r0 + kStage < e1) ? r0 + kStage : e1;
        for (int32_t p0 = r0 + threadIdx.x; p0 < r1; p0 += kThreads * kUnroll) {
            int32_t c[kUnroll];
            float w[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int32_t p = p0 + u * kThreads;
                c[u] = p < r1 ? cb[p] : -1;
                w[u] = p < r1 ? vb[p] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                if (c[u] >= 0) {
                    const int32_t q = p0 + u * kThreads - r0;
                    xs[q] = v[c[u]];
                    ws[q] = w[u];
                }
            }
        }
        __syncthreads();
        const int32_t a = (rs > r0) ? rs : r0;
        const int32_t z = (re < r1) ? re : r1;
        for (int32_t p = a; p < z; ++p)
            s = fma((double)ws[p - r0], xs[p - r0], s);
        __syncthreads();                         // before the next round's stage
    }
    if (i < n)
        ypart[b * n + i] = s;
}

// y_i = sum over blocks of the block sums (block order); per-workgroup
// partial sums of |y_i| for the L1 norm.
__global__ __launch_bounds__(kThreads) void spmv_finalize_kernel(
    const double *__restrict__ ypart, int64_t n, int nb, double *__restrict__ y,
    double *__restrict__ partial, StopCtl ctl)
{
    __shared__ double red[kThreads / kWave];
    if (stop_reached(ctl))
        return;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    double yabs = 0.0;
    if (i < n) {
        double s = 0.0;
        for (int b = 0; b < nb; ++b)
            s += ypart[(int64_t)b * n + i];
        y[i] = s;
        yabs = fabs(s);
    }
    const double t = block_sum<kThreads>(yabs, red);
    if (threadIdx.x == 0)
        partial[blockIdx.x] = t;
}

int64_t col_blocks(int64_t n) { return (n + ((int64_t)1 << kColShift) - 1) >> kColShift; }

} // namespace

bool csr_blocked_applies(int64_t n)
{
    const int64_t nb = col_blocks(n);
    return nb >= 2 && nb <= kMaxBlocks;
}

int64_t csr_blocked_partials(int64_t n) { return (n + kThreads - 1) / kThreads; }

// [flags 256][base (nb+1) int64][rpb nb (n+1) int32][colb nnz int32]
// [valb nnz float][ypart nb n float64 (scan offsets during the copy)]
// [counts nb n int32][tile sums]
size_t csr_blocked_ws(int64_t n, int64_t nnz)
{
    if (!csr_blocked_applies(n))
        return 0;
    const int64_t nb = col_blocks(n);
    const int64_t m = nb * n;
    const int64_t ntiles = (m + kScanTile - 1) / kScanTile;
    return (size_t)(256 + al((nb + 1) * 8) + al(nb * (n + 1) * 4) + 2 * al(nnz * 4) +
                    al(m * 8) + al(m * 4) + al(ntiles * 8));
}

hipError_t build_csr_blocked(const int64_t *row_ptr, const int32_t *col,
                             const float *val, int64_t n, int64_t nnz, void *ws,
                             CsrBlocked *out, hipStream_t s, int *usable_host)
{
    const int64_t nb = col_blocks(n);
    const int64_t m = nb * n;
    const int64_t ntiles = (m + kScanTile - 1) / kScanTile;
    char *w = static_cast<char *>(ws);
    int *flags = reinterpret_cast<int *>(w);
    size_t o = 256;
    auto take = [&](int64_t bytes) {
        char *p = w + o;
        o += (size_t)al(bytes);
        return p;
    };
    CsrBlocked B;
    B.n = n;
    B.nb = nb;
    // lanes per row: about 4 entries per lane of a row's average segment
    const int64_t avg = nnz / (nb * n);
    B.lanes = avg >= 64 ? 16 : avg >= 32 ? 8 : avg >= 16 ? 4 : avg >= 8 ? 2 : 1;
    B.base = reinterpret_cast<int64_t *>(take((nb + 1) * 8));
    B.rpb = reinterpret_cast<int32_t *>(take(nb * (n + 1) * 4));
    B.colb = reinterpret_cast<int32_t *>(take(nnz * 4));
    B.valb = reinterpret_cast<float *>(take(nnz * 4));
    B.ypart = reinterpret_cast<double *>(take(m * 8));
    int32_t *counts = reinterpret_cast<int32_t *>(take(m * 4));
    int64_t *tsum = reinterpret_cast<int64_t *>(take(ntiles * 8));
    int64_t *offs = reinterpret_cast<int64_t *>(B.ypart);      // reused below

    unsigned long long *far = reinterpret_cast<unsigned long long *>(w + 64);
    const int64_t scan_rows = kThreads / kLanes;
    const unsigned scan_grid =
        (unsigned)std::min<int64_t>((n + scan_rows - 1) / scan_rows, kScanBlocks);
    // the workgroup counts go in the counts buffer, unused until the copy is made
    unsigned long long *far_part = reinterpret_cast<unsigned long long *>(counts);
    hipLaunchKernelGGL(clear_flags_kernel, dim3(1), dim3(1), 0, s, flags, far);
    hipLaunchKernelGGL(far_scan_kernel, dim3(scan_grid), dim3(kThreads), 0, s, row_ptr, col,
                       n, flags, far_part);
    hipLaunchKernelGGL(far_total_kernel, dim3(1), dim3(kThreads), 0, s,
                       (const unsigned long long *)far_part, (int)scan_grid, far);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    struct {
        int flag;
        int pad;
        unsigned long long far;
    } h{};
    if ((e = hipMemcpyAsync(&h.flag, flags, sizeof(int), hipMemcpyDeviceToHost, s)) !=
            hipSuccess ||
        (e = hipMemcpyAsync(&h.far, far, 8, hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return e;
    // unsorted rows, or a numbering that already keeps most gathers near
    // the diagonal (fewer than a quarter of the entries far): row-wise
    *usable_host = 0;
    if (h.flag || 4 * h.far < (unsigned long long)nnz)
        return hipSuccess;
    const unsigned group_grid = (unsigned)((n + kRowsPerBlock - 1) / kRowsPerBlock);
    hipLaunchKernelGGL(block_count_kernel, dim3(group_grid), dim3(kThreads), 0, s, row_ptr,
                       col, n, (int)nb, counts, flags);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    hipLaunchKernelGGL(scan_tile_sums_kernel, dim3((unsigned)ntiles), dim3(kThreads), 0, s,
                       counts, m, tsum);
    hipLaunchKernelGGL(scan_tile_offsets_kernel, dim3(1), dim3(1024), 0, s, tsum, ntiles);
    hipLaunchKernelGGL(scan_apply_kernel, dim3((unsigned)ntiles), dim3(kThreads), 0, s,
                       counts, m, tsum, offs);
    hipLaunchKernelGGL(block_rows_kernel,
                       dim3((unsigned)((nb * (n + 1) + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, offs, n, (int)nb, nnz, B.base, B.rpb, flags);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    int bad = 0;
    if ((e = hipMemcpyAsync(&bad, flags, sizeof(int), hipMemcpyDeviceToHost, s)) !=
            hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return e;
    if (bad)                             // a block of 2^30 entries or more
        return hipSuccess;
    *usable_host = 1;
    // rows are sorted: every entry lands in its block's range
    hipLaunchKernelGGL(block_scatter_kernel, dim3(group_grid), dim3(kThreads), 0, s, row_ptr,
                       col, val, n, (int)nb, offs, B.colb, B.valb);
    *out = B;
    return hipGetLastError();
}

hipError_t launch_spmv_blocked(const CsrBlocked &B, const double *v, double *y,
                               double *partial, StopCtl ctl, hipStream_t s)
{
#define GPIC_BLOCKED(L)                                                         \
    {                                                                          \
        const int64_t tiles = (B.n + kThreads / L - 1) / (kThreads / L);      \
        hipLaunchKernelGGL(spmv_blocked_kernel<L>, dim3((unsigned)(B.nb * tiles)),  \
                           dim3(kThreads), 0, s, B.base, B.rpb, B.colb, B.valb, B.n, \
                           tiles, v, B.ypart, ctl);                            \
    }
    switch (B.lanes) {
    case 1: {
        const int64_t tiles = (B.n + kThreads - 1) / kThreads;
        hipLaunchKernelGGL(spmv_blocked_staged_kernel, dim3((unsigned)(B.nb * tiles)),
                           dim3(kThreads), 0, s, B.base, B.rpb, B.colb, B.valb, B.n, tiles,
                           v, B.ypart, ctl);
        break;
    }
    case 2: GPIC_BLOCKED(2); break;
    case 4: GPIC_BLOCKED(4); break;
    case 8: GPIC_BLOCKED(8); break;
    default: GPIC_BLOCKED(16); break;
    }
#undef GPIC_BLOCKED
    hipLaunchKernelGGL(spmv_finalize_kernel,
                       dim3((unsigned)csr_blocked_partials(B.n)), dim3(kThreads), 0, s,
                       B.ypart, B.n, (int)B.nb, y, partial, ctl);
    return hipGetLastError();
}

} // namespace gpic
