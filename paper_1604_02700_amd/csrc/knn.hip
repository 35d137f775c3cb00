// Exact k-nearest-neighbour input graph for the sparse path, on gfx950.
//
// N(i) = the k points j != i with the smallest (||x_i - x_j||^2, j); edge
// {i, j} when j is in N(i) or i in N(j); weight exp(-||x_i - x_j||^2 /
// (2 sigma^2)) in float64, rounded once to float32; rows sorted by column.
// This is the graph the CSR power iteration takes as its affinity (the
// paper's method needs an affinity matrix; a kNN graph is its sparse form).
//
// Brute force in four steps, exact in the end:
//   1. bound: the points are put in Morton order of their quantised centred
//      coordinates; for every row, the k-th smallest float32 squared
//      distance to the points within 256 positions of it in that order and
//      to a fixed sample of 65,536 positions, which bounds the true k-th
//      neighbour distance from above;
//   2. collect: squared distances on the fp32 matrix cores (Gram form over
//      the centred points augmented as [x_j, |x_j|^2, 1] .
//      [-2 x_i, 1, |x_i|^2]), appending every j that passes the row's bound
//      widened by the float32 error bounds of both forms to a per-row
//      candidate list.  In Morton order a tile of 64 consecutive points is
//      spatially compact; a pair of tiles whose bounding boxes are farther
//      apart than every bound of the row tile is skipped whole (no pair in
//      it can be a neighbour: its true distance exceeds the row's bound,
//      which is at least the true k-th neighbour distance);
//   3. select: a wave per row recomputes the candidates' squared distances
//      in float64 and keeps the k smallest (ties to the smaller index); a
//      row whose list overflowed gets the k-th distance among the kept
//      candidates as its new bound and is collected again;
//   4. symmetrise: both directions of every kept pair as 64-bit keys
//      (row, column), radix sorted, duplicates dropped, CSR built, weights
//      from float64 distances.
// Supports d <= 16 and k <= 64.
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kCap = 2048;                // candidate slots per row
constexpr int kPerLane = kCap / kWave;    // candidates per lane in the selection
constexpr int kRowsPerGroup = 64;         // collect: 4 waves x 16 rows
constexpr int kTileCols = 64;
constexpr float kEps32 = 5.9604645e-08f;  // 2^-24
constexpr int kMeanBlocks = 256;

typedef float floatx4 __attribute__((ext_vector_type(4)));

int64_t al(int64_t x) { return (x + 255) & ~(int64_t)255; }
int64_t padded_points(int64_t n) { return (n + kTileCols - 1) / kTileCols * kTileCols; }
// augmented dimension / 4, rounded up to an instantiated engine (3 or 5)
int ks_for(int d) { return (d + 2 + 3) / 4 <= 3 ? 3 : 5; }

// float64 squared distance summed over coordinates in order, without
// fused multiply-adds (the same value a plain C loop gives)
__device__ __forceinline__ double sq_dist64(const float *__restrict__ X, int d, int64_t i,
                                            int64_t j)
{
    double s = 0.0;
    for (int c = 0; c < d; ++c) {
        const double df = __dsub_rn((double)X[i * d + c], (double)X[j * d + c]);
        s = __dadd_rn(s, __dmul_rn(df, df));
    }
    return s;
}

// ------------------------------------------------------------ 1. bound

// Thread per Morton position p, row i = perm[p]: the KT smallest float32
// squared distances from x_i to the points at positions p - kWindow ..
// p + kWindow and at the sample positions outside that window (every
// n / kSample-th position, all of them when n is smaller; each point is
// counted once), then tau_i = the k-th of them.  The k-th distance to any k
// other points bounds the true k-th neighbour distance from above: Morton
// neighbours are mostly near (a tight bound), the sample caps the bound
// where the Morton order jumps.  Both sets go through LDS 256 points at a
// time.
constexpr int kWindow = 256;           // Morton positions on each side
constexpr int64_t kSample = 65536;     // sample positions

__device__ __forceinline__ int64_t sample_point(int64_t t, int64_t n, int64_t m)
{
    return (m == n) ? t : (t * n) / m;
}

template <int D, int KT>
__global__ __launch_bounds__(kThreads) void knn_bound_kernel(
    const float *__restrict__ X, const int32_t *__restrict__ perm, int64_t n, int k,
    float *__restrict__ tau)
{
    __shared__ float tile[kThreads * D];
    __shared__ int64_t tid_[kThreads];
    const int64_t p0 = (int64_t)blockIdx.x * kThreads;
    const int64_t p = p0 + threadIdx.x;
    const int64_t pc = p < n ? p : n - 1;
    const int64_t i = perm[pc];
    float xi[D];
#pragma unroll
    for (int c = 0; c < D; ++c)
        xi[c] = X[i * D + c];
    float best[KT];
#pragma unroll
    for (int u = 0; u < KT; ++u)
        best[u] = INFINITY;
    auto consider = [&](const float *xj) {
        float s = 0.0f;
#pragma unroll
        for (int c = 0; c < D; ++c) {
            const float df = xi[c] - xj[c];
            s = fmaf(df, df, s);
        }
        if (s < best[KT - 1]) {
#pragma unroll
            for (int u = KT - 1; u > 0; --u) {
                const float lo = best[u - 1];
                best[u] = (s < lo) ? lo : fminf(s, best[u]);
            }
            best[0] = fminf(s, best[0]);
        }
    };
    // the Morton window (positions, skipping p and anything beyond kWindow)
    for (int64_t q0 = p0 - kWindow; q0 < p0 + kThreads + kWindow; q0 += kThreads) {
        __syncthreads();
        const int64_t q = q0 + threadIdx.x;
        const bool ok = q >= 0 && q < n;
        const int64_t pt = ok ? (int64_t)perm[q] : 0;
#pragma unroll
        for (int c = 0; c < D; ++c)
            tile[threadIdx.x * D + c] = ok ? X[pt * D + c] : 0.0f;
        __syncthreads();
        for (int u = 0; u < kThreads; ++u) {
            const int64_t qq = q0 + u;
            if (qq < 0 || qq >= n || qq == pc || qq < pc - kWindow || qq > pc + kWindow)
                continue;
            consider(tile + u * D);
        }
    }
    // the sample positions outside the window (the window already holds
    // the others, and the row itself)
    const int64_t m = n < kSample ? n : kSample;
    for (int64_t t0 = 0; t0 < m; t0 += kThreads) {
        __syncthreads();
        const int64_t t = t0 + threadIdx.x;
        const int64_t q = (t < m) ? sample_point(t, n, m) : -1;
        tid_[threadIdx.x] = q;
        const int64_t pt = (q >= 0) ? (int64_t)perm[q] : 0;
#pragma unroll
        for (int c = 0; c < D; ++c)
            tile[threadIdx.x * D + c] = (q >= 0) ? X[pt * D + c] : 0.0f;
        __syncthreads();
        const int cnt = (m - t0 < kThreads) ? (int)(m - t0) : kThreads;
        for (int u = 0; u < cnt; ++u) {
            const int64_t qq = tid_[u];
            if (qq >= pc - kWindow && qq <= pc + kWindow)
                continue;
            consider(tile + u * D);
        }
    }
    if (p < n) {
        float t = best[0];
#pragma unroll
        for (int u = 1; u < KT; ++u)
            if (u == k - 1)
                t = best[u];
        tau[i] = t;
    }
}

// max_j |x_j|^2 (non-negative floats compare as their bit patterns)
__global__ __launch_bounds__(kThreads) void max_norm_kernel(const float *__restrict__ norm2,
                                                            int64_t n,
                                                            unsigned int *__restrict__ out)
{
    unsigned int m = 0;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads)
        m = max(m, __float_as_uint(norm2[i]));
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        m = max(m, (unsigned int)__shfl_xor((int)m, o, kWave));
    if ((threadIdx.x % kWave) == 0)
        atomicMax(out, m);
}

// Collection threshold: the exact k-th neighbour distance is at most
// tau (1 + 4 (d + 2) eps32) (tau is a float32 difference-form value); a
// Gram-form value over the centred points x' = x - mean (rounded once), a
// float32 sum of KP terms whose magnitudes add up to at most
// 2 (|x'_i|^2 + |x'_j|^2), is below the exact squared distance by at most
// (2 KP + 20) eps32 (|x'_i|^2 + max |x'|^2) with margin (4 of it for the
// rounding of the centred coordinates).  Formed in float64 and rounded up.
// Rows not active get -1 (nothing passes).
__global__ __launch_bounds__(kThreads) void threshold_kernel(
    const float *__restrict__ tau, const double *__restrict__ kth,
    const float *__restrict__ norm2, const unsigned int *__restrict__ maxn, int64_t n,
    int d, int kp, const int *__restrict__ active, float *__restrict__ thr)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n)
        return;
    if (active != nullptr && !active[i]) {
        thr[i] = -1.0f;
        return;
    }
    const double eps = (double)kEps32;
    const double base = (kth != nullptr) ? kth[i] : (double)tau[i];
    const double t = base * (1.0 + 4.0 * (d + 2) * eps) +
                     (2 * kp + 20) * eps * ((double)norm2[i] + (double)__uint_as_float(*maxn));
    float f = (float)t;
    if ((double)f < t)
        f = nextafterf(f, INFINITY);
    thr[i] = f;
}

// ------------------------------------------------------------ 2. collect

// Mean of the points per coordinate (float64): per-workgroup partial sums,
// then one workgroup adds them in order.
__global__ __launch_bounds__(kThreads) void mean_partials_kernel(const float *__restrict__ X,
                                                                 int64_t n, int d,
                                                                 double *__restrict__ part)
{
    __shared__ double red[kThreads / kWave];
    for (int c = 0; c < d; ++c) {
        double s = 0.0;
        for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < n;
             p += (int64_t)gridDim.x * kThreads)
            s += (double)X[p * d + c];
        const double t = block_sum<kThreads>(s, red);
        if (threadIdx.x == 0)
            part[(int64_t)blockIdx.x * d + c] = t;
    }
}

__global__ void mean_finish_kernel(const double *__restrict__ part, int nb, int d, int64_t n,
                                   double *__restrict__ mu)
{
    const int c = threadIdx.x;
    if (c >= d)
        return;
    double s = 0.0;
    for (int b = 0; b < nb; ++b)
        s += part[(int64_t)b * d + c];
    mu[c] = s / (double)n;
}

// Augmented operands of the centred points x' = float32(x - mean):
// column xa[k * np + p] = [x'_p, |x'_p|^2, 1, 0...], row
// xb[p * KP + k] = [-2 x'_p, 1, |x'_p|^2, 0...]; |x'_p|^2 a float64 sum
// rounded once (also written to norm2).  Padding points are zeros.
// With perm, position p holds point perm[p] (norm2 stays indexed by point).
__global__ __launch_bounds__(kThreads) void knn_augment_kernel(
    const float *__restrict__ X, const double *__restrict__ mu, const int32_t *__restrict__ perm,
    int64_t n, int64_t np, int d, int KP, float *__restrict__ xa, float *__restrict__ xb,
    float *__restrict__ norm2)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= np)
        return;
    const int64_t pt = (p < n && perm != nullptr) ? (int64_t)perm[p] : p;
    float xc[16];
    double s = 0.0;
    for (int c = 0; c < 16; ++c) {
        xc[c] = 0.0f;
        if (c < d && p < n) {
            xc[c] = (float)((double)X[pt * d + c] - mu[c]);
            s = fma((double)xc[c], (double)xc[c], s);
        }
    }
    const float nrm = (float)s;
    if (p < n)
        norm2[pt] = nrm;
    for (int k = 0; k < KP; ++k) {
        float a = 0.0f, b = 0.0f;
        if (p < n) {
            if (k < d) {
                a = xc[k];
                b = -2.0f * a;
            } else if (k == d) {
                a = nrm;
                b = 1.0f;
            } else if (k == d + 1) {
                a = 1.0f;
                b = nrm;
            }
        }
        xa[k * np + p] = a;
        xb[p * KP + k] = b;
    }
}

// Morton key of point p: its centred coordinates quantised to b = min(64 / d,
// 32) bits over [-R, R] (R^2 = the largest |x - mean|^2), bits interleaved
// from the most significant down; the payload is the point's index.
__global__ __launch_bounds__(kThreads) void morton_key_kernel(
    const float *__restrict__ X, const double *__restrict__ mu,
    const unsigned int *__restrict__ maxn, int64_t n, int d, uint64_t *__restrict__ key,
    int32_t *__restrict__ idx)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= n)
        return;
    const double R = sqrt((double)__uint_as_float(*maxn));
    const int b = (64 / d < 32) ? 64 / d : 32;
    const double levels = ldexp(1.0, b);
    uint32_t q[16];
    for (int c = 0; c < d; ++c) {
        const double xc = (double)(float)((double)X[p * d + c] - mu[c]);
        double u = (R > 0.0) ? (xc + R) / (2.0 * R) * levels : 0.0;
        u = u < 0.0 ? 0.0 : (u > levels - 1.0 ? levels - 1.0 : u);
        q[c] = (uint32_t)u;
    }
    uint64_t k = 0;
    for (int l = b - 1; l >= 0; --l)
        for (int c = 0; c < d; ++c)
            k = (k << 1) | ((q[c] >> l) & 1u);
    key[p] = k;
    idx[p] = (int32_t)p;
}

// Bounding box of the raw coordinates of every tile of kTileCols
// consecutive positions: box[t][c] = min, box[t][16 + c] = max.  A thread
// per (tile, coordinate); padding positions are left out.
__global__ __launch_bounds__(kThreads) void tile_box_kernel(
    const float *__restrict__ X, const int32_t *__restrict__ perm, int64_t n, int d,
    int64_t ntiles, float *__restrict__ box)
{
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= ntiles * 16)
        return;
    const int64_t t = e / 16;
    const int c = (int)(e % 16);
    if (c >= d)
        return;
    float lo = INFINITY, hi = -INFINITY;
    for (int64_t p = t * kTileCols; p < (t + 1) * kTileCols && p < n; ++p) {
        const float x = X[(int64_t)perm[p] * d + c];
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
    }
    box[t * 32 + c] = lo;
    box[t * 32 + 16 + c] = hi;
}

// 4 waves x 16 rows; all columns in tiles of 64 through double-buffered
// LDS (coordinate-major, XOR-swizzled as in the affinity engine);
// v_mfma_f32_16x16x4f32 with the A operand on the columns and the B operand
// on the wave's rows, so lane (m, g) holds row wrow0 + m and columns
// 16 q + 4 g + r of block q.  Every (i, j != i) whose squared distance
// passes thr_i is appended to row i's list (an integer atomic counter;
// slots beyond kCap are counted, not written).
template <int KS>
__global__ __launch_bounds__(kThreads) void knn_collect_kernel(
    const float *__restrict__ xa, int64_t np, const float *__restrict__ xb, int64_t n, int d,
    const int32_t *__restrict__ perm, const float *__restrict__ box,
    const float *__restrict__ thr, int *__restrict__ count, int32_t *__restrict__ cand)
{
    constexpr int KP = 4 * KS;
    constexpr int kRow4 = kTileCols / 4;
    static_assert(kRowsPerGroup == kTileCols, "a row group is one tile");
    __shared__ floatx4 xs[2][KP * kRow4];
    __shared__ int tl[kThreads];                 // column tiles of the current chunk
    __shared__ int wcnt[kThreads / kWave];
    __shared__ float wmax[kThreads / kWave];
    __shared__ float rbox[32];
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int g = lane >> 4;
    const int m = lane & 15;
    const int64_t wrow0 = (int64_t)blockIdx.x * kRowsPerGroup + wave * 16;
    const int64_t i = wrow0 + m;                 // position in Morton order
    const int64_t ic = i < n ? i : n - 1;
    const int64_t io = (i < n) ? (int64_t)perm[i] : -1;   // the point it holds
    const float t_i = (i < n) ? thr[io] : -1.0f;

    // a workgroup with no active row has nothing to collect
    if (__syncthreads_or(t_i >= 0.0f) == 0)
        return;

    // the largest bound among the workgroup's rows, and their box
    float tm = t_i;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1)
        tm = fmaxf(tm, __shfl_xor(tm, o, kWave));
    if (lane == 0)
        wmax[wave] = tm;
    if (threadIdx.x < 32)
        rbox[threadIdx.x] = box[(int64_t)blockIdx.x * 32 + threadIdx.x];
    __syncthreads();
    float tmax = wmax[0];
#pragma unroll
    for (int w = 1; w < kThreads / kWave; ++w)
        tmax = fmaxf(tmax, wmax[w]);
    // a tile is skipped when the squared gap between the boxes (float64,
    // exact differences of float32 coordinates) exceeds every bound
    const double cut = (double)tmax * (1.0 + 1e-12);

    float bop[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s)
        bop[s] = xb[ic * KP + 4 * s + g];

    constexpr int kPieces = KP * kRow4;
    constexpr int kPer = (kPieces + kThreads - 1) / kThreads;
    floatx4 stage[kPer];
    auto fetch = [&](int64_t jt) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = threadIdx.x + u * kThreads;
            if (kPieces % kThreads == 0 || f < kPieces)
                stage[u] = *reinterpret_cast<const floatx4 *>(
                    xa + (int64_t)(f / kRow4) * np + jt + 4 * (f % kRow4));
        }
    };
    auto commit = [&](int buf) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = threadIdx.x + u * kThreads;
            if (kPieces % kThreads == 0 || f < kPieces) {
                const int k = f / kRow4;
                xs[buf][k * kRow4 + ((f % kRow4) ^ (4 * (k & 3)))] = stage[u];
            }
        }
    };

    const int64_t ntiles = (n + kTileCols - 1) / kTileCols;
    for (int64_t c0 = 0; c0 < ntiles; c0 += kThreads) {
    // this chunk's tiles that may hold neighbours, in order
    bool pass = false;
    const int64_t tt = c0 + threadIdx.x;
    if (tt < ntiles) {
        const float *bx = box + tt * 32;
        double lb = 0.0;
        for (int c = 0; c < d; ++c) {
            double gap = (double)bx[c] - (double)rbox[16 + c];
            const double g2 = (double)rbox[c] - (double)bx[16 + c];
            gap = gap > g2 ? gap : g2;
            if (gap > 0.0)
                lb += gap * gap;
        }
        pass = !(lb > cut);
    }
    const unsigned long long bal = __ballot(pass);
    if (lane == 0)
        wcnt[wave] = __popcll(bal);
    __syncthreads();
    int before = 0, cnt = 0;
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) {
        before += (w < wave) ? wcnt[w] : 0;
        cnt += wcnt[w];
    }
    if (pass)
        tl[before + __popcll(bal & ((lane == 0) ? 0ull : (~0ull >> (kWave - lane))))] = (int)tt;
    __syncthreads();
    if (cnt == 0)
        continue;                                // uniform over the workgroup
    fetch((int64_t)tl[0] * kTileCols);
    commit(0);
    __syncthreads();
    for (int u = 0; u < cnt; ++u) {
        const int buf = u & 1;
        const int64_t jt = (int64_t)tl[u] * kTileCols;
        if (u + 1 < cnt)
            fetch((int64_t)tl[u + 1] * kTileCols);
        const float *tile = reinterpret_cast<const float *>(xs[buf]) + g * kTileCols;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            floatx4 cacc = {0.0f, 0.0f, 0.0f, 0.0f};
            const float *ap = tile + ((16 * q + m) ^ (16 * g));
#pragma unroll
            for (int s = 0; s < KS; ++s)
                cacc = __builtin_amdgcn_mfma_f32_16x16x4f32(ap[4 * s * kTileCols], bop[s],
                                                            cacc, 0, 0, 0);
            const int64_t j0 = jt + 16 * q + 4 * g;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t j = j0 + r;
                if (t_i >= 0.0f && cacc[r] <= t_i && j < n && j != i) {
                    const int c = atomicAdd(&count[io], 1);
                    if (c < kCap)
                        cand[io * kCap + c] = perm[j];
                }
            }
        }
        if (u + 1 < cnt) {
            commit(buf ^ 1);
            __syncthreads();
        }
    }
    __syncthreads();                             // tl and xs are refilled next chunk
    }
}

// ------------------------------------------------------------- 3. select

// A wave per active row: float64 squared distances of the kept candidates
// (at most kCap, 32 per lane, in registers), then k rounds of a wave
// argmin over (distance, index).  nbr[i k + t] are the k nearest in order;
// kth[i] is the k-th distance; a row whose list overflowed is flagged.
__global__ __launch_bounds__(kThreads) void knn_select_kernel(
    const float *__restrict__ X, int64_t n, int d, int k, const int *__restrict__ active,
    int *__restrict__ count, const int32_t *__restrict__ cand, int32_t *__restrict__ nbr,
    double *__restrict__ kth, int *__restrict__ flags)
{
    const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / kWave;
    const int lane = threadIdx.x % kWave;
    if (i >= n || (active != nullptr && !active[i]))
        return;                                             // uniform per wave
    const int cnt = count[i];
    const int kept = cnt < kCap ? cnt : kCap;
    double dv[kPerLane];
    int32_t jv[kPerLane];
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
        const int e = u * kWave + lane;
        if (e < kept) {
            jv[u] = cand[i * kCap + e];
            dv[u] = sq_dist64(X, d, i, jv[u]);
        } else {
            jv[u] = INT32_MAX;
            dv[u] = INFINITY;
        }
    }
    double last = 0.0;
    for (int t = 0; t < k; ++t) {
        double bd = INFINITY;
        int32_t bj = INT32_MAX;
#pragma unroll
        for (int u = 0; u < kPerLane; ++u)
            if (dv[u] < bd || (dv[u] == bd && jv[u] < bj)) {
                bd = dv[u];
                bj = jv[u];
            }
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) {
            const double od = __shfl_xor(bd, o, kWave);
            const int32_t oj = __shfl_xor(bj, o, kWave);
            if (od < bd || (od == bd && oj < bj)) {
                bd = od;
                bj = oj;
            }
        }
#pragma unroll
        for (int u = 0; u < kPerLane; ++u)
            if (jv[u] == bj)
                dv[u] = INFINITY, jv[u] = INT32_MAX;
        if (lane == 0)
            nbr[i * k + t] = bj;
        last = bd;
    }
    if (lane == 0) {
        kth[i] = last;
        if (cnt > kCap || last == INFINITY)
            atomicAdd(&flags[0], 1);
    }
}

// rows to collect again (count reset): the overflowed ones, and any with
// fewer than k candidates (an infinite k-th distance widens its bound to
// everything, so it overflows next and then shrinks)
__global__ __launch_bounds__(kThreads) void knn_rearm_kernel(int64_t n, int *__restrict__ count,
                                                             const double *__restrict__ kth,
                                                             int *__restrict__ active)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n)
        return;
    const int again = count[i] > kCap || kth[i] == INFINITY;
    active[i] = again;
    if (again)
        count[i] = 0;
}

__global__ __launch_bounds__(kThreads) void fill_i32_kernel(int *__restrict__ a, int64_t n,
                                                            int v)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads)
        a[i] = v;
}

// --------------------------------------------------------- 4. symmetrise

// Both directions of every kNN edge as (row, column) keys; with rank, in
// the node numbering rank[point] (the Morton position) instead of point
// indices.
__global__ __launch_bounds__(kThreads) void edge_keys_kernel(const int32_t *__restrict__ nbr,
                                                             int64_t n, int k, int bits,
                                                             const int32_t *__restrict__ rank,
                                                             uint64_t *__restrict__ key)
{
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= n * k)
        return;
    uint64_t a = (uint64_t)(e / k), b = (uint64_t)nbr[e];
    if (rank != nullptr) {
        a = (uint64_t)rank[a];
        b = (uint64_t)rank[b];
    }
    key[2 * e] = (a << bits) | b;
    key[2 * e + 1] = (b << bits) | a;
}

// rank[perm[p]] = p: the node number of every point in Morton numbering
__global__ __launch_bounds__(kThreads) void rank_kernel(const int32_t *__restrict__ perm,
                                                        int64_t n, int32_t *__restrict__ rank)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p < n)
        rank[perm[p]] = (int32_t)p;
}

// first[p] = 1 where sorted key p differs from key p - 1
__global__ __launch_bounds__(kThreads) void first_flags_kernel(const uint64_t *__restrict__ key,
                                                               int64_t m,
                                                               uint32_t *__restrict__ first)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p < m)
        first[p] = (p == 0 || key[p] != key[p - 1]) ? 1u : 0u;
}

// After an exclusive scan of the flags: column, row start and weight of
// every distinct key; row_ptr[n] = nnz.  With perm, node r is point
// perm[r] (the weight comes from the points' coordinates).
__global__ __launch_bounds__(kThreads) void build_csr_kernel(
    const uint64_t *__restrict__ key, const uint32_t *__restrict__ pos, int64_t m, int bits,
    const float *__restrict__ X, int64_t n, int d, double two_sigma2,
    const int32_t *__restrict__ perm, int64_t *__restrict__ row_ptr,
    int32_t *__restrict__ col, float *__restrict__ val)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= m)
        return;
    const uint64_t kp = key[p];
    const bool first = (p == 0 || kp != key[p - 1]);
    const uint64_t mask = (1ull << bits) - 1;
    const int64_t r = (int64_t)(kp >> bits), c = (int64_t)(kp & mask);
    if (p == m - 1)
        row_ptr[n] = (int64_t)pos[p] + (first ? 1 : 0);
    if (!first)
        return;
    const int64_t q = pos[p];
    col[q] = (int32_t)c;
    const int64_t pr = (perm != nullptr) ? (int64_t)perm[r] : r;
    const int64_t pc = (perm != nullptr) ? (int64_t)perm[c] : c;
    val[q] = (float)exp(-sq_dist64(X, d, pr, pc) / two_sigma2);
    if (p == 0 || (int64_t)(key[p - 1] >> bits) != r)
        row_ptr[r] = q;
}

int bits_for(int64_t n)
{
    int b = 1;
    while (((int64_t)1 << b) < n)
        ++b;
    return b;
}

struct KnnLayout {
    size_t xa, xb, mpart, mu, tau, norm2, maxn, thr, count, active, cand, nbr, kth, flags,
        keyA, keyB, first, hist, hsum, permA, permB, box, total;
};

KnnLayout knn_layout(int64_t n, int32_t k)
{
    KnnLayout L{};
    const int64_t np = padded_points(n);
    const int64_t m = 2 * n * (int64_t)k;
    size_t o = 0;
    auto take = [&](int64_t bytes) {
        const size_t at = o;
        o += (size_t)al(bytes);
        return at;
    };
    L.xa = take(np * 20 * 4);               // KP <= 20 for d <= 16
    L.xb = take(np * 20 * 4);
    L.mpart = take(kMeanBlocks * 16 * 8);
    L.mu = take(16 * 8);
    L.tau = take(n * 4);
    L.norm2 = take(n * 4);
    L.maxn = take(4);
    L.thr = take(n * 4);
    L.count = take(n * 4);
    L.active = take(n * 4);
    L.cand = take(n * (int64_t)kCap * 4);
    L.nbr = take(n * (int64_t)k * 4);
    L.kth = take(n * 8);
    L.flags = take(4);
    L.keyA = take(m * 8);
    L.keyB = take(m * 8);
    L.first = take(m * 4);
    L.hist = take((int64_t)radix_hist_bytes(m));
    L.hsum = take((int64_t)(radix_hsum_bytes(m) > scan_sums_bytes(m) ? radix_hsum_bytes(m)
                                                                      : scan_sums_bytes(m)));
    L.permA = take(n * 4);
    L.permB = take(n * 4);
    L.box = take(np / kTileCols * 32 * 4);
    L.total = o;
    return L;
}

template <int D>
void launch_bound(int KT, const float *X, const int32_t *perm, int64_t n, int k, float *tau,
                  hipStream_t s)
{
    const dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
    switch (KT) {
    case 8:
        hipLaunchKernelGGL((knn_bound_kernel<D, 8>), grid, dim3(kThreads), 0, s, X, perm, n, k,
                           tau);
        break;
    case 16:
        hipLaunchKernelGGL((knn_bound_kernel<D, 16>), grid, dim3(kThreads), 0, s, X, perm, n,
                           k, tau);
        break;
    case 32:
        hipLaunchKernelGGL((knn_bound_kernel<D, 32>), grid, dim3(kThreads), 0, s, X, perm, n,
                           k, tau);
        break;
    default:
        hipLaunchKernelGGL((knn_bound_kernel<D, 64>), grid, dim3(kThreads), 0, s, X, perm, n,
                           k, tau);
        break;
    }
}

} // namespace

size_t knn_graph_ws(int64_t n, int32_t k) { return knn_layout(n, k).total; }

hipError_t run_knn_graph(const float *X, int64_t n, int d, int k, float sigma,
                         int64_t *row_ptr, int32_t *col, float *val, int64_t *nnz_host,
                         int *status_host, void *ws, hipStream_t s, int32_t *perm_out)
{
    const KnnLayout L = knn_layout(n, k);
    char *w = static_cast<char *>(ws);
    float *xa = (float *)(w + L.xa), *xb = (float *)(w + L.xb);
    double *mpart = (double *)(w + L.mpart), *mu = (double *)(w + L.mu);
    float *tau = (float *)(w + L.tau), *norm2 = (float *)(w + L.norm2);
    unsigned int *maxn = (unsigned int *)(w + L.maxn);
    float *thr = (float *)(w + L.thr);
    int *count = (int *)(w + L.count), *active = (int *)(w + L.active);
    int32_t *cand = (int32_t *)(w + L.cand), *nbr = (int32_t *)(w + L.nbr);
    double *kth = (double *)(w + L.kth);
    int *flags = (int *)(w + L.flags);
    uint64_t *keyA = (uint64_t *)(w + L.keyA), *keyB = (uint64_t *)(w + L.keyB);
    uint32_t *first = (uint32_t *)(w + L.first);
    uint32_t *hist = (uint32_t *)(w + L.hist), *hsum = (uint32_t *)(w + L.hsum);
    const unsigned rows_grid = (unsigned)((n + kThreads - 1) / kThreads);
    *status_host = 0;

    if (d < 1 || d > 16)
        return hipErrorInvalidValue;
    const int KS = ks_for(d);
    const int64_t np = padded_points(n);
    hipLaunchKernelGGL(mean_partials_kernel, dim3(kMeanBlocks), dim3(kThreads), 0, s, X, n, d,
                       mpart);
    hipLaunchKernelGGL(mean_finish_kernel, dim3(1), dim3(64), 0, s, mpart, kMeanBlocks, d, n,
                       mu);
    const unsigned pgrid = (unsigned)((np + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(knn_augment_kernel, dim3(pgrid), dim3(kThreads), 0, s, X, mu,
                       (const int32_t *)nullptr, n, np, d, 4 * KS, xa, xb, norm2);
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(kThreads), 0, s, (int *)maxn,
                       (int64_t)1, 0);
    hipLaunchKernelGGL(max_norm_kernel, dim3(1024), dim3(kThreads), 0, s, norm2, n, maxn);
    // Morton order of the points, the operands in that order, tile boxes
    int32_t *perm = (int32_t *)(w + L.permA), *permB = (int32_t *)(w + L.permB);
    uint64_t *mkA = keyA, *mkB = keyB;
    hipLaunchKernelGGL(morton_key_kernel, dim3(rows_grid), dim3(kThreads), 0, s, X, mu,
                       (const unsigned int *)maxn, n, d, mkA, perm);
    hipError_t e0 = radix_sort_u64(mkA, perm, mkB, permB, n, 64, hist, hsum, s);
    if (e0 != hipSuccess)
        return e0;
    hipLaunchKernelGGL(knn_augment_kernel, dim3(pgrid), dim3(kThreads), 0, s, X, mu,
                       (const int32_t *)perm, n, np, d, 4 * KS, xa, xb, norm2);
    const int64_t ntiles = np / kTileCols;
    float *box = (float *)(w + L.box);
    hipLaunchKernelGGL(tile_box_kernel, dim3((unsigned)((ntiles * 16 + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, X, (const int32_t *)perm, n, d, ntiles, box);

    // 1. bound, over the Morton neighbours
    const int KT = k <= 8 ? 8 : k <= 16 ? 16 : k <= 32 ? 32 : 64;
#define GPIC_BOUND(D)                                                          \
    case D:                                                                    \
        launch_bound<D>(KT, X, perm, n, k, tau, s);                            \
        break;
    switch (d) {
        GPIC_BOUND(1) GPIC_BOUND(2) GPIC_BOUND(3) GPIC_BOUND(4) GPIC_BOUND(5) GPIC_BOUND(6)
        GPIC_BOUND(7) GPIC_BOUND(8) GPIC_BOUND(9) GPIC_BOUND(10) GPIC_BOUND(11)
        GPIC_BOUND(12) GPIC_BOUND(13) GPIC_BOUND(14) GPIC_BOUND(15) GPIC_BOUND(16)
    default:
        return hipErrorInvalidValue;
    }
#undef GPIC_BOUND
    hipLaunchKernelGGL(threshold_kernel, dim3(rows_grid), dim3(kThreads), 0, s, tau,
                       (const double *)nullptr, norm2, maxn, n, d, 4 * KS,
                       (const int *)nullptr, thr);
    hipLaunchKernelGGL(fill_i32_kernel, dim3(4096), dim3(kThreads), 0, s, count, n, 0);

    // 2-3. collect and select, again for overflowed rows
    const int *act = nullptr;
    for (int round = 0;; ++round) {
        const dim3 cgrid((unsigned)((n + kRowsPerGroup - 1) / kRowsPerGroup));
        if (KS <= 3)
            hipLaunchKernelGGL(knn_collect_kernel<3>, cgrid, dim3(kThreads), 0, s, xa, np,
                               xb, n, d, (const int32_t *)perm, (const float *)box, thr, count,
                               cand);
        else
            hipLaunchKernelGGL(knn_collect_kernel<5>, cgrid, dim3(kThreads), 0, s, xa, np,
                               xb, n, d, (const int32_t *)perm, (const float *)box, thr, count,
                               cand);
        hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(kThreads), 0, s, flags, (int64_t)1,
                           0);
        hipLaunchKernelGGL(knn_select_kernel,
                           dim3((unsigned)((n * kWave + kThreads - 1) / kThreads)),
                           dim3(kThreads), 0, s, X, n, d, k, act, count, cand, nbr, kth,
                           flags);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        int bad = 0;
        if ((e = hipMemcpyAsync(&bad, flags, sizeof(int), hipMemcpyDeviceToHost, s)) !=
                hipSuccess ||
            (e = hipStreamSynchronize(s)) != hipSuccess)
            return e;
        if (bad == 0)
            break;
        if (round == 8) {                   // bounds that do not shrink: give up
            *status_host = 1;
            return hipSuccess;
        }
        hipLaunchKernelGGL(knn_rearm_kernel, dim3(rows_grid), dim3(kThreads), 0, s, n,
                           count, (const double *)kth, active);
        hipLaunchKernelGGL(threshold_kernel, dim3(rows_grid), dim3(kThreads), 0, s, tau,
                           (const double *)kth, norm2, maxn, n, d, 4 * KS,
                           (const int *)active, thr);
        act = active;
    }

    // 4. symmetrise (in Morton numbering when the caller takes the order:
    // the sort's spare index buffer holds the ranks)
    const int bits = bits_for(n);
    const int64_t mm = 2 * n * (int64_t)k;
    int32_t *rank = nullptr;
    if (perm_out != nullptr) {
        rank = permB;
        hipLaunchKernelGGL(rank_kernel, dim3(rows_grid), dim3(kThreads), 0, s,
                           (const int32_t *)perm, n, rank);
    }
    hipLaunchKernelGGL(edge_keys_kernel, dim3((unsigned)((n * k + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, nbr, n, k, bits, (const int32_t *)rank, keyA);
    int32_t *none_a = nullptr, *none_b = nullptr;
    hipError_t e = radix_sort_u64(keyA, none_a, keyB, none_b, mm, (2 * bits + 7) / 8 * 8,
                                  hist, hsum, s);
    if (e != hipSuccess)
        return e;
    const unsigned egrid = (unsigned)((mm + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(first_flags_kernel, dim3(egrid), dim3(kThreads), 0, s, keyA, mm, first);
    if ((e = exclusive_scan_u32(first, mm, hsum, s)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(build_csr_kernel, dim3(egrid), dim3(kThreads), 0, s, keyA, first, mm,
                       bits, X, n, d, 2.0 * (double)sigma * (double)sigma,
                       perm_out != nullptr ? (const int32_t *)perm : nullptr, row_ptr, col,
                       val);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (perm_out != nullptr &&
        (e = hipMemcpyAsync(perm_out, perm, (size_t)n * 4, hipMemcpyDeviceToDevice, s)) !=
            hipSuccess)
        return e;
    if ((e = hipMemcpyAsync(nnz_host, row_ptr + n, sizeof(int64_t), hipMemcpyDeviceToHost,
                            s)) != hipSuccess)
        return e;
    return hipStreamSynchronize(s);
}

} // namespace gpic
