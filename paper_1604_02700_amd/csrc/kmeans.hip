// Exact one-dimensional k-means for gfx950: the "k-means of v" step that
// ends Algorithms 1 and 2, read as the minimum within-cluster sum of
// squares partition of the scalars v_i.
//
// Steps (all deterministic):
//   1. order-preserving 64-bit keys of v, stable LSD radix sort (8 passes of
//      8 bits) of (key, index) pairs: tile histograms, one exclusive scan,
//      stable scatter with in-wave ranks from ballots;
//   2. run starts of equal values (a cluster never splits equal values),
//      their count, the mean, and float64 prefix sums S1, S2 of the centred
//      values u = v_sorted - mean;
//   3. dynamic programme over layers c = 1..k_eff-1:
//        D_c(i) = min_{j <= i, j starts a run} D_{c-1}(j-1) + cost(j, i),
//        cost(j, i) = max(0, (S2[i+1]-S2[j]) - (S1[i+1]-S1[j])^2 / (i-j+1)),
//      with the leftmost argmin; split points are monotone in i (quadrangle
//      inequality of the 1-D within-cluster sum of squares), so each layer
//      is solved by F-ary divide and conquer (a few dependent levels);
//   4. backtrack, per-cluster means and sums of squares, labels by
//      ascending centroid.
#include "common.h"

namespace gpic {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;   // elements per sort / scan tile
constexpr int kRadix = 256;

__host__ __device__ inline int64_t tiles(int64_t n) { return (n + kTile - 1) / kTile; }

__device__ __forceinline__ uint64_t to_key(double x)
{
    if (x == 0.0)
        x = 0.0;                       // -0 and +0 are equal values
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double from_key(uint64_t k)
{
    const uint64_t b = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
    return __longlong_as_double((long long)b);
}

__global__ __launch_bounds__(kThreads) void make_keys_kernel(
    const double *__restrict__ v, int64_t n, uint64_t *__restrict__ key,
    int32_t *__restrict__ idx)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) {
        key[i] = to_key(v[i]);
        idx[i] = (int32_t)i;
    }
}


// Sorted values, run starts, and per-tile sums of values and run starts.
__global__ __launch_bounds__(kThreads) void decode_kernel(
    const uint64_t *__restrict__ key, int64_t n, double *__restrict__ sv,
    int32_t *__restrict__ run, double *__restrict__ tsum,
    double *__restrict__ truns)
{
    __shared__ double red[kThreads / kWave];
    const int64_t tb = (int64_t)blockIdx.x * kTile;
    double s = 0.0, r = 0.0;
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = tb + it * kThreads + threadIdx.x;
        if (i < n) {
            const uint64_t k = key[i];
            const double x = from_key(k);
            sv[i] = x;
            const int st = (i == 0) || (key[i - 1] != k);
            run[i] = st;
            s += x;
            r += st;
        }
    }
    const double ts = block_sum<kThreads>(s, red);
    const double tr = block_sum<kThreads>(r, red);
    if (threadIdx.x == 0) {
        tsum[blockIdx.x] = ts;
        truns[blockIdx.x] = tr;
    }
}

struct KmScalars {
    double mean;
    double distinct;
};

__global__ __launch_bounds__(1024) void totals_kernel(
    const double *__restrict__ tsum, const double *__restrict__ truns,
    int64_t nt, int64_t n, KmScalars *__restrict__ sc)
{
    __shared__ double red[1024 / kWave];
    double s = 0.0, r = 0.0;
    for (int64_t b = threadIdx.x; b < nt; b += 1024) {
        s += tsum[b];
        r += truns[b];
    }
    const double ts = block_sum<1024>(s, red);
    const double tr = block_sum<1024>(r, red);
    if (threadIdx.x == 0) {
        sc->mean = ts / (double)n;
        sc->distinct = tr;
    }
}

// Per-tile totals of u and u^2 (u = value - mean), each thread summing its
// kItems consecutive elements.
__global__ __launch_bounds__(kThreads) void tile_moments_kernel(
    const double *__restrict__ sv, int64_t n, const KmScalars *__restrict__ sc,
    double *__restrict__ t1, double *__restrict__ t2)
{
    __shared__ double red[kThreads / kWave];
    const double mu = sc->mean;
    const int64_t b = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    double s1 = 0.0, s2 = 0.0;
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = b + it;
        if (i < n) {
            const double u = sv[i] - mu;
            s1 += u;
            s2 += u * u;
        }
    }
    // thread totals in thread order: serial over the block's 256 totals
    __shared__ double a1[kThreads], a2[kThreads];
    a1[threadIdx.x] = s1;
    a2[threadIdx.x] = s2;
    __syncthreads();
    if (threadIdx.x == 0) {
        double x1 = 0.0, x2 = 0.0;
        for (int t = 0; t < kThreads; ++t) {
            x1 += a1[t];
            x2 += a2[t];
        }
        t1[blockIdx.x] = x1;
        t2[blockIdx.x] = x2;
    }
    (void)red;
}

// Exclusive scan of the tile totals (serial: there are few tiles).
__global__ void scan_tiles_kernel(double *__restrict__ t1, double *__restrict__ t2,
                                  int64_t nt)
{
    if (threadIdx.x != 0)
        return;
    double r1 = 0.0, r2 = 0.0;
    for (int64_t b = 0; b < nt; ++b) {
        const double x1 = t1[b], x2 = t2[b];
        t1[b] = r1;
        t2[b] = r2;
        r1 += x1;
        r2 += x2;
    }
}

// S1[i+1], S2[i+1] = tile offset + in-tile running sums (each thread walks
// its kItems elements after an exclusive scan of the thread totals).
__global__ __launch_bounds__(kThreads) void prefix_kernel(
    const double *__restrict__ sv, int64_t n, const KmScalars *__restrict__ sc,
    const double *__restrict__ o1, const double *__restrict__ o2,
    double *__restrict__ S1, double *__restrict__ S2)
{
    __shared__ double a1[kThreads], a2[kThreads];
    const double mu = sc->mean;
    const int64_t b = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    double s1 = 0.0, s2 = 0.0;
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = b + it;
        if (i < n) {
            const double u = sv[i] - mu;
            s1 += u;
            s2 += u * u;
        }
    }
    a1[threadIdx.x] = s1;
    a2[threadIdx.x] = s2;
    __syncthreads();
    if (threadIdx.x == 0) {
        double r1 = o1[blockIdx.x], r2 = o2[blockIdx.x];
        for (int t = 0; t < kThreads; ++t) {
            const double x1 = a1[t], x2 = a2[t];
            a1[t] = r1;
            a2[t] = r2;
            r1 += x1;
            r2 += x2;
        }
    }
    __syncthreads();
    double r1 = a1[threadIdx.x], r2 = a2[threadIdx.x];
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = b + it;
        if (i < n) {
            const double u = sv[i] - mu;
            r1 += u;
            r2 += u * u;
            S1[i + 1] = r1;
            S2[i + 1] = r2;
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        S1[0] = 0.0;
        S2[0] = 0.0;
    }
}

__device__ __forceinline__ double seg_cost(const double *__restrict__ S1,
                                           const double *__restrict__ S2,
                                           int64_t j, int64_t i)
{
    const double m = (double)(i - j + 1);
    const double s1 = S1[i + 1] - S1[j];
    const double s2 = S2[i + 1] - S2[j];
    const double c = s2 - s1 * s1 / m;
    return c > 0.0 ? c : 0.0;
}

__global__ __launch_bounds__(kThreads) void first_layer_kernel(
    const double *__restrict__ S1, const double *__restrict__ S2, int64_t n,
    double *__restrict__ D, unsigned long long *__restrict__ qlen)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n)
        D[i] = seg_cost(S1, S2, 0, i);
    if (i < 4)
        qlen[i] = 0ull;                 // the recursion's part and row counters
}

// ---------------------------------------------------------------- layers
//
// Each layer is solved by F-ary divide and conquer: an interval of rows
// [lo, hi] whose neighbours' optimal split points are known takes F evenly
// spaced sample rows (all its rows if it has at most F) and computes their
// leftmost argmins in parallel, each over the interval's bounds
// [opt(lo-1), opt(hi+1)]; the F+1 gaps between samples are the next
// level's intervals.  ceil(log_{F+1} n) levels replace the log2 n of a
// binary split, which matters because every level is a dependent step; in
// exchange every candidate of a level is scanned by F samples.  F = 64 up
// to 2^18 rows (few dependent steps), F = 8 above (less redundant work).
constexpr int kFSmall = 64;
constexpr int kFLarge = 8;
constexpr int64_t kFLargeFrom = (int64_t)1 << 18;
constexpr int kMaxLevels = 16;
constexpr int kShortScan = 32;        // longer ranges go to the work queue
constexpr int kChunk = 1024;          // candidates per queued part (16 per lane)

// Sample f of interval [lo, hi] (m = hi - lo + 1 rows): every row if m <= F,
// else lo + (f + 1)(m + 1) / (F + 1) - 1; returns -1 if there is none.
template <int F>
__device__ __forceinline__ int64_t sample_row(int64_t lo, int64_t hi, int f)
{
    const int64_t m = hi - lo + 1;
    if (m <= F)
        return (f < m) ? lo + f : -1;
    return lo + ((int64_t)(f + 1) * (m + 1)) / (F + 1) - 1;
}

// Interval of node q at level L (digits of q in base F + 1, most significant
// first, choose the gap between samples); false if the node does not exist.
template <int F>
__device__ __forceinline__ bool fary_node(int64_t n, int L, int64_t q, int64_t &lo,
                                          int64_t &hi)
{
    int dig[kMaxLevels];
    for (int l = 0; l < L; ++l) {
        dig[l] = (int)(q % (F + 1));
        q /= (F + 1);
    }
    lo = 0;
    hi = n - 1;
    for (int l = L - 1; l >= 0; --l) {
        if (hi - lo + 1 <= F)
            return false;                     // a leaf interval has no gaps
        const int c = dig[l];
        const int64_t nlo = (c == 0) ? lo : sample_row<F>(lo, hi, c - 1) + 1;
        const int64_t nhi = (c == F) ? hi : sample_row<F>(lo, hi, c) - 1;
        lo = nlo;
        hi = nhi;
        if (lo > hi)
            return false;
    }
    return true;
}

// Leftmost-argmin merge of (value, index) pairs.
__device__ __forceinline__ void amin_merge(double &b, int64_t &a, double ob,
                                           int64_t oa)
{
    if (ob < b || (ob == b && oa < a)) {
        b = ob;
        a = oa;
    }
}

// Scan split points j = from, from + stride, ... <= ahi for row r, keeping
// the leftmost minimum of Dprev[j-1] + cost(j, r) over run starts.  Every
// candidate is evaluated without branching so successive loads overlap.
__device__ __forceinline__ void scan_range(const double *__restrict__ S1,
                                           const double *__restrict__ S2,
                                           const int32_t *__restrict__ run,
                                           const double *__restrict__ Dprev,
                                           int64_t r, int64_t from, int64_t ahi,
                                           int64_t stride, double &best,
                                           int64_t &arg)
{
#pragma unroll 4
    for (int64_t j = from; j <= ahi; j += stride) {
        const double cst = Dprev[j - 1] + seg_cost(S1, S2, j, r);
        const double c = run[j] ? cst : INFINITY;
        if (c < best) {
            best = c;
            arg = j;
        }
    }
}

__device__ __forceinline__ void wave_argmin(double &best, int64_t &arg)
{
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const double ob = __shfl_xor(best, o, kWave);
        const long long oa = __shfl_xor((long long)arg, o, kWave);
        amin_merge(best, arg, ob, (int64_t)oa);
    }
}

// Row r of interval [lo, hi]: candidate split points [alo, ahi].
__device__ __forceinline__ void row_bounds(const int32_t *__restrict__ opt, int64_t n,
                                           int64_t lo, int64_t hi, int64_t r,
                                           int64_t &alo, int64_t &ahi)
{
    const int64_t olo = (lo > 0) ? (int64_t)opt[lo - 1] : 1;
    const int64_t ohi = (hi < n - 1) ? (int64_t)opt[hi + 1] : n - 1;
    alo = olo < 1 ? 1 : olo;
    ahi = ohi < r ? ohi : r;
}

__device__ __forceinline__ void store_result(double *__restrict__ Dcur,
                                             int32_t *__restrict__ opt, int64_t r,
                                             double best, int64_t arg, int64_t alo)
{
    Dcur[r] = best;
    opt[r] = (int32_t)((arg == INT64_MAX) ? alo : arg);
}

// A queued part: candidates [alo, ahi] of row r; head is the slot of the
// row's first part (its part count lives there).  r < 0
// marks a slot that holds no work.
struct QueuePart {
    int32_t r, alo, ahi, head;
};

struct LevelQueue {
    QueuePart *part;
    int32_t *nparts;                     // indexed by head
    int32_t *heads;                      // heads of rows with more than one part
    double *pbest;                       // per part
    int32_t *parg;
    unsigned long long *qlen;            // parts: [g & 1]; rows: [2 + (g & 1)]
    int64_t cap;
};

// One recursion level: a thread per (node, sample).  A short range is
// scanned by the thread itself; a long one is cut into parts of kChunk
// candidates appended to the queue (the order of appends does not matter:
// every row's parts are merged by an order-independent minimum).  Item 0
// clears the other pair of counters, whose level has finished.
template <int F>
__global__ __launch_bounds__(kThreads) void fary_level_kernel(
    const double *__restrict__ S1, const double *__restrict__ S2,
    const int32_t *__restrict__ run, const double *__restrict__ Dprev,
    double *__restrict__ Dcur, int32_t *__restrict__ opt, int64_t n, int L,
    int64_t items, LevelQueue Q, int g)
{
    const int64_t item = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (item == 0) {
        Q.qlen[(g + 1) & 1] = 0ull;
        Q.qlen[2 + ((g + 1) & 1)] = 0ull;
    }
    int64_t lo = 0, hi = -1, r = -1, alo = 1, ahi = 0;
    if (item < items && fary_node<F>(n, L, item / F, lo, hi)) {
        r = sample_row<F>(lo, hi, (int)(item % F));
        if (r >= 0)
            row_bounds(opt, n, lo, hi, r, alo, ahi);
    }
    const int64_t len = ahi - alo + 1;
    // long ranges: reserve parts; up to 64 parts are written by their own
    // thread, more by the whole wave, one such lane after the other
    bool queued = false;
    int64_t e0 = 0, C = 0;
    if (r >= 0 && len > kShortScan) {
        C = (len + kChunk - 1) / kChunk;
        e0 = (int64_t)atomicAdd(&Q.qlen[g & 1], (unsigned long long)C);
        queued = e0 + C <= Q.cap;
        if (queued) {
            Q.nparts[e0] = (int32_t)C;
            if (C > 1) {
                const unsigned long long h = atomicAdd(&Q.qlen[2 + (g & 1)], 1ull);
                Q.heads[h] = (int32_t)e0;             // h < e0 + 1 <= cap
            }
        } else {
            // no room left (only if split points were far from monotone):
            // void the reserved slots below the capacity and scan here
            for (int64_t e = e0; e < e0 + C && e < Q.cap; ++e)
                Q.part[e] = QueuePart{-1, 0, -1, 0};
        }
    }
    if (queued && C <= kWave) {
        for (int64_t p = 0; p < C; ++p) {
            const int64_t plo = alo + p * kChunk;
            const int64_t phi = plo + kChunk - 1 < ahi ? plo + kChunk - 1 : ahi;
            Q.part[e0 + p] = QueuePart{(int32_t)r, (int32_t)plo, (int32_t)phi,
                                       (int32_t)e0};
        }
    }
    const int lane = threadIdx.x % kWave;
    unsigned long long mask = __ballot(queued && C > kWave);
    while (mask) {
        const int src = __ffsll((long long)mask) - 1;
        mask &= mask - 1;
        const long long qe0 = __shfl((long long)e0, src, kWave);
        const long long qC = __shfl((long long)C, src, kWave);
        const long long qr = __shfl((long long)r, src, kWave);
        const long long qalo = __shfl((long long)alo, src, kWave);
        const long long qahi = __shfl((long long)ahi, src, kWave);
        for (long long p = lane; p < qC; p += kWave) {
            const long long plo = qalo + p * kChunk;
            const long long phi = plo + kChunk - 1 < qahi ? plo + kChunk - 1 : qahi;
            Q.part[qe0 + p] = QueuePart{(int32_t)qr, (int32_t)plo, (int32_t)phi,
                                        (int32_t)qe0};
        }
    }
    if (r < 0 || queued)
        return;
    double best = INFINITY;
    int64_t arg = INT64_MAX;
    scan_range(S1, S2, run, Dprev, r, alo, ahi, 1, best, arg);
    store_result(Dcur, opt, r, best, arg, alo);
}

// The level's queued parts: wave w of the grid takes parts w, w + waves, ...
// and scans each with its 64 lanes.  A row with one part is finished here;
// otherwise the part leaves its minimum for fary_merge_kernel.
__global__ __launch_bounds__(kThreads) void fary_queue_kernel(
    const double *__restrict__ S1, const double *__restrict__ S2,
    const int32_t *__restrict__ run, const double *__restrict__ Dprev,
    double *__restrict__ Dcur, int32_t *__restrict__ opt, LevelQueue Q, int g)
{
    const int64_t total = (int64_t)Q.qlen[g & 1];
    const int64_t len = total < Q.cap ? total : Q.cap;
    const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
    const int lane = threadIdx.x % kWave;
    for (int64_t e = (int64_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
         e < len; e += waves) {
        const QueuePart q = Q.part[e];
        if (q.r < 0)
            continue;                                   // uniform per wave
        double best = INFINITY;
        int64_t arg = INT64_MAX;
        scan_range(S1, S2, run, Dprev, q.r, (int64_t)q.alo + lane, q.ahi, kWave, best,
                   arg);
        wave_argmin(best, arg);
        if (lane == 0) {
            if (Q.nparts[q.head] == 1) {
                store_result(Dcur, opt, q.r, best, arg, q.alo);
            } else {
                Q.pbest[e] = best;
                Q.parg[e] = (arg == INT64_MAX) ? INT32_MAX : (int32_t)arg;
            }
        }
    }
}

// Rows with several parts: a wave per row merges its parts' minima.
__global__ __launch_bounds__(kThreads) void fary_merge_kernel(
    double *__restrict__ Dcur, int32_t *__restrict__ opt, LevelQueue Q, int g)
{
    const int64_t nh = (int64_t)Q.qlen[2 + (g & 1)];
    const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
    const int lane = threadIdx.x % kWave;
    for (int64_t h = (int64_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
         h < nh; h += waves) {
        const int64_t head = Q.heads[h];
        const QueuePart q = Q.part[head];
        const int C = Q.nparts[head];
        double best = INFINITY;
        int64_t arg = INT64_MAX;
        for (int p = lane; p < C; p += kWave) {
            const int32_t a = Q.parg[head + p];
            amin_merge(best, arg, Q.pbest[head + p],
                       a == INT32_MAX ? INT64_MAX : (int64_t)a);
        }
        wave_argmin(best, arg);
        if (lane == 0)
            store_result(Dcur, opt, q.r, best, arg, q.alo);
    }
}

__global__ void backtrack_kernel(const int32_t *__restrict__ opt, int64_t n,
                                 int ke, int64_t *__restrict__ first)
{
    if (threadIdx.x != 0 || blockIdx.x != 0)
        return;
    int64_t i = n - 1;
    for (int c = ke - 1; c >= 1; --c) {
        const int64_t j = opt[(int64_t)c * n + i];
        first[c] = j;
        i = j - 1;
    }
    first[0] = 0;
    first[ke] = n;
}

// One workgroup per cluster: mean (sum in a fixed order / count) and the
// sum of squared deviations from it.
__global__ __launch_bounds__(kThreads) void cluster_stats_kernel(
    const double *__restrict__ sv, const int64_t *__restrict__ first,
    double *__restrict__ centroids, double *__restrict__ costs)
{
    __shared__ double red[kThreads / kWave];
    const int c = blockIdx.x;
    const int64_t b = first[c], e = first[c + 1];
    double s = 0.0;
    for (int64_t p = b + threadIdx.x; p < e; p += kThreads)
        s += sv[p];
    const double mu = block_sum<kThreads>(s, red) / (double)(e - b);
    double q = 0.0;
    for (int64_t p = b + threadIdx.x; p < e; p += kThreads)
        q += (sv[p] - mu) * (sv[p] - mu);
    const double tq = block_sum<kThreads>(q, red);
    if (threadIdx.x == 0) {
        centroids[c] = mu;
        costs[c] = tq;
    }
}

__global__ __launch_bounds__(kThreads) void labels_kernel(
    const int32_t *__restrict__ idx, int64_t n, const int64_t *__restrict__ first,
    int ke, int32_t *__restrict__ labels)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= n)
        return;
    int lo = 0, hi = ke - 1;        // last c with first[c] <= p
    while (lo < hi) {
        const int m = (lo + hi + 1) / 2;
        if (first[m] <= p)
            lo = m;
        else
            hi = m - 1;
    }
    labels[idx[p]] = lo;
}

inline size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

struct KmLayout {
    size_t keyA, keyB, idxA, idxB, hist, hsum, sv, run, t1, t2, S1, S2, Da, Db, opt,
        qpart, qnparts, qheads, qbest, qarg, qlen, sc, first, costs, total;
};

// Queue slots per level.  With monotone split points the ranges of one
// level overlap only at their ends, so they hold at most 2 F n candidates
// and at most n + 2 F n / kChunk parts; a level that would need more
// scans the excess in place.
int64_t queue_cap(int64_t n) { return n + (2 * kFSmall * n) / kChunk + 1024; }

KmLayout layout(int64_t n, int32_t k)
{
    KmLayout L{};
    const int64_t nt = tiles(n);
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += al(bytes);
        return at;
    };
    L.keyA = take(n * 8);
    L.keyB = take(n * 8);
    L.idxA = take(n * 4);
    L.idxB = take(n * 4);
    L.hist = take((size_t)kRadix * nt * 4);
    L.hsum = take((size_t)tiles(kRadix * nt) * 4);
    L.sv = take(n * 8);
    L.run = take(n * 4);
    L.t1 = take(nt * 8);
    L.t2 = take(nt * 8);
    L.S1 = take((n + 1) * 8);
    L.S2 = take((n + 1) * 8);
    L.Da = take(n * 8);
    L.Db = take(n * 8);
    L.opt = take((size_t)k * n * 4);
    const size_t cap = (size_t)queue_cap(n);
    L.qpart = take(cap * sizeof(QueuePart));
    L.qnparts = take(cap * 4);
    L.qheads = take(cap * 4);
    L.qbest = take(cap * 8);
    L.qarg = take(cap * 4);
    L.qlen = take(4 * 8);
    L.sc = take(sizeof(KmScalars));
    L.first = take((size_t)(k + 1) * 8);
    L.costs = take((size_t)k * 8);
    L.total = o;
    return L;
}

unsigned blocks_for(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

} // namespace

size_t kmeans_ws(int64_t n, int32_t k) { return layout(n, k).total; }

#define GPIC_TRY(x)                                                            \
    do {                                                                       \
        hipError_t e_ = (x);                                                   \
        if (e_ != hipSuccess)                                                  \
            return e_;                                                         \
    } while (0)

hipError_t run_kmeans1d(const double *v, int64_t n, int32_t k, int32_t *labels,
                        double *centroids, int32_t *k_eff, double *cost,
                        void *ws, hipStream_t s)
{
    const KmLayout L = layout(n, k);
    char *w = static_cast<char *>(ws);
    uint64_t *keyA = (uint64_t *)(w + L.keyA), *keyB = (uint64_t *)(w + L.keyB);
    int32_t *idxA = (int32_t *)(w + L.idxA), *idxB = (int32_t *)(w + L.idxB);
    uint32_t *hist = (uint32_t *)(w + L.hist);
    uint32_t *hsum = (uint32_t *)(w + L.hsum);
    double *sv = (double *)(w + L.sv);
    int32_t *run = (int32_t *)(w + L.run);
    double *t1 = (double *)(w + L.t1), *t2 = (double *)(w + L.t2);
    double *S1 = (double *)(w + L.S1), *S2 = (double *)(w + L.S2);
    double *Da = (double *)(w + L.Da), *Db = (double *)(w + L.Db);
    int32_t *opt = (int32_t *)(w + L.opt);
    LevelQueue Q;
    Q.part = (QueuePart *)(w + L.qpart);
    Q.nparts = (int32_t *)(w + L.qnparts);
    Q.heads = (int32_t *)(w + L.qheads);
    Q.pbest = (double *)(w + L.qbest);
    Q.parg = (int32_t *)(w + L.qarg);
    Q.qlen = (unsigned long long *)(w + L.qlen);
    Q.cap = queue_cap(n);
    KmScalars *sc = (KmScalars *)(w + L.sc);
    int64_t *first = (int64_t *)(w + L.first);
    double *costs = (double *)(w + L.costs);
    const int64_t nt = tiles(n);

    // 1. radix sort
    hipLaunchKernelGGL(make_keys_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s,
                       v, n, keyA, idxA);
    GPIC_TRY(radix_sort_u64(keyA, idxA, keyB, idxB, n, 64, hist, hsum, s));
    GPIC_TRY(hipGetLastError());

    // 2. values, runs, mean, prefix sums
    hipLaunchKernelGGL(decode_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s, keyA,
                       n, sv, run, t1, t2);
    hipLaunchKernelGGL(totals_kernel, dim3(1), dim3(1024), 0, s, t1, t2, nt, n, sc);
    hipLaunchKernelGGL(tile_moments_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s,
                       sv, n, sc, t1, t2);
    hipLaunchKernelGGL(scan_tiles_kernel, dim3(1), dim3(64), 0, s, t1, t2, nt);
    hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s, sv,
                       n, sc, t1, t2, S1, S2);
    GPIC_TRY(hipGetLastError());
    KmScalars hsc{};
    GPIC_TRY(hipMemcpyAsync(&hsc, sc, sizeof(hsc), hipMemcpyDeviceToHost, s));
    GPIC_TRY(hipStreamSynchronize(s));
    const int64_t distinct = (int64_t)hsc.distinct;
    const int ke = (int)((int64_t)k < distinct ? k : distinct);

    // 3. layers
    hipLaunchKernelGGL(first_layer_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s,
                       S1, S2, n, Da, Q.qlen);
    const int F = (n >= kFLargeFrom) ? kFLarge : kFSmall;
    // levels of the F-ary recursion: until every interval has <= F rows
    int levels = 1;
    for (int64_t m = n; m > F; m /= (F + 1))       // gaps hold <= m / (F+1) rows
        ++levels;
    if (levels > kMaxLevels)
        return hipErrorInvalidValue;               // not reachable for n <= 2^30
    double *Dprev = Da, *Dcur = Db;
    int g = 0;                                     // levels run so far
    for (int c = 1; c < ke; ++c) {
        int32_t *oc = opt + (int64_t)c * n;
        int64_t nodes = 1;
        for (int Lv = 0; Lv < levels; ++Lv, nodes *= (F + 1), ++g) {
            const int64_t items = nodes * F;
            const dim3 grid((unsigned)((items + kThreads - 1) / kThreads));
            if (F == kFSmall)
                hipLaunchKernelGGL(fary_level_kernel<kFSmall>, grid, dim3(kThreads), 0, s,
                                   S1, S2, run, Dprev, Dcur, oc, n, Lv, items, Q, g);
            else
                hipLaunchKernelGGL(fary_level_kernel<kFLarge>, grid, dim3(kThreads), 0, s,
                                   S1, S2, run, Dprev, Dcur, oc, n, Lv, items, Q, g);
            hipLaunchKernelGGL(fary_queue_kernel, dim3(2048), dim3(kThreads), 0, s, S1,
                               S2, run, Dprev, Dcur, oc, Q, g);
            hipLaunchKernelGGL(fary_merge_kernel, dim3(512), dim3(kThreads), 0, s, Dcur,
                               oc, Q, g);
        }
        double *tmp = Dprev; Dprev = Dcur; Dcur = tmp;
    }
    GPIC_TRY(hipGetLastError());

    // 4. boundaries, cluster statistics, labels
    hipLaunchKernelGGL(backtrack_kernel, dim3(1), dim3(64), 0, s, opt, n, ke, first);
    hipLaunchKernelGGL(cluster_stats_kernel, dim3((unsigned)ke), dim3(kThreads), 0, s,
                       sv, first, centroids, costs);
    hipLaunchKernelGGL(labels_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, idxA,
                       n, first, ke, labels);
    GPIC_TRY(hipGetLastError());
    double hc[1024];
    double total = 0.0;
    for (int c0 = 0; c0 < ke; c0 += 1024) {
        const int m = (ke - c0 < 1024) ? ke - c0 : 1024;
        GPIC_TRY(hipMemcpyAsync(hc, costs + c0, m * sizeof(double),
                                hipMemcpyDeviceToHost, s));
        GPIC_TRY(hipStreamSynchronize(s));
        for (int c = 0; c < m; ++c)
            total += hc[c];
    }
    GPIC_TRY(hipStreamSynchronize(s));
    *k_eff = ke;
    if (cost != nullptr)
        *cost = total;
    return hipSuccess;
}

} // namespace gpic
