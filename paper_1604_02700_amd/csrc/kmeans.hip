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
//      values u = v_sorted - mean (stored as (S1, S2) pairs);
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

// Inclusive scan of (x1, x2) over the NT threads of a block (Hillis-Steele
// steps in LDS, a fixed order); a1, a2 must hold NT doubles each.
template <int NT>
__device__ __forceinline__ void block_scan2(double &x1, double &x2, double *a1, double *a2)
{
    const int t = threadIdx.x;
    a1[t] = x1;
    a2[t] = x2;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {
        const double y1 = t >= off ? a1[t - off] : 0.0;
        const double y2 = t >= off ? a2[t - off] : 0.0;
        __syncthreads();
        x1 += y1;
        x2 += y2;
        a1[t] = x1;
        a2[t] = x2;
        __syncthreads();
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
    // the block's total: the last element of the scan of the thread totals
    __shared__ double a1[kThreads], a2[kThreads];
    block_scan2<kThreads>(s1, s2, a1, a2);
    if (threadIdx.x == kThreads - 1) {
        t1[blockIdx.x] = s1;
        t2[blockIdx.x] = s2;
    }
    (void)red;
}

// Exclusive scan of the tile totals by one workgroup: each thread sums a
// contiguous run of tiles, the runs' totals are scanned across the block,
// then each thread walks its run again.
constexpr int kScanThreads = 1024;
__global__ __launch_bounds__(kScanThreads) void scan_tiles_kernel(
    double *__restrict__ t1, double *__restrict__ t2, int64_t nt)
{
    __shared__ double a1[kScanThreads], a2[kScanThreads];
    const int64_t per = (nt + kScanThreads - 1) / kScanThreads;
    const int64_t b0 = (int64_t)threadIdx.x * per;
    const int64_t b1 = (b0 + per < nt) ? b0 + per : nt;
    double x1 = 0.0, x2 = 0.0;
    for (int64_t b = b0; b < b1; ++b) {
        x1 += t1[b];
        x2 += t2[b];
    }
    double i1 = x1, i2 = x2;
    block_scan2<kScanThreads>(i1, i2, a1, a2);
    double r1 = threadIdx.x > 0 ? a1[threadIdx.x - 1] : 0.0;
    double r2 = threadIdx.x > 0 ? a2[threadIdx.x - 1] : 0.0;
    for (int64_t b = b0; b < b1; ++b) {
        const double y1 = t1[b], y2 = t2[b];
        t1[b] = r1;
        t2[b] = r2;
        r1 += y1;
        r2 += y2;
    }
}

// SS[i+1] = (S1[i+1], S2[i+1]) = tile offset + in-tile running sums (each
// thread walks its kItems elements after an exclusive scan of the thread
// totals); the two sums of a position sit together, one 16-byte load.
__global__ __launch_bounds__(kThreads) void prefix_kernel(
    const double *__restrict__ sv, int64_t n, const KmScalars *__restrict__ sc,
    const double *__restrict__ o1, const double *__restrict__ o2,
    double2 *__restrict__ SS)
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
    // exclusive offset of this thread: the tile's offset plus the scan of
    // the earlier threads' totals
    double i1 = s1, i2 = s2;
    block_scan2<kThreads>(i1, i2, a1, a2);
    double r1 = o1[blockIdx.x] + (threadIdx.x > 0 ? a1[threadIdx.x - 1] : 0.0);
    double r2 = o2[blockIdx.x] + (threadIdx.x > 0 ? a2[threadIdx.x - 1] : 0.0);
    for (int it = 0; it < kItems; ++it) {
        const int64_t i = b + it;
        if (i < n) {
            const double u = sv[i] - mu;
            r1 += u;
            r2 += u * u;
            SS[i + 1] = double2{r1, r2};
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0)
        SS[0] = double2{0.0, 0.0};
}

// cost(j, i) from the prefix sums at j and i + 1
__device__ __forceinline__ double seg_cost(double2 a, double2 e, int64_t j, int64_t i)
{
    const double m = (double)(i - j + 1);
    const double s1 = e.x - a.x;
    const double s2 = e.y - a.y;
    const double c = s2 - s1 * s1 / m;
    return c > 0.0 ? c : 0.0;
}

// A layer's values as its successor reads them: E[j] = D(j - 1) where j
// starts a run of equal values, +infinity where it does not (a split there
// would separate equal values), so a candidate needs no separate flag.
__device__ __forceinline__ void store_next(double *__restrict__ E,
                                           const int32_t *__restrict__ run, int64_t n,
                                           int64_t r, double d)
{
    if (r + 1 < n)
        E[r + 1] = run[r + 1] ? d : INFINITY;
}

__global__ __launch_bounds__(kThreads) void first_layer_kernel(
    const double2 *__restrict__ SS, const int32_t *__restrict__ run, int64_t n,
    double *__restrict__ E, unsigned long long *__restrict__ qlen)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n)
        store_next(E, run, n, i, seg_cost(SS[0], SS[i + 1], 0, i));
    if (i < 4)
        qlen[i] = 0ull;                 // the recursion's part and row counters
}

// ---------------------------------------------------------------- layers
//
// Each layer is solved by F-ary divide and conquer: an interval of rows
// [lo, hi] whose neighbours' optimal split points are known takes F evenly
// spaced sample rows (all its rows if it has at most F) and computes their
// leftmost argmins in parallel, over the interval's bounds
// [opt(lo-1), opt(hi+1)] (and j <= r for row r); the F+1 gaps between
// samples are the next level's intervals.  ceil(log_{F+1} n) levels replace
// the log2 n of a binary split, which matters because every level is a
// dependent step.  F = 64 up to 2^18 rows, F = 8 above.
//
// All samples of an interval share its candidates, so an interval whose
// range is long is queued as parts of candidates, and one wave per (part,
// group of samples) reads each candidate once and evaluates it for the
// group's samples; short ranges are scanned by a thread per sample.  The
// recursion's shape (which rows are the samples of which interval at which
// level) depends on n and F only and is laid out once per call as per-level
// row lists.  Sample rows use 32-bit arithmetic (n <= 2^30).
constexpr int kFSmall = 64;
constexpr int kFLarge = 8;
constexpr int64_t kFLargeFrom = (int64_t)1 << 18;
constexpr int kMaxLevels = 16;
constexpr int kShortScan = 64;        // longer ranges go to the work queue
// candidates per queued part and samples evaluated per pass over it: two
// samples per wave keep four times as many waves in flight as one wave
// for all eight, which the long, few parts of the first levels need
// (measured, n = 2M, k = 50: groups of 8, 4, 2, 1 samples: 22.5, 20.4,
// 19.8, 22.2 ms; parts of 512 or 2,048 candidates: slower); for F = 64
// (n = 50,000, k = 10: 0.98 ms against 1.35 ms with the F = 8 setting of
// that time)
template <int F> constexpr int chunk_for() { return F == kFLarge ? 1024 : 512; }
template <int F> constexpr int group_for() { return 2; }
constexpr int kMinChunk = 512;

// Sample f of interval [lo, hi] (m = hi - lo + 1 rows): every row if m <= F,
// else lo + (f + 1)(m + 1) / (F + 1) - 1 (evaluated as (f + 1) a +
// (f + 1) b / (F + 1) with m + 1 = (F + 1) a + b); -1 if there is none.
template <int F>
__host__ __device__ __forceinline__ int32_t sample_row(int32_t lo, int32_t hi, int f)
{
    const uint32_t m = (uint32_t)(hi - lo + 1);
    if (m <= (uint32_t)F)
        return (f < (int)m) ? lo + f : -1;
    const uint32_t a = (m + 1) / (F + 1), b = (m + 1) % (F + 1);
    const uint32_t f1 = (uint32_t)(f + 1);
    return lo + (int32_t)(f1 * a + (f1 * b) / (F + 1)) - 1;
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

// Scan split points j = from .. ahi for row r, keeping the leftmost
// minimum of D(j - 1) + cost(j, r) over run starts (E[j] is +infinity
// elsewhere, and so is the sum).  Every candidate is evaluated without
// branching so successive loads overlap.
__device__ __forceinline__ void scan_range(const double2 *__restrict__ SS,
                                           const double *__restrict__ Ep, int64_t r,
                                           int64_t from, int64_t ahi, double &best,
                                           int64_t &arg)
{
    const double2 e = SS[r + 1];
#pragma unroll 4
    for (int64_t j = from; j <= ahi; ++j) {
        const double c = Ep[j] + seg_cost(SS[j], e, j, r);
        if (c < best) {
            best = c;
            arg = j;
        }
    }
}

// The value of lane (lane xor K): data-parallel moves for K = 1, 2, 8
// (quad permutations, a rotation by 8 within a row of 16), swizzles for
// K = 4, 16, a permute for K = 32.
template <int K>
__device__ __forceinline__ int lane_xor(int x)
{
    if (K == 1)
        return __builtin_amdgcn_mov_dpp(x, 0xb1, 0xf, 0xf, false);
    if (K == 2)
        return __builtin_amdgcn_mov_dpp(x, 0x4e, 0xf, 0xf, false);
    if (K == 4)
        return __builtin_amdgcn_ds_swizzle(x, 0x101f);
    if (K == 8)
        return __builtin_amdgcn_mov_dpp(x, 0x128, 0xf, 0xf, false);
    if (K == 16)
        return __builtin_amdgcn_ds_swizzle(x, 0x401f);
    return __shfl_xor(x, 32, kWave);
}

template <int K>
__device__ __forceinline__ void argmin_step(double &best, int32_t &arg)
{
    const long long bb = __double_as_longlong(best);
    const int lo = lane_xor<K>((int)(bb & 0xffffffffll));
    const int hi = lane_xor<K>((int)(bb >> 32));
    const double ob = __longlong_as_double(((long long)(unsigned)hi << 32) |
                                           (long long)(unsigned)lo);
    const int32_t oa = lane_xor<K>(arg);
    if (ob < best || (ob == best && oa < arg)) {
        best = ob;
        arg = oa;
    }
}

// Leftmost minimum of (value, index) over the wave, in every lane (an
// index of INT64_MAX, no candidate, travels as INT32_MAX).
__device__ __forceinline__ void wave_argmin(double &best, int64_t &arg)
{
    int32_t a = (arg == INT64_MAX) ? INT32_MAX : (int32_t)arg;
    argmin_step<32>(best, a);
    argmin_step<16>(best, a);
    argmin_step<8>(best, a);
    argmin_step<4>(best, a);
    argmin_step<2>(best, a);
    argmin_step<1>(best, a);
    arg = (a == INT32_MAX) ? INT64_MAX : (int64_t)a;
}

// Candidate bounds of interval [lo, hi]: [alo, ohi]; row r takes j <= r.
__device__ __forceinline__ void interval_bounds(const int32_t *__restrict__ opt, int32_t n,
                                                int32_t lo, int32_t hi, int32_t &alo,
                                                int32_t &ohi)
{
    const int32_t olo = (lo > 0) ? opt[lo - 1] : 1;
    ohi = (hi < n - 1) ? opt[hi + 1] : n - 1;
    alo = olo < 1 ? 1 : olo;
}

__device__ __forceinline__ void store_result(double *__restrict__ Ec,
                                             const int32_t *__restrict__ run, int64_t n,
                                             int32_t *__restrict__ opt, int64_t r,
                                             double best, int64_t arg, int64_t alo)
{
    store_next(Ec, run, n, r, best);
    opt[r] = (int32_t)((arg == INT64_MAX) ? alo : arg);
}

// A queued part: candidates [plo, phi] of interval [lo, hi] with bounds
// [alo, ohi]; head is the slot of the interval's first part (its part count
// lives there).  lo < 0 marks a slot that holds no work.
struct QueuePart {
    int32_t lo, hi, plo, phi, alo, ohi, head, pad;
};

struct LevelQueue {
    QueuePart *part;
    int32_t *nparts;                     // indexed by head
    int32_t *heads;                      // heads of intervals with more than one part
    double *pbest;                       // per part and sample: [e * F + f]
    int32_t *parg;
    unsigned long long *qlen;            // parts: [g & 1]; intervals: [2 + (g & 1)]
    int64_t cap;
};

// Number of samples of interval [lo, hi] (m > F rows) at or before row r:
// sample f sits at lo - 1 + floor((f + 1)(m + 1) / (F + 1)), so the count
// is the largest c <= F with floor(c (m + 1) / (F + 1)) <= r - lo + 1;
// a float64 estimate is corrected against the exact sample rows.
template <int F>
__device__ __forceinline__ int samples_upto(int32_t lo, int32_t hi, int32_t r)
{
    const double x = (double)(r - lo + 1), m1 = (double)(hi - lo + 2);
    int c = (int)((x + 1.0) * (double)(F + 1) / m1) - 1;
    c = c < 0 ? 0 : (c > F ? F : c);
    while (c < F && sample_row<F>(lo, hi, c) <= r)
        ++c;
    while (c > 0 && sample_row<F>(lo, hi, c - 1) > r)
        --c;
    return c;
}

// The recursion's shape does not depend on the values: which rows are the
// samples of which level, and the interval each belongs to, follow from n
// and F alone.  It is laid out once per call as one list per level of
// (row, interval, last sample row of the interval, first-sample flag) in
// ascending row order, so each layer's level kernels read a row's interval
// instead of deriving it.
struct RowEntry {
    int32_t r, lo, hi, rl;               // rl: last sample row; bit 31: first sample
};
constexpr int32_t kFirstSample = (int32_t)0x80000000;

// A thread per row: the level at which the row is a sample and its entry
// (the row descends the recursion, gap by gap, until it is a sample), and
// its rank among the rows of its block at that level.
template <int F>
__global__ __launch_bounds__(kThreads) void row_level_kernel(
    int32_t n, int levels, RowEntry *__restrict__ ent, int32_t *__restrict__ lr,
    int32_t *__restrict__ bh)
{
    __shared__ int32_t wl[kThreads / kWave][kMaxLevels];
    const int64_t item = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int32_t r = (int32_t)(item < n ? item : -1);
    int lev = -1;
    RowEntry e{r, 0, n - 1, 0};
    if (r >= 0) {
        int32_t lo = 0, hi = n - 1;
        for (int l = 0; l < levels; ++l) {
            if (hi - lo + 1 <= F) {
                lev = l;                                     // every row a sample
                e = RowEntry{r, lo, hi, hi | (r == lo ? kFirstSample : 0)};
                break;
            }
            const int c = samples_upto<F>(lo, hi, r);
            if (c > 0 && sample_row<F>(lo, hi, c - 1) == r) {
                lev = l;
                const int32_t rl = sample_row<F>(lo, hi, F - 1);
                e = RowEntry{r, lo, hi, rl | (c == 1 ? kFirstSample : 0)};
                break;
            }
            const int32_t nlo = (c == 0) ? lo : sample_row<F>(lo, hi, c - 1) + 1;
            const int32_t nhi = (c == F) ? hi : sample_row<F>(lo, hi, c) - 1;
            lo = nlo;
            hi = nhi;
        }
    }
    // rank within the block among rows of the same level (ballots per level)
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    int rank = 0;
    for (int l = 0; l < levels; ++l) {
        const unsigned long long m = __ballot(lev == l);
        if (lev == l)
            rank = __popcll(m & below);
        if (lane == 0)
            wl[w][l] = __popcll(m);
    }
    __syncthreads();
    if (lev >= 0) {
        for (int u = 0; u < w; ++u)
            rank += wl[u][lev];
        ent[r] = e;
        lr[r] = (lev << 24) | rank;                          // rank < 256
    } else if (r >= 0) {
        lr[r] = -1;                                          // not reached for n <= 2^30
    }
    if (threadIdx.x < levels) {
        int32_t t = 0;
        for (int u = 0; u < kThreads / kWave; ++u)
            t += wl[u][threadIdx.x];
        bh[(int64_t)blockIdx.x * kMaxLevels + threadIdx.x] = t;
    }
}

// One workgroup: per level, exclusive scan of the block counts, plus the
// level's base (the levels' lists are stored one after another); base[l]
// for l <= levels.
__global__ __launch_bounds__(1024) void level_scan_kernel(
    int32_t *__restrict__ bh, int64_t nb, int levels, int32_t *__restrict__ base)
{
    __shared__ int32_t ts[1024];
    __shared__ int32_t tot[kMaxLevels + 1];
    const int64_t per = (nb + 1023) / 1024;
    const int64_t b0 = (int64_t)threadIdx.x * per;
    for (int l = 0; l < levels; ++l) {
        int32_t t = 0;
        for (int64_t b = b0; b < b0 + per && b < nb; ++b)
            t += bh[b * kMaxLevels + l];
        ts[threadIdx.x] = t;
        __syncthreads();
        if (threadIdx.x == 0) {
            int32_t run = 0;
            for (int u = 0; u < 1024; ++u) {
                const int32_t x = ts[u];
                ts[u] = run;
                run += x;
            }
            tot[l] = run;
        }
        __syncthreads();
        int32_t run = ts[threadIdx.x];
        for (int64_t b = b0; b < b0 + per && b < nb; ++b) {
            const int32_t x = bh[b * kMaxLevels + l];
            bh[b * kMaxLevels + l] = run;
            run += x;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        int32_t run = 0;
        for (int l = 0; l < levels; ++l) {
            base[l] = run;
            run += tot[l];
        }
        base[levels] = run;
    }
}

__global__ __launch_bounds__(kThreads) void level_scatter_kernel(
    int32_t n, const RowEntry *__restrict__ ent, const int32_t *__restrict__ lr,
    const int32_t *__restrict__ bh, const int32_t *__restrict__ base,
    RowEntry *__restrict__ list)
{
    const int64_t r = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (r >= n)
        return;
    const int32_t x = lr[r];
    if (x < 0)
        return;
    const int l = x >> 24;
    const int64_t pos = (int64_t)base[l] + bh[(int64_t)blockIdx.x * kMaxLevels + l] +
                        (x & 0xffffff);
    if (pos < n)
        list[pos] = ent[r];
}

// One level of a layer, a thread per sample row of the level (in row
// order).  A node whose range is at most kShortScan long has each sample
// scan its own row; a longer one is queued by its first sample, and its
// other samples leave it to the queue; if the queue has no room the first
// sample scans every sample row of the node itself.  Item 0 clears the
// other pair of counters, whose level has finished.
template <int F>
__global__ __launch_bounds__(kThreads) void fary_rows_kernel(
    const double2 *__restrict__ SS, const int32_t *__restrict__ run,
    const double *__restrict__ Ep, double *__restrict__ Ec, int32_t *__restrict__ opt,
    int32_t n, const RowEntry *__restrict__ list, const int32_t *__restrict__ base, int L,
    LevelQueue Q, int g)
{
    const int64_t item = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (item == 0) {
        Q.qlen[(g + 1) & 1] = 0ull;
        Q.qlen[2 + ((g + 1) & 1)] = 0ull;
    }
    const int64_t b0 = base[L];
    const int64_t cnt = ((int64_t)base[L + 1] < n ? (int64_t)base[L + 1] : n) - b0;
    const bool has = item < cnt;
    int32_t r = -1, lo = 0, hi = -1, rl = 0, alo = 1, ohi = 0;
    bool first = false;
    int64_t len = 0;
    if (has) {
        const RowEntry e = list[b0 + item];
        r = e.r;
        lo = e.lo;
        hi = e.hi;
        first = (e.rl & kFirstSample) != 0;
        rl = e.rl & ~kFirstSample;
        interval_bounds(opt, n, lo, hi, alo, ohi);
        len = (int64_t)(ohi < rl ? ohi : rl) - alo + 1;
    }
    const bool lead = has && first && len > kShortScan;
    int64_t e0 = 0, C = 0;
    int ok = 0;
    if (lead) {
        C = (len + chunk_for<F>() - 1) / chunk_for<F>();
        e0 = (int64_t)atomicAdd(&Q.qlen[g & 1], (unsigned long long)C);
        ok = e0 + C <= Q.cap;
        if (ok) {
            Q.nparts[e0] = (int32_t)C;
            if (C > 1) {
                const unsigned long long h = atomicAdd(&Q.qlen[2 + (g & 1)], 1ull);
                Q.heads[h] = (int32_t)e0;             // h < e0 + 1 <= cap
            }
        } else {
            // no room left (only if split points were far from monotone):
            // void the reserved slots below the capacity
            for (int64_t e = e0; e < e0 + C && e < Q.cap; ++e)
                Q.part[e] = QueuePart{-1, 0, 0, -1, 0, 0, 0, 0};
        }
    }
    const int lane = threadIdx.x % kWave;
    const int32_t aend = alo + (int32_t)len - 1;    // end of the longest sample range
    if (ok && C <= kWave) {
        for (int64_t p = 0; p < C; ++p) {
            const int32_t plo = alo + (int32_t)(p * chunk_for<F>());
            const int32_t phi = plo + chunk_for<F>() - 1 < aend ? plo + chunk_for<F>() - 1 : aend;
            Q.part[e0 + p] = QueuePart{lo, hi, plo, phi, alo, ohi, (int32_t)e0, 0};
        }
    }
    unsigned long long mask = __ballot(ok && C > kWave);
    while (mask) {
        const int src = __ffsll((long long)mask) - 1;
        mask &= mask - 1;
        const long long qe0 = __shfl((long long)e0, src, kWave);
        const long long qC = __shfl((long long)C, src, kWave);
        const int qlo = __shfl(lo, src, kWave), qhi = __shfl(hi, src, kWave);
        const int qalo = __shfl(alo, src, kWave), qohi = __shfl(ohi, src, kWave);
        const int qend = __shfl(aend, src, kWave);
        for (long long p = lane; p < qC; p += kWave) {
            const int32_t plo = qalo + (int32_t)(p * chunk_for<F>());
            const int32_t phi = plo + chunk_for<F>() - 1 < qend ? plo + chunk_for<F>() - 1 : qend;
            Q.part[qe0 + p] = QueuePart{qlo, qhi, plo, phi, qalo, qohi, (int32_t)qe0, 0};
        }
    }
    if (!has)
        return;
    if (len <= kShortScan) {
        double best = INFINITY;
        int64_t arg = INT64_MAX;
        scan_range(SS, Ep, r, alo, ohi < r ? ohi : r, best, arg);
        store_result(Ec, run, n, opt, r, best, arg, alo);
    } else if (lead && !ok) {
        const int ns = (hi - lo + 1 < F) ? hi - lo + 1 : F;
        for (int f = 0; f < ns; ++f) {
            const int32_t q = sample_row<F>(lo, hi, f);
            double best = INFINITY;
            int64_t arg = INT64_MAX;
            scan_range(SS, Ep, q, alo, ohi < q ? ohi : q, best, arg);
            store_result(Ec, run, n, opt, q, best, arg, alo);
        }
    }
}

// The level's queued parts: a wave per (part, group of kGroup samples);
// its lanes read each candidate of the part once and evaluate it for the
// group's samples (candidate j counts for row r if j <= r and j <= ohi).  An interval with one part is finished here; otherwise
// the part leaves each sample's minimum for fary_merge_kernel.
template <int F>
__global__ __launch_bounds__(kThreads) void fary_queue_kernel(
    const double2 *__restrict__ SS, const int32_t *__restrict__ run,
    const double *__restrict__ Ep, double *__restrict__ Ec, int32_t *__restrict__ opt,
    int32_t n, LevelQueue Q, int g)
{
    constexpr int kGroup = group_for<F>();
    constexpr int kGroups = (F + kGroup - 1) / kGroup;
    const int64_t total = (int64_t)Q.qlen[g & 1];
    const int64_t len = total < Q.cap ? total : Q.cap;
    const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
    const int lane = threadIdx.x % kWave;
    // work item t: part t / kGroups, samples kGroup (t % kGroups) ..
    for (int64_t t = (int64_t)blockIdx.x * (kThreads / kWave) + threadIdx.x / kWave;
         t < len * kGroups; t += waves) {
        const int64_t e = t / kGroups;
        const QueuePart q = Q.part[e];
        if (q.lo < 0)
            continue;                                   // uniform per wave
        const int m = q.hi - q.lo + 1;
        const int ns = m < F ? m : F;
        const bool single = Q.nparts[q.head] == 1;
        const int g0 = (int)(t % kGroups) * kGroup;
        if (g0 < ns) {
            int64_t rr[kGroup], lim[kGroup];
            double s1e[kGroup], s2e[kGroup], best[kGroup];
            int64_t arg[kGroup];
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                rr[u] = (g0 + u < ns) ? (int64_t)sample_row<F>(q.lo, q.hi, g0 + u) : -1;
                lim[u] = (rr[u] < q.ohi) ? rr[u] : q.ohi;
                const double2 e = (rr[u] >= 0) ? SS[rr[u] + 1] : double2{0.0, 0.0};
                s1e[u] = e.x;
                s2e[u] = e.y;
                best[u] = INFINITY;
                arg[u] = INT64_MAX;
            }
            for (int64_t j = (int64_t)q.plo + lane; j <= q.phi; j += kWave) {
                const double dp = Ep[j];
                const double2 a = SS[j];
                const double a1 = a.x, a2 = a.y;
#pragma unroll
                for (int u = 0; u < kGroup; ++u) {
                    // seg_cost(SS[j], SS[rr[u] + 1], j, rr[u]), term by term
                    const double mm = (double)(rr[u] - j + 1);
                    const double s1 = s1e[u] - a1;
                    const double s2 = s2e[u] - a2;
                    const double c0 = s2 - s1 * s1 / mm;
                    const double c = dp + (c0 > 0.0 ? c0 : 0.0);
                    if (j <= lim[u] && c < best[u]) {
                        best[u] = c;
                        arg[u] = j;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kGroup; ++u) {
                if (g0 + u >= ns)
                    break;                                  // uniform per wave
                wave_argmin(best[u], arg[u]);
                if (lane == 0) {
                    if (single) {
                        store_result(Ec, run, n, opt, rr[u], best[u], arg[u], q.alo);
                    } else {
                        Q.pbest[e * F + g0 + u] = best[u];
                        Q.parg[e * F + g0 + u] =
                            (arg[u] == INT64_MAX) ? INT32_MAX : (int32_t)arg[u];
                    }
                }
            }
        }
    }
}

// Intervals with several parts: the parts' minima of each (interval,
// sample) merged in an order-independent leftmost minimum, by a wave, or
// by a whole workgroup at the first levels (few intervals with thousands
// of parts each; `whole` is uniform over the launch).
template <int F>
__global__ __launch_bounds__(kThreads) void fary_merge_kernel(
    double *__restrict__ Ec, const int32_t *__restrict__ run, int32_t n,
    int32_t *__restrict__ opt, LevelQueue Q, int g, int whole)
{
    __shared__ double wb[kThreads / kWave];
    __shared__ int64_t wa[kThreads / kWave];
    const int64_t nh = (int64_t)Q.qlen[2 + (g & 1)];
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    const int64_t t0 = whole ? (int64_t)blockIdx.x
                             : (int64_t)blockIdx.x * (kThreads / kWave) + w;
    const int64_t step = whole ? (int64_t)gridDim.x : (int64_t)gridDim.x * (kThreads / kWave);
    const int p0 = whole ? (int)threadIdx.x : lane;
    const int pstep = whole ? kThreads : kWave;
    // work item t: interval t / F, sample t % F
    for (int64_t t = t0; t < nh * F; t += step) {
        const int64_t head = Q.heads[t / F];
        const int f = (int)(t % F);
        const QueuePart q = Q.part[head];
        const int C = Q.nparts[head];
        const int m = q.hi - q.lo + 1;
        const int ns = m < F ? m : F;
        if (f >= ns)
            continue;                                   // uniform per item
        double best = INFINITY;
        int64_t arg = INT64_MAX;
        for (int p = p0; p < C; p += pstep) {
            const int32_t a = Q.parg[(head + p) * F + f];
            amin_merge(best, arg, Q.pbest[(head + p) * F + f],
                       a == INT32_MAX ? INT64_MAX : (int64_t)a);
        }
        wave_argmin(best, arg);
        if (whole) {
            if (lane == 0) {
                wb[w] = best;
                wa[w] = arg;
            }
            __syncthreads();
            if (threadIdx.x == 0)
                for (int u = 1; u < kThreads / kWave; ++u)
                    amin_merge(best, arg, wb[u], wa[u]);
            __syncthreads();
        }
        if (threadIdx.x % (whole ? kThreads : kWave) == 0)
            store_result(Ec, run, n, opt, sample_row<F>(q.lo, q.hi, f), best, arg, q.alo);
    }
}

// The last layer: the backtrack reads its split point at row n - 1 only,
// so that row's leftmost argmin over every candidate j in [1, n - 1] is
// found by one scan instead of the layer's recursion (the same candidates,
// cost expression and tie rule as a row's own scan).  Workgroup b scans a
// contiguous chunk (each lane in ascending j, strict improvement), leaving
// its leftmost minimum in pbest[b], parg[b].
constexpr int kLastBlocks = 256;
__global__ __launch_bounds__(kThreads) void last_row_kernel(
    const double2 *__restrict__ SS, const double *__restrict__ Ep, int64_t n,
    double *__restrict__ pbest, int32_t *__restrict__ parg)
{
    __shared__ double wb[kThreads / kWave];
    __shared__ int64_t wa[kThreads / kWave];
    const int64_t r = n - 1;
    const double2 e = SS[r + 1];
    const int64_t per = (n - 1 + gridDim.x - 1) / gridDim.x;
    const int64_t j0 = 1 + (int64_t)blockIdx.x * per;
    const int64_t j1 = (j0 + per - 1 < r) ? j0 + per - 1 : r;
    double best = INFINITY;
    int64_t arg = INT64_MAX;
    for (int64_t j = j0 + threadIdx.x; j <= j1; j += kThreads) {
        const double c = Ep[j] + seg_cost(SS[j], e, j, r);
        if (c < best) {
            best = c;
            arg = j;
        }
    }
    wave_argmin(best, arg);
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    if (lane == 0) {
        wb[w] = best;
        wa[w] = arg;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int u = 1; u < kThreads / kWave; ++u)
            amin_merge(best, arg, wb[u], wa[u]);
        pbest[blockIdx.x] = best;
        parg[blockIdx.x] = (arg == INT64_MAX) ? INT32_MAX : (int32_t)arg;
    }
}

// The chunks' minima merged (order-independent leftmost minimum) into the
// last layer's split point at row n - 1.
__global__ __launch_bounds__(kWave) void last_row_merge_kernel(
    const double *__restrict__ pbest, const int32_t *__restrict__ parg, int nb, int64_t n,
    int32_t *__restrict__ opt)
{
    double best = INFINITY;
    int64_t arg = INT64_MAX;
    for (int b = threadIdx.x; b < nb; b += kWave)
        amin_merge(best, arg, pbest[b], parg[b] == INT32_MAX ? INT64_MAX : (int64_t)parg[b]);
    wave_argmin(best, arg);
    if (threadIdx.x == 0)
        opt[n - 1] = (int32_t)((arg == INT64_MAX) ? 1 : arg);
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
constexpr int kStatThreads = 1024;
__global__ __launch_bounds__(kStatThreads) void cluster_stats_kernel(
    const double *__restrict__ sv, const int64_t *__restrict__ first,
    double *__restrict__ centroids, double *__restrict__ costs)
{
    __shared__ double red[kStatThreads / kWave];
    const int c = blockIdx.x;
    const int64_t b = first[c], e = first[c + 1];
    double s = 0.0;
#pragma unroll 4
    for (int64_t p = b + threadIdx.x; p < e; p += kStatThreads)
        s += sv[p];
    const double mu = block_sum<kStatThreads>(s, red) / (double)(e - b);
    double q = 0.0;
#pragma unroll 4
    for (int64_t p = b + threadIdx.x; p < e; p += kStatThreads)
        q += (sv[p] - mu) * (sv[p] - mu);
    const double tq = block_sum<kStatThreads>(q, red);
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

unsigned blocks_for(int64_t n) { return (unsigned)((n + kThreads - 1) / kThreads); }

struct KmLayout {
    size_t keyA, keyB, idxA, idxB, hist, hsum, sv, run, t1, t2, SS, Ea, Eb, opt,
        qpart, qnparts, qheads, qbest, qarg, qlen, sc, first, costs, ent, lr, bh, lbase,
        list, total;
};

// Queue slots per level.  With monotone split points the interval ranges
// of one level overlap only at their ends (at most 2n candidates in all)
// and a queued range is longer than kShortScan, so a level holds at most
// 2n / kShortScan intervals and 2n / kMinChunk + 2n / kShortScan parts; a
// level that would need more scans the excess in place.
int64_t queue_cap(int64_t n) { return 2 * n / kShortScan + 2 * n / kMinChunk + 1024; }
int fary_f(int64_t n) { return (n >= kFLargeFrom) ? kFLarge : kFSmall; }

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
    L.SS = take((n + 1) * 16);
    L.Ea = take(n * 8);
    L.Eb = take(n * 8);
    L.opt = take((size_t)k * n * 4);
    const size_t cap = (size_t)queue_cap(n);
    L.qpart = take(cap * sizeof(QueuePart));
    L.qnparts = take(cap * 4);
    L.qheads = take(cap * 4);
    L.qbest = take(cap * fary_f(n) * 8);
    L.qarg = take(cap * fary_f(n) * 4);
    L.qlen = take(4 * 8);
    L.sc = take(sizeof(KmScalars));
    L.first = take((size_t)(k + 1) * 8);
    L.costs = take((size_t)k * 8);
    L.ent = take(n * sizeof(RowEntry));
    L.lr = take(n * 4);
    L.bh = take((size_t)blocks_for(n) * kMaxLevels * 4);
    L.lbase = take((kMaxLevels + 1) * 4);
    L.list = take(n * sizeof(RowEntry));
    L.total = o;
    return L;
}

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
    double2 *SS = (double2 *)(w + L.SS);
    double *Ea = (double *)(w + L.Ea), *Eb = (double *)(w + L.Eb);
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
    hipLaunchKernelGGL(scan_tiles_kernel, dim3(1), dim3(kScanThreads), 0, s, t1, t2, nt);
    hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)nt), dim3(kThreads), 0, s, sv,
                       n, sc, t1, t2, SS);
    GPIC_TRY(hipGetLastError());
    KmScalars hsc{};
    GPIC_TRY(hipMemcpyAsync(&hsc, sc, sizeof(hsc), hipMemcpyDeviceToHost, s));
    GPIC_TRY(hipStreamSynchronize(s));
    const int64_t distinct = (int64_t)hsc.distinct;
    const int ke = (int)((int64_t)k < distinct ? k : distinct);

    // 3. layers
    hipLaunchKernelGGL(first_layer_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s,
                       SS, run, n, Ea, Q.qlen);
    const int F = fary_f(n);
    // levels of the F-ary recursion: until every interval has <= F rows
    int levels = 1;
    for (int64_t m = n; m > F; m /= (F + 1))       // gaps hold <= m / (F+1) rows
        ++levels;
    if (levels > kMaxLevels)
        return hipErrorInvalidValue;               // not reachable for n <= 2^30
    double *Ep = Ea, *Ec = Eb;
    if (ke > 1) {
        // samples per level, from the interval sizes alone (each level's
        // intervals take at most a few distinct sizes)
        int64_t count[kMaxLevels] = {};
        {
            int64_t sz[64], mult[64];
            int ns = 1;
            sz[0] = n;
            mult[0] = 1;
            int64_t total = 0;
            for (int Lv = 0; Lv < levels; ++Lv) {
                int64_t nsz[64], nmult[64];
                int nn = 0;
                auto add = [&](int64_t m, int64_t c) {
                    if (m <= 0)
                        return true;
                    for (int u = 0; u < nn; ++u)
                        if (nsz[u] == m) {
                            nmult[u] += c;
                            return true;
                        }
                    if (nn == 64)
                        return false;
                    nsz[nn] = m;
                    nmult[nn++] = c;
                    return true;
                };
                for (int u = 0; u < ns; ++u) {
                    const int64_t m = sz[u], c = mult[u];
                    if (m <= F) {
                        count[Lv] += m * c;
                        continue;
                    }
                    count[Lv] += (int64_t)F * c;
                    int32_t prev = -1;
                    for (int f = 0; f <= F; ++f) {
                        const int32_t sr = (f < F)
                            ? (F == kFSmall ? sample_row<kFSmall>(0, (int32_t)m - 1, f)
                                            : sample_row<kFLarge>(0, (int32_t)m - 1, f))
                            : (int32_t)m;
                        if (!add(sr - prev - 1, c))
                            return hipErrorInvalidValue;
                        prev = sr;
                    }
                }
                total += count[Lv];
                ns = nn;
                for (int u = 0; u < nn; ++u) {
                    sz[u] = nsz[u];
                    mult[u] = nmult[u];
                }
            }
            if (total != n || ns != 0)
                return hipErrorInvalidValue;       // the recursion does not cover every row
        }
        RowEntry *ent = (RowEntry *)(w + L.ent), *list = (RowEntry *)(w + L.list);
        int32_t *lr = (int32_t *)(w + L.lr), *bh = (int32_t *)(w + L.bh);
        int32_t *lbase = (int32_t *)(w + L.lbase);
        if (F == kFSmall)
            hipLaunchKernelGGL(row_level_kernel<kFSmall>, dim3(blocks_for(n)), dim3(kThreads),
                               0, s, (int32_t)n, levels, ent, lr, bh);
        else
            hipLaunchKernelGGL(row_level_kernel<kFLarge>, dim3(blocks_for(n)), dim3(kThreads),
                               0, s, (int32_t)n, levels, ent, lr, bh);
        hipLaunchKernelGGL(level_scan_kernel, dim3(1), dim3(1024), 0, s, bh,
                           (int64_t)blocks_for(n), levels, lbase);
        hipLaunchKernelGGL(level_scatter_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s,
                           (int32_t)n, ent, lr, bh, lbase, list);
        int g = 0;                                 // levels run so far
        for (int c = 1; c < ke; ++c) {
            int32_t *oc = opt + (int64_t)c * n;
            if (c == ke - 1) {
                // only row n - 1 of the last layer is read
                const int64_t want = (n - 1 + kThreads - 1) / kThreads;
                const int nbl = (int)(want < kLastBlocks ? want : kLastBlocks);
                hipLaunchKernelGGL(last_row_kernel, dim3(nbl), dim3(kThreads), 0, s, SS, Ep,
                                   n, Q.pbest, Q.parg);
                hipLaunchKernelGGL(last_row_merge_kernel, dim3(1), dim3(kWave), 0, s,
                                   (const double *)Q.pbest, (const int32_t *)Q.parg, nbl, n,
                                   oc);
                break;
            }
            for (int Lv = 0; Lv < levels; ++Lv, ++g) {
                const dim3 grid(blocks_for(count[Lv] > 0 ? count[Lv] : 1));
                const int whole = count[Lv] <= 512;    // few intervals, many parts each
                if (F == kFSmall) {
                    hipLaunchKernelGGL(fary_rows_kernel<kFSmall>, grid, dim3(kThreads), 0, s,
                                       SS, run, Ep, Ec, oc, (int32_t)n, list, lbase,
                                       Lv, Q, g);
                    hipLaunchKernelGGL(fary_queue_kernel<kFSmall>, dim3(2048), dim3(kThreads),
                                       0, s, SS, run, Ep, Ec, oc, (int32_t)n, Q, g);
                    hipLaunchKernelGGL(fary_merge_kernel<kFSmall>, dim3(512), dim3(kThreads),
                                       0, s, Ec, run, (int32_t)n, oc, Q, g, whole);
                } else {
                    hipLaunchKernelGGL(fary_rows_kernel<kFLarge>, grid, dim3(kThreads), 0, s,
                                       SS, run, Ep, Ec, oc, (int32_t)n, list, lbase,
                                       Lv, Q, g);
                    hipLaunchKernelGGL(fary_queue_kernel<kFLarge>, dim3(2048), dim3(kThreads),
                                       0, s, SS, run, Ep, Ec, oc, (int32_t)n, Q, g);
                    hipLaunchKernelGGL(fary_merge_kernel<kFLarge>, dim3(512), dim3(kThreads),
                                       0, s, Ec, run, (int32_t)n, oc, Q, g, whole);
                }
            }
            double *tmp = Ep; Ep = Ec; Ec = tmp;
        }
    }
    GPIC_TRY(hipGetLastError());

    // 4. boundaries, cluster statistics, labels
    hipLaunchKernelGGL(backtrack_kernel, dim3(1), dim3(64), 0, s, opt, n, ke, first);
    hipLaunchKernelGGL(cluster_stats_kernel, dim3((unsigned)ke), dim3(kStatThreads), 0, s,
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
