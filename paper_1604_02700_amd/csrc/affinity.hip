// Gaussian affinity tiles for gfx950, the fused operator built on them, and
// the cosine affinity of the paper's Experiment I.
//
// A_ij = exp(-||x_i - x_j||^2 / (2 sigma^2)) for i != j, A_ii = 0: the
// affinity matrix of section "Spectral Cluster" (AffinityMatrix step of
// Algorithm 2) with the Gaussian kernel read in for it.  The exponential is
// evaluated as exp2(-c * dist2) with c = log2(e) / (2 sigma^2), formed in
// float64 on the host and rounded once to float32.
//
// Two tile engines:
//   * MFMA, 16 <= d <= 128.  Squared distances in the Gram form
//     |x_i|^2 + |x_j|^2 - 2 x_i.x_j over the centred points x - centre
//     (a per-coordinate median of a sample; distances are unchanged, and
//     the cancellation then scales with the spread of the points, not
//     their offset from the origin), with the dot
//     products on the fp16 matrix cores: every point, scaled by its own
//     power of two into [-1, 1], has each coordinate split into a
//     half-precision high part and the half-precision remainder, and three
//     products per pair of parts (hi.hi, lo.hi, hi.lo, float32
//     accumulation) reproduce the float32 dot product to about 2^-22 of
//     |x_i||x_j| per coordinate, at about a fifth of the fp32 matrix-core
//     time.  With a median centre and a scale per point, a point far from
//     the others coarsens only its own rows and columns.  A prologue (the
//     centre, then the split)
//     writes the operands once per call in the order the matrix cores take
//     them, so a column tile is staged into LDS by contiguous 16-byte
//     copies and every operand read from LDS is one conflict-free 16-byte
//     read.
//   * VALU, other d: squared distances from coordinate differences.
// A workgroup owns a block of rows and a range of columns (a chunk); when
// the rows alone would not fill the chip the columns are split in chunks,
// and the per-chunk row sums are added in chunk order by a second kernel,
// so results do not depend on scheduling.
//
// Four epilogues (template MODE):
//   kStore : write A (float32) and, if requested, the float64 row sums,
//   kStoreW: write W_ij = A_ij * r_i, r_i = float32(1 / d_i), given d,
//   kApply : y_i = (sum_j A_ij v_j) / d_i (the Multiply step with the
//            affinity recomputed; W = D^-1 A is never stored),
//   kDegree: d_i = sum_j A_ij with nothing of size n^2 written,
//   kStoreSym: write A (float32) into the packed upper tiles of the
//            symmetric storage (tiles (I, J), I <= J, of 256 x 256: see
//            sym.hip); only column tiles at or right of the row's block are
//            computed, and the storage's tile count nb comes in place of lda.
//   kApplySym: the fused product with each pair evaluated once (A = A^T):
//            a workgroup's rows (384 up to 64 coordinates, 256 above) take
//            the columns from their own first row on; the row sums go to its
//            rows, and for columns past its
//            rows A_ij v_i also goes to column sums that a second kernel
//            adds to the later rows (fused_sym_reduce_kernel).  With v = 1
//            and no division it is the degree sweep of that same A.
// Every mode evaluates the same float32 A_ij for a (row i, column j) pair
// and sums rows in the same order, so kDegree reproduces kStore's degrees
// bit for bit and kStoreW writes exactly what kStore followed by the row
// scaling writes.  A_ij and A_ji can differ in the last float32 bits (the
// two points play different parts in the Gram form); the symmetric modes
// use the value computed with the earlier point as the row.
#include "common.h"

#include <type_traits>

namespace gpic {
namespace {

enum { kStore = 0, kApply = 1, kDegree = 2, kStoreW = 3, kStoreSym = 4, kApplySym = 5 };
enum { kGauss = 0, kCosine = 1 };             // affinity kind (VALU engine)

constexpr int kThreads = 256;
constexpr int kMaxChunks = 16;

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));

// exp2 on the transcendental unit (1 ulp; results below the smallest
// normal float flush to zero, far below anything a row sum can notice)
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Address of entry (i, j), i <= j rounded to blocks of 256, in the packed
// upper tiles of the symmetric storage (nb blocks; see sym.hip).
__device__ __forceinline__ float *sym_entry(float *As, int64_t i, int64_t j, int64_t nb)
{
    const int64_t I = i >> 8, J = j >> 8;
    const int64_t t = I * nb - I * (I - 1) / 2 + (J - I);
    return As + t * 65536 + (i & 255) * 256 + (j & 255);
}

// Plain (cached) stores: measured on MI355X, non-temporal stores of this
// 16-rows-by-64-bytes pattern reach only about 60 % of the bandwidth of
// ordinary ones.
__device__ __forceinline__ void store4(float *dst, float a, float b, float c, float d)
{
    floatx4 t = {a, b, c, d};
    *reinterpret_cast<floatx4 *>(dst) = t;
}

// ------------------------------------------------------------ prologue

// rinv[p] = 1 / ||x_p|| (float64, rounded once), 0 for the origin: the
// cosine affinity (1 + x_i.x_j rinv_i rinv_j) / 2 then gives the origin
// 1/2 against every point.
__global__ __launch_bounds__(kThreads) void inv_norm_kernel(const float *__restrict__ X,
                                                            int64_t n, int d,
                                                            float *__restrict__ rinv)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= n)
        return;
    double s = 0.0;
    for (int k = 0; k < d; ++k) {
        const double x = (double)X[p * d + k];
        s = fma(x, x, s);
    }
    rinv[p] = (s > 0.0) ? (float)(1.0 / sqrt(s)) : 0.0f;
}

// The centre the Gram form works on (distances do not change under a
// shift, and the cancellation in |x_i|^2 + |x_j|^2 - 2 x_i.x_j scales with
// |x - centre|): per coordinate, the lower median of a sample of
// m = min(n, 1024) points at the evenly spaced indices floor(t n / m).  A
// median, unlike the mean, does not move with a few far points, so such
// points coarsen only their own rows and columns.  One workgroup per
// coordinate: every sampled value gets its rank in the order of (value,
// sample position), compared as integers that order like the floats, and
// the value of rank (m - 1) / 2 is the centre (exact, a float32 value).
constexpr int kCentreSample = 1024;

__device__ __forceinline__ unsigned float_order_key(float x)
{
    const unsigned b = __float_as_uint(x);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__global__ __launch_bounds__(kThreads) void centre_kernel(const float *__restrict__ X,
                                                          int64_t n, int d,
                                                          double *__restrict__ mu)
{
    __shared__ unsigned key[kCentreSample];
    __shared__ float val[kCentreSample];
    const int k = blockIdx.x;                    // coordinate
    const int m = (n < kCentreSample) ? (int)n : kCentreSample;
    for (int t = threadIdx.x; t < m; t += kThreads) {
        const float x = X[((int64_t)t * n / m) * d + k];
        val[t] = x;
        key[t] = float_order_key(x);
    }
    __syncthreads();
    const int target = (m - 1) / 2;
    for (int t = threadIdx.x; t < m; t += kThreads) {
        const unsigned kt = key[t];
        int rank = 0;
        for (int u = 0; u < m; ++u) {
            const unsigned ku = key[u];
            rank += (ku < kt || (ku == kt && u < t)) ? 1 : 0;
        }
        if (rank == target)                      // exactly one sample position
            mu[k] = (double)val[t];
    }
}

// The centred coordinate x - centre, rounded once to float32 (the same
// expression wherever it is formed).
__device__ __forceinline__ float centred(float x, double mu)
{
    return (float)((double)x - mu);
}

// Split-operand prologue of the matrix-core engine.  Every point p gets
// its own scale 2^-S_p (S_p the smallest integer with |x_pk| < 2^S_p for
// every coordinate k of the centred point; 0 for the centre itself), so
// that its scaled coordinates x'_p = x_p 2^-S_p lie in [-1, 1] whatever
// the spread of the other points; their two half-precision parts are
//   hi = fp16(x'),  lo = fp16(x' - hi)   (x' - hi is exact in float32),
// so hi + lo carries x' to within max(2^-22 |x'|, 2^-25), i.e. each
// coordinate of x_p to within max(2^-22 |x_pk|, 2^-25 2^S_p).  Layout, for
// point p (np padded points, zeros past n), chunk c of 32 coordinates,
// part h (0 hi, 1 lo) and lane group g:
//   xh[((c * 2 + h) * 4 + g) * np + p] = the 8 halves of coordinates
//                                        32 c + 8 g .. 32 c + 8 g + 7
// (the matrix-core k slots of lane group g), which makes every column
// tile a set of contiguous 1 KB runs.  Per point also (float64, each
// rounded once to float32)
//   cn[p]  = c |x_p|^2,       gam[p] = c |x_p|^2 2^-S_p,
//   sc[p]  = 2^S_p,           mr[p]  = -2 c 2^S_p,
// so that with D = x'_i . x'_j
//   c dist2(i, j) = sc_j (mr_i D + gam_j) + cn_i.
__global__ __launch_bounds__(kThreads) void split_kernel(
    const float *__restrict__ X, const double *__restrict__ mu, int64_t n, int64_t np, int d,
    int nch, float c, half8 *__restrict__ xh, float *__restrict__ cn,
    float *__restrict__ gam, float *__restrict__ sc, float *__restrict__ mr)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= np)
        return;
    const bool live = p < n;
    // the point's largest centred coordinate fixes its exponent
    float mx = 0.0f;
    if (live)
        for (int k = 0; k < d; ++k)
            mx = fmaxf(mx, fabsf(centred(X[p * d + k], mu[k])));
    int S = 0;
    if (mx > 0.0f && isfinite(mx))
        frexpf(mx, &S);                          // mx = f 2^S, f in [0.5, 1)
    double s = 0.0;
    for (int ch = 0; ch < nch; ++ch)
        for (int g = 0; g < 4; ++g) {
            half8 hi, lo;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = 32 * ch + 8 * g + e;
                const float x = (live && k < d) ? centred(X[p * d + k], mu[k]) : 0.0f;
                s = fma((double)x, (double)x, s);
                const float xs = ldexpf(x, -S);
                const _Float16 h = (_Float16)xs;
                hi[e] = h;
                lo[e] = (_Float16)(xs - (float)h);
            }
            xh[((int64_t)(ch * 2 + 0) * 4 + g) * np + p] = hi;
            xh[((int64_t)(ch * 2 + 1) * 4 + g) * np + p] = lo;
        }
    const double cs = (double)c * s;
    cn[p] = (float)cs;
    gam[p] = (float)ldexp(cs, -S);
    sc[p] = ldexpf(1.0f, S);
    mr[p] = ldexpf(-2.0f * c, S);
}

// ---------------------------------------------------- chunk row-sum reduce

// out_i = sum over chunks of part[c][i] (chunk order); kApply divides by
// d_i and writes per-workgroup partial sums of |y_i| for the L1 norm.
template <int MODE>
__global__ __launch_bounds__(kThreads) void chunk_reduce_kernel(
    const double *__restrict__ part, int nchunks, int64_t n,
    const double *__restrict__ degree_in, double *__restrict__ out,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    __shared__ double red[kThreads / kWave];
    if (MODE == kApply && use_ctl && stop_reached(ctl))
        return;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    double yabs = 0.0;
    if (i < n) {
        double s = 0.0;
        for (int c = 0; c < nchunks; ++c)
            s += part[(int64_t)c * n + i];
        if (MODE == kApply) {
            const double di = degree_in[i];
            const double yi = (di == 0.0) ? 0.0 : s / di;
            out[i] = yi;
            yabs = fabs(yi);
        } else {
            out[i] = s;
        }
    }
    if (MODE == kApply && partial != nullptr) {
        const double t = block_sum<kThreads>(yabs, red);
        if (threadIdx.x == 0)
            partial[blockIdx.x] = t;
    }
}

// Column partial sums of the symmetric fused product: row group R (rows
// R G .. R G + G - 1) holds one float64 per column j >= (R + 1) G, packed
// group after group, so group R starts at sum over R' < R of
// n - (R' + 1) G = R n - G R (R + 1) / 2 (every earlier group ends before n).
__device__ __host__ __forceinline__ int64_t colpart_offset(int64_t R, int64_t n, int64_t G)
{
    return R * n - G * R * (R + 1) / 2;
}

// y_i for the symmetric fused product: the row sums of row i's group (its
// chunk partials, chunks from the one holding the group's first row on, in
// chunk order), then the column sums that every earlier row group left for
// column i (in group order), divided by d_i; per-workgroup partial sums of
// |y_i| for the L1 norm.  With degree_in null (the degree sweep, v = 1) the
// sum itself is written.
__global__ __launch_bounds__(kThreads) void fused_sym_reduce_kernel(
    const double *__restrict__ part, int nchunks, int64_t chunk_cols,
    const double *__restrict__ colpart, int64_t n, int64_t G,
    const double *__restrict__ degree_in, double *__restrict__ out,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    __shared__ double red[kThreads / kWave];
    if (use_ctl && stop_reached(ctl))
        return;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    double yabs = 0.0;
    if (i < n) {
        const int64_t R = i / G;
        double s = 0.0;
        for (int c = (int)((R * G) / chunk_cols); c < nchunks; ++c)
            s += part[(int64_t)c * n + i];
        int64_t Rp = 0;
        for (; Rp + 4 <= R; Rp += 4) {
            double x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                x[u] = colpart[colpart_offset(Rp + u, n, G) + i - (Rp + u + 1) * G];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                s += x[u];
        }
        for (; Rp < R; ++Rp)
            s += colpart[colpart_offset(Rp, n, G) + i - (Rp + 1) * G];
        if (degree_in == nullptr) {
            out[i] = s;
        } else {
            const double di = degree_in[i];
            const double yi = (di == 0.0) ? 0.0 : s / di;
            out[i] = yi;
            yabs = fabs(yi);
        }
    }
    if (partial != nullptr) {
        const double t = block_sum<kThreads>(yabs, red);
        if (threadIdx.x == 0)
            partial[blockIdx.x] = t;
    }
}

// ------------------------------------------------------------------ MFMA

// Workgroup: W waves, each owning RB blocks of 16 rows; columns [c0, c1)
// of its chunk in tiles of TC staged through double-buffered LDS while the
// previous tile is computed.  A tile holds, per (chunk, part, lane group)
// slot, TC consecutive half8 pieces: xs[buf][slot * TC + col].  Every
// staged tile feeds 16 W RB rows, so the operand traffic from L2 per pair
// of points is 4 d / (16 W RB) bytes.
//
// v_mfma_f32_16x16x32_f16 operand layout (lane l, g = l / 16, m = l % 16;
// checked on the device):
//   A operand : row m,      k = 8 g .. 8 g + 7
//   B operand : column m,   k = 8 g .. 8 g + 7
//   result    : rows 4 g + r (r = 0..3), column m
// The A operand carries tile columns 16 q + m and the B operand the wave's
// rows i, so lane (m, g) ends with row i and columns 16 q + 4 g + r: a
// row's sum is in-lane until the end.  The symmetric product (kApplySym),
// which also sums columns, swaps the two (the per-lane operand layouts
// coincide, so the same registers serve): lane (m, g) ends with rows
// 16 rb + 4 g + r and column 16 q + m, a column's sum over the wave's rows
// is in-lane plus one sum over the four lane groups, and the row sums stay
// spread over the 16 lanes m until the end.  Each 32-coordinate chunk takes
// three products (hi.hi, lo.hi, hi.lo) into one float32 accumulator, which
// leaves D = x'_i.x'_j (each point in its own scale), and two fused
// multiply-adds give
//   c dist2 = sc_j (mr_i D + gam_j) + cn_i
// (row values in registers, column values staged with the tile);
// exp2(-c dist2) is clamped to [0, 1], which equals clamping c dist2 at 0.
// The matrix-core chain of one 16-column block is issued before the
// epilogue of the previous block, except in the symmetric product up to 64
// coordinates, which runs each block's chain and then its epilogue (the
// compiler then needs fewer registers for the three row blocks; measured
// 4 % faster at n = 200,000, d = 64 and 13 % at d = 16).
// When A or W is written (W = 4, RB = 1), the wave's 16 x TC tile goes
// through LDS and is stored as 4 rows x 4 TC contiguous bytes per store.
// s_waitcnt operand: outstanding vector memory operations 0, the other
// counters at their maximum (no wait)
constexpr int kWaitVm0 = 0x0F70;
constexpr int kChunkRows = 128;               // nominal rows per workgroup (chunking)
constexpr int kColAlign = 128;                // chunk and padding granularity (the widest tile)

template <int NCH, int RB, int TC, int MODE, int W>
__global__ __launch_bounds__(W * 64) void affinity_mfma_kernel(
    const half8 *__restrict__ xh, int64_t np, const float *__restrict__ cn,
    const float *__restrict__ gam, const float *__restrict__ sc,
    const float *__restrict__ mr, int64_t n,
    int64_t chunk_cols, float *__restrict__ A, int64_t lda,
    const double *__restrict__ v, const double *__restrict__ degree_in,
    double *__restrict__ out, double *__restrict__ part, double *__restrict__ colpart,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    constexpr int NT = W * 64;
    constexpr bool kApplyAny = (MODE == kApply || MODE == kApplySym);
    constexpr bool kSymA = (MODE == kApplySym);
    // kApplySym swaps the operands' roles (rows as A, columns as B), so lane
    // (m, g) ends with rows 16 rb + 4 g + r and tile column 16 q + m: a
    // column's sum over the wave's rows is in-lane over (rb, r) plus one
    // sum over the four lane groups, and the row sums stay spread over the
    // 16 lanes m until the end
    constexpr bool kSwap = kSymA;
    constexpr int kRV = kSwap ? 4 : 1;           // row values per row block
    // kSwap up to 64 coordinates: one block at a time (its chain, then its
    // epilogue); otherwise the next block's chain is issued before the
    // current block's epilogue
    constexpr bool kSeq = kSwap && NCH <= 2;
    constexpr int64_t kGroupRows = (int64_t)W * 16 * RB;
    constexpr int kSlots = NCH * 8;              // (chunk, part, lane group)
    constexpr int kQ = TC / 16;                  // 16-column blocks per tile
    constexpr bool kWrites = (MODE == kStore || MODE == kStoreW || MODE == kStoreSym);
    constexpr int kOutStride = TC + 4;
    static_assert(!kWrites || RB == 1, "one staged output tile per wave");
    __shared__ half8 xs[2][kSlots * TC];
    __shared__ float gs[2][TC];                  // gam_j of the staged columns
    __shared__ float ss[2][TC];                  // sc_j
    __shared__ double vs[2][kApplyAny ? TC : 1];
    __shared__ double cred[kSymA ? 2 : 1][kSymA ? W : 1][kSymA ? TC : 1];
    __shared__ double red[W];
    __shared__ float ot[kWrites ? W : 1][kWrites ? 16 * kOutStride : 1];

    if (kApplyAny && use_ctl) {
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int g = lane >> 4;
    const int m = lane & 15;
    const int64_t wrow0 = ((int64_t)blockIdx.x * W + wave) * (16 * RB);
    int64_t c0 = (int64_t)blockIdx.y * chunk_cols;
    const int64_t c1 = (c0 + chunk_cols < n) ? c0 + chunk_cols : n;
    if (MODE == kStoreSym) {
        // the workgroup's rows lie in one block of 256: only the tiles at
        // or right of the diagonal tile are stored
        const int64_t cs = (((int64_t)blockIdx.x * W * 16 * RB) >> 8) << 8;
        if (cs > c0)
            c0 = cs;
        if (c0 >= c1)
            return;                                  // uniform over the workgroup
    }
    // kApplySym: columns from the workgroup's first row on; tiles from its
    // last row + 1 on are off the diagonal block and give column sums too
    const int64_t grow0 = (int64_t)blockIdx.x * kGroupRows;
    const int64_t grow1 = grow0 + kGroupRows;
    if (kSymA) {
        if (grow0 > c0)
            c0 = grow0;
        if (c0 >= c1)
            return;                                  // uniform over the workgroup
    }
    // row operands (B; A in the symmetric product): this lane's rows, hi
    // and lo of every chunk
    half8 bh[RB][NCH], bl[RB][NCH];
    float cni[RB][kRV], mri[RB][kRV], rs[RB];
    double vi[kSwap ? RB : 1][kRV];              // kSwap: v of the lane's rows
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const int64_t i = wrow0 + 16 * rb + m;
        const int64_t ic = i < n ? i : n - 1;
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            bh[rb][ch] = xh[((int64_t)(ch * 2 + 0) * 4 + g) * np + ic];
            bl[rb][ch] = xh[((int64_t)(ch * 2 + 1) * 4 + g) * np + ic];
        }
        if (kSwap) {
#pragma unroll
            for (int r = 0; r < kRV; ++r) {
                const int64_t i2 = wrow0 + 16 * rb + 4 * g + r;
                const int64_t ic2 = i2 < n ? i2 : n - 1;
                cni[rb][r] = cn[ic2];
                mri[rb][r] = mr[ic2];
                vi[rb % (kSwap ? RB : 1)][r] = (i2 < n) ? (v != nullptr ? v[i2] : 1.0) : 0.0;
            }
        } else {
            cni[rb][0] = cn[ic];
            mri[rb][0] = mr[ic];
        }
        rs[rb] = 0.0f;

        if (MODE == kStoreW) {
            const double di = degree_in[ic];
            rs[rb] = (di == 0.0) ? 0.0f : (float)(1.0 / di);
        }
    }

    // staging: piece f = slot * TC + col (tiles start at multiples of TC,
    // chunks and row groups at multiples of kColAlign, and np is one too,
    // so every tile ends at or before np and every load is in bounds)
    // In the symmetric product the operand pieces go from memory straight
    // into LDS (a wave's 64 pieces are 1 KB of consecutive LDS; kPieces is
    // a multiple of 256, so whether a wave has a piece is uniform over it),
    // which frees the staging registers for its row values; the other
    // sweeps stage them in registers (measured: as fast or faster there,
    // and the sweeps that write A or W would otherwise wait for their
    // stores at every tile).  The column values go through registers.
    constexpr int kPieces = kSlots * TC;
    constexpr int kPer = (kPieces + NT - 1) / NT;
    static_assert(kPieces % kWave == 0, "whole waves of pieces");
    constexpr bool kDirect = kSymA;
    half8 stage[kDirect ? 1 : kPer];
    float gstage = 0.0f, sstage = 0.0f;
    double vstage = 0.0;
    auto fetch = [&](int64_t jt, int buf) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = threadIdx.x + u * NT;
            if (!kDirect && (kPieces % NT == 0 || f < kPieces))
                stage[u % (kDirect ? 1 : kPer)] = xh[(int64_t)(f / TC) * np + jt + (f % TC)];
            if (kDirect && (kPieces % NT == 0 || f < kPieces)) {
                const int fw = f - lane;                 // the wave's first piece
                __builtin_amdgcn_global_load_lds(
                    (const void *)(xh + (int64_t)(f / TC) * np + jt + (f % TC)),
                    (__attribute__((address_space(3))) void *)(&xs[buf][fw]), 16, 0, 0);
            }
        }
        if (threadIdx.x < TC) {
            gstage = gam[jt + threadIdx.x];
            sstage = sc[jt + threadIdx.x];
            if (kApplyAny) {
                const int64_t j = jt + threadIdx.x;
                vstage = (j < c1) ? (v != nullptr ? v[j] : 1.0) : 0.0;
            }
        }
    };
    auto commit = [&](int buf) {
        if (kDirect) {
            // the pieces' loads into LDS complete before the barrier that follows
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
        } else {
#pragma unroll
            for (int u = 0; u < kPer; ++u) {
                const int f = threadIdx.x + u * NT;
                if (kPieces % NT == 0 || f < kPieces)
                    xs[buf][f] = stage[u % (kDirect ? 1 : kPer)];
            }
        }
        if (threadIdx.x < TC) {
            gs[buf][threadIdx.x] = gstage;
            ss[buf][threadIdx.x] = sstage;
            if (kApplyAny)
                vs[buf][threadIdx.x] = vstage;
        }
    };

    // two float64 accumulators per row block (even and odd q), added at the
    // end; kSwap: one per row of the lane (rb, r)
    constexpr int kAcc = kSwap ? 4 : 2;
    double acc[RB][kAcc];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int u = 0; u < kAcc; ++u)
            acc[rb][u] = 0.0;

    auto tile = [&](int buf, int64_t jt, auto masked, auto offdiag) {
        constexpr bool kMask = decltype(masked)::value;
        constexpr bool kOff = kSymA && decltype(offdiag)::value;
        // one 16-column block: the matrix-core chain into cc[rb] ...
        auto chain = [&](int q, floatx4 (&cc)[RB]) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
                cc[rb] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch) {
                const half8 ah = xs[buf][((ch * 2 + 0) * 4 + g) * TC + 16 * q + m];
                const half8 al = xs[buf][((ch * 2 + 1) * 4 + g) * TC + 16 * q + m];
                // the row blocks' chains are independent: interleaved, no
                // product waits for the one before it
                // (the operands' layouts per lane coincide: swapping them
                // transposes the 16 x 16 result)
                auto mm = [&](const half8 &col, const half8 &row, const floatx4 &acc4) {
                    return kSwap ? __builtin_amdgcn_mfma_f32_16x16x32_f16(row, col, acc4, 0, 0, 0)
                                 : __builtin_amdgcn_mfma_f32_16x16x32_f16(col, row, acc4, 0, 0, 0);
                };
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
                    cc[rb] = mm(ah, bh[rb][ch], cc[rb]);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
                    cc[rb] = mm(al, bh[rb][ch], cc[rb]);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb)
                    cc[rb] = mm(ah, bl[rb][ch], cc[rb]);
            }
        };
        // ... and its epilogue
        auto epi_swap = [&](int q, const floatx4 (&cc)[RB]) {
            // lane (m, g): tile column 16 q + m, rows 16 rb + 4 g + r
            const int jl = 16 * q + m;
            const float gj = gs[buf][jl], sj = ss[buf][jl];
            const double vj = vs[buf][jl];
            // kMask: j == i  <=>  (jt - wrow0) + jl - 4 g == 16 rb + r, in
            // 32 bits (the offset clamped far outside the tile's range)
            int key = 0;
            bool colbad = false;
            if (kMask) {
                const int64_t dj = jt - wrow0;
                const int dk = (int)(dj < -(1 << 20) ? -(1 << 20) : (dj > (1 << 20) ? (1 << 20) : dj));
                key = dk + jl - 4 * g;
                colbad = (int64_t)jl >= c1 - jt;     // j >= c1
            }
            double cq = 0.0;                         // kOff: the column's sum
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float a = __builtin_amdgcn_fmed3f(
                        exp2_fast(-fmaf(fmaf(cc[rb][r], mri[rb][r % kRV], gj), sj,
                                        cni[rb][r % kRV])),
                        0.0f, 1.0f);
                    if (kMask && (key == 16 * rb + r || colbad))
                        a = 0.0f;
                    acc[rb][r % kAcc] = fma((double)a, vj, acc[rb][r % kAcc]);
                    if (kOff)
                        cq = fma((double)a, vi[rb % (kSwap ? RB : 1)][r % kRV], cq);
                }
            }
            if (kOff) {
                // add the four lane groups (rows 4 g + r): swap the upper and
                // lower 32 lanes, then odd and even rows of 16 lanes, on the
                // two halves of the float64; every lane ends with the same
                // sum (each addition takes the lower group's value first)
                auto sumx = [&](double x, bool half32) {
                    const long long b = __double_as_longlong(x);
                    const unsigned lo = (unsigned)(b & 0xffffffffll);
                    const unsigned hi = (unsigned)((unsigned long long)b >> 32);
                    unsigned l0, l1, h0, h1;
                    if (half32) {
                        const auto pl = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
                        const auto ph = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
                        l0 = pl[0]; l1 = pl[1]; h0 = ph[0]; h1 = ph[1];
                    } else {
                        const auto pl = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
                        const auto ph = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
                        l0 = pl[0]; l1 = pl[1]; h0 = ph[0]; h1 = ph[1];
                    }
                    const double x0 = __longlong_as_double((long long)(((unsigned long long)h0 << 32) | l0));
                    const double x1 = __longlong_as_double((long long)(((unsigned long long)h1 << 32) | l1));
                    return x0 + x1;
                };
                cq = sumx(cq, true);
                cq = sumx(cq, false);
                cred[buf][wave][jl] = cq;
            }
        };
        auto epi = [&](int q, const floatx4 (&cc)[RB]) {
            if constexpr (kSwap) {
                epi_swap(q, cc);
            } else {
                const floatx4 gj = *reinterpret_cast<const floatx4 *>(&gs[buf][16 * q + 4 * g]);
                const floatx4 sj = *reinterpret_cast<const floatx4 *>(&ss[buf][16 * q + 4 * g]);
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    const int64_t i = wrow0 + 16 * rb + m;
                    float a[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        a[r] = __builtin_amdgcn_fmed3f(
                            exp2_fast(-fmaf(fmaf(cc[rb][r], mri[rb][0], gj[r]), sj[r],
                                            cni[rb][0])),
                            0.0f, 1.0f);
                    const int64_t j0 = jt + 16 * q + 4 * g;    // this lane's columns
                    if (kMask) {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (j0 + r == i || j0 + r >= c1)
                                a[r] = 0.0f;
                    }
                    if (kWrites) {
                        float *ow = ot[wave] + m * kOutStride + 16 * q + 4 * g;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            ow[r] = (MODE == kStoreW) ? a[r] * rs[rb] : a[r];
                    }
                    if (MODE == kStore || MODE == kDegree) {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            acc[rb][q & 1] += (double)a[r];
                    } else if (kApplyAny) {
                        const double *vp = vs[buf] + 16 * q + 4 * g;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            acc[rb][q & 1] = fma((double)a[r], vp[r], acc[rb][q & 1]);
                    }
                }
            }
        };
        floatx4 ca[RB], cb[RB];
        if constexpr (kSeq) {
            // one block at a time: the chain, then its epilogue
#pragma unroll
            for (int q = 0; q < kQ; ++q) {
                chain(q, ca);
                epi(q, ca);
            }
        } else {
            chain(0, ca);
#pragma unroll
            for (int q = 0; q < kQ; q += 2) {
                if (q + 1 < kQ)
                    chain(q + 1, cb);
                epi(q, ca);
                if (q + 2 < kQ)
                    chain(q + 2, ca);
                if (q + 1 < kQ)
                    epi(q + 1, cb);
            }
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            if (kWrites) {
                // the wave's 16 x TC tile, 4 rows x 4 TC contiguous bytes per store
                const int64_t rrow0 = wrow0 + 16 * rb;
                constexpr int kLanesPerRow = TC / 4;
                constexpr int kRowsPerStore = kWave / kLanesPerRow;
#pragma unroll
                for (int u = 0; u < 16 / kRowsPerStore; ++u) {
                    const int rr = kRowsPerStore * u + lane / kLanesPerRow;
                    const int cc = 4 * (lane % kLanesPerRow);
                    const int64_t ii = rrow0 + rr;
                    const int64_t jj = jt + cc;
                    const float *src = ot[wave] + rr * kOutStride + cc;
                    if (ii < n) {
                        float *dst = (MODE == kStoreSym) ? sym_entry(A, ii, jj, lda)
                                                         : A + ii * lda + jj;
                        if (!kMask || jj + 3 < c1) {
                            store4(dst, src[0], src[1], src[2], src[3]);
                        } else {
                            for (int e = 0; e < 4 && jj + e < c1; ++e)
                                dst[e] = src[e];
                        }
                    }
                }
            }
        }
    };

    const int64_t ntiles = (c1 - c0 + TC - 1) / TC;
    const int64_t rlo = wrow0, rhi = wrow0 + 16 * RB;   // this wave's rows
    fetch(c0, 0);
    commit(0);
    __syncthreads();
    for (int64_t t = 0; t < ntiles; ++t) {
        const int buf = (int)(t & 1);
        const int64_t jt = c0 + t * TC;
        if (t + 1 < ntiles)
            fetch(jt + TC, buf ^ 1);                 // in flight during compute
        const bool diag = (rlo < jt + TC) && (jt < rhi);
        const bool tail = jt + TC > c1;
        const bool off = kSymA && jt >= grow1;
        if (off) {
            if (tail)
                tile(buf, jt, std::true_type{}, std::true_type{});
            else
                tile(buf, jt, std::false_type{}, std::true_type{});
        } else if (diag || tail) {
            tile(buf, jt, std::true_type{}, std::false_type{});
        } else {
            tile(buf, jt, std::false_type{}, std::false_type{});
        }
        if (t + 1 < ntiles) {
            // the barrier ending the previous iteration ordered every wave's
            // reads of buffer buf ^ 1 before this tile's loads into it; this
            // one orders them before the next tile's reads
            commit(buf ^ 1);
            __syncthreads();
        } else if (kSymA) {
            __syncthreads();
        }
        if (off && threadIdx.x < TC) {
            // the tile's column sums over the workgroup's rows, in wave order
            // (cred[buf] is written again two tiles on, after the next barrier)
            const int64_t j = jt + threadIdx.x;
            if (j < c1) {
                double cs = 0.0;
#pragma unroll
                for (int w = 0; w < W; ++w)
                    cs += cred[buf][w][threadIdx.x];
                colpart[colpart_offset(blockIdx.x, n, kGroupRows) + (j - grow1)] = cs;
            }
        }
    }

    if (MODE == kStoreW || MODE == kStoreSym)
        return;
    double yabs = 0.0;
#pragma unroll
    for (int rb = 0; rb < RB * kRV; ++rb) {
        int64_t i;
        double s;
        if (kSwap) {
            // row 16 rb + 4 g + r: the 16 lanes m of its lane group hold
            // disjoint columns
            const int b = rb / kRV, r = rb % kRV;
            i = wrow0 + 16 * b + 4 * g + r;
            s = acc[b][r % kAcc];
            s += __shfl_xor(s, 8, kWave);
            s += __shfl_xor(s, 4, kWave);
            s += __shfl_xor(s, 2, kWave);
            s += __shfl_xor(s, 1, kWave);
            if (m != 0 || i >= n)
                continue;
        } else {
            i = wrow0 + 16 * rb + m;
            s = acc[rb][0] + acc[rb][1 % kAcc];
            // the four lanes sharing a row (g = 0..3) hold disjoint columns
            s += __shfl_xor(s, 16, kWave);
            s += __shfl_xor(s, 32, kWave);
            if (g != 0 || i >= n)
                continue;
        }
        if (part != nullptr) {
            // chunk partial, reduced in chunk order by chunk_reduce_kernel
            part[(int64_t)blockIdx.y * n + i] = s;
        } else if (MODE == kApply) {
            const double di = degree_in[i];
            const double yi = (di == 0.0) ? 0.0 : s / di;
            out[i] = yi;
            yabs += fabs(yi);
        } else if (out != nullptr) {
            out[i] = s;
        }
    }
    if (MODE == kApply && part == nullptr && partial != nullptr) {
        const double sum = block_sum<NT>(yabs, red);
        if (threadIdx.x == 0)
            partial[blockIdx.x] = sum;
    }
}

// ------------------------------------------------------------------ VALU

// Block: 256 threads, RB rows; each thread takes groups of 4 consecutive
// columns (one 16-byte store per row), stepping by 1024 columns.
// KIND kGauss: exp2(-c dist^2) from coordinate differences; kCosine:
// max(0, (1 + (x_i.x_j) rinv_i rinv_j) / 2), the float32 dot product of the
// raw coordinates scaled by the reciprocal norms.
template <int D, int RB, int MODE, int KIND = kGauss>
__global__ __launch_bounds__(kThreads) void affinity_valu_kernel(
    const float *__restrict__ X, int64_t n, int dyn_d, float c,
    float *__restrict__ A, int64_t lda, const double *__restrict__ v,
    const double *__restrict__ degree_in, double *__restrict__ out,
    double *__restrict__ partial, StopCtl ctl, int use_ctl,
    const float *__restrict__ rinv = nullptr)
{
    __shared__ double red[kThreads / kWave];
    if (MODE == kApply && use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int d = (D > 0) ? D : dyn_d;
    const int64_t row0 = (int64_t)blockIdx.x * RB;
    constexpr int DR = (D > 0) ? D : 1;
    float xi[RB][DR];
    if (D > 0) {
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            const int64_t i = (row0 + r < n) ? row0 + r : n - 1;
#pragma unroll
            for (int k = 0; k < DR; ++k)
                xi[r][k] = X[i * d + k];
        }
    }
    double acc[RB];
    float rs[RB];
    float ri[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        acc[r] = 0.0;
        rs[r] = 0.0f;
        ri[r] = (KIND == kCosine) ? rinv[(row0 + r < n) ? row0 + r : n - 1] : 0.0f;
        if (MODE == kStoreW) {
            const int64_t i = (row0 + r < n) ? row0 + r : n - 1;
            const double di = degree_in[i];
            rs[r] = (di == 0.0) ? 0.0f : (float)(1.0 / di);
        }
    }

    const int64_t ngroups = (n + 3) >> 2;
    // kStoreSym: the RB rows lie in one block of 256; columns from that
    // block's diagonal tile on
    const int64_t g0 = (MODE == kStoreSym) ? (((row0 >> 8) << 8) >> 2) : 0;
    for (int64_t gi = g0 + threadIdx.x; gi < ngroups; gi += kThreads) {
        const int64_t j0 = gi << 2;
        float a[RB][4];
        if (D > 0) {
            float xj[4][DR];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t j = (j0 + q < n) ? j0 + q : n - 1;
#pragma unroll
                for (int k = 0; k < DR; ++k)
                    xj[q][k] = X[j * d + k];
            }
            float rj[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if (KIND == kCosine) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    rj[q] = rinv[(j0 + q < n) ? j0 + q : n - 1];
            }
#pragma unroll
            for (int r = 0; r < RB; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float s = 0.0f;
                    if (KIND == kCosine) {
#pragma unroll
                        for (int k = 0; k < DR; ++k)
                            s = fmaf(xi[r][k], xj[q][k], s);
                        a[r][q] = fmaxf(fmaf(0.5f, s * (ri[r] * rj[q]), 0.5f), 0.0f);
                    } else {
#pragma unroll
                        for (int k = 0; k < DR; ++k) {
                            const float df = xi[r][k] - xj[q][k];
                            s = fmaf(df, df, s);
                        }
                        a[r][q] = exp2_fast(-c * s);
                    }
                }
        } else {
            // any d (used above the matrix-core range): coordinates re-read
#pragma unroll
            for (int r = 0; r < RB; ++r) {
                const int64_t i = (row0 + r < n) ? row0 + r : n - 1;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t j = (j0 + q < n) ? j0 + q : n - 1;
                    float s = 0.0f;
                    if (KIND == kCosine) {
                        for (int k = 0; k < d; ++k)
                            s = fmaf(X[i * d + k], X[j * d + k], s);
                        a[r][q] = fmaxf(fmaf(0.5f, s * (ri[r] * rinv[j]), 0.5f), 0.0f);
                    } else {
                        for (int k = 0; k < d; ++k) {
                            const float df = X[i * d + k] - X[j * d + k];
                            s = fmaf(df, df, s);
                        }
                        a[r][q] = exp2_fast(-c * s);
                    }
                }
            }
        }
        double vj[4] = {1.0, 1.0, 1.0, 1.0};
        if (MODE == kApply) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                vj[q] = (j0 + q < n) ? v[j0 + q] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            const int64_t i = row0 + r;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (i == j0 + q || j0 + q >= n)
                    a[r][q] = 0.0f;
            if ((MODE == kStore || MODE == kStoreW || MODE == kStoreSym) && i < n) {
                float o[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    o[q] = (MODE == kStoreW) ? a[r][q] * rs[r] : a[r][q];
                float *dst = (MODE == kStoreSym) ? sym_entry(A, i, j0, lda) : A + i * lda + j0;
                if (j0 + 3 < n) {
                    store4(dst, o[0], o[1], o[2], o[3]);
                } else {
                    for (int q = 0; q < 4 && j0 + q < n; ++q)
                        dst[q] = o[q];
                }
            }
            if (MODE != kStoreW && MODE != kStoreSym) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    acc[r] = fma((double)a[r][q], vj[q], acc[r]);
            }
        }
    }

    if (MODE == kStoreW || MODE == kStoreSym)
        return;
    double part = 0.0;
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        const double t = block_sum<kThreads>(acc[r], red);
        const int64_t i = row0 + r;
        if (i < n) {
            if (MODE == kStore) {
                if (out != nullptr && threadIdx.x == 0)
                    out[i] = t;
            } else if (MODE == kDegree) {
                if (threadIdx.x == 0)
                    out[i] = t;
            } else {
                const double di = degree_in[i];
                const double yi = (di == 0.0) ? 0.0 : t / di;
                if (threadIdx.x == 0)
                    out[i] = yi;
                part += fabs(yi);
            }
        }
    }
    if (MODE == kApply && partial != nullptr && threadIdx.x == 0)
        partial[blockIdx.x] = part;
}

// ------------------------------------------------------------- dispatch

bool use_mfma(int d) { return d >= 16 && d <= 128; }

constexpr int kMaxNch = 4;                   // 32-coordinate chunks for d <= 128

int nch_for(int d) { return (d + 31) / 32; }

// Row blocking: the sweeps that only sum rows take four 16-row blocks per
// wave and 8 waves per workgroup (512 rows share every staged column tile,
// and four independent matrix-core chains per wave hide each other's
// latency; measured 14.9 ms per product at n = 200,000, d = 64, against
// 16.4 with 128 rows); the symmetric product, which also keeps column sums
// and v of its rows, takes three blocks per wave (384 rows) with 128-column
// tiles up to 64 coordinates (n = 200,000, d = 64: 9.1 ms per product
// against 10.6 with two blocks and 64-column tiles; four blocks spill) and
// two blocks with 32-column tiles above (three spill there); the sweeps
// that write A or W take one block per wave and 4 waves (their bound is
// the stores).
constexpr bool sums_rows(int mode)
{
    return mode == kApply || mode == kDegree || mode == kApplySym;
}
constexpr int rb_for(int mode, int nch)
{
    return mode == kApplySym ? (nch <= 2 ? 3 : 2) : (sums_rows(mode) ? 4 : 1);
}
constexpr int waves_for(int mode) { return sums_rows(mode) ? 8 : 4; }
constexpr int tc_for(int mode, int nch)
{
    return (mode == kApplySym && nch <= 2) ? 128 : (nch <= 2 ? 64 : 32);
}
constexpr int64_t rows_per_group(int mode, int nch)
{
    return 16 * rb_for(mode, nch) * waves_for(mode);
}

int64_t row_groups(int64_t n, int mode, int nch)
{
    return (n + rows_per_group(mode, nch) - 1) / rows_per_group(mode, nch);
}

// Column chunks: enough workgroups to fill the chip when rows are few.
// The chunk width depends on n alone, so every mode sums a row's columns
// in the same order.
void chunking(int64_t n, int64_t *chunk_cols, int *nchunks)
{
    const int64_t groups = (n + kChunkRows - 1) / kChunkRows;
    int64_t want = (4096 + groups - 1) / groups;     // >= 4 workgroups per CU
    if (want < 1)
        want = 1;
    if (want > kMaxChunks)
        want = kMaxChunks;
    int64_t cols = (n + want - 1) / want;
    cols = (cols + kColAlign - 1) / kColAlign * kColAlign;
    *chunk_cols = cols;
    *nchunks = (int)((n + cols - 1) / cols);
}

int64_t padded_points(int64_t n) { return (n + kColAlign - 1) / kColAlign * kColAlign; }

// The symmetric fused product (each pair once: row sums for the row's
// group, column sums for the column's) up to this many points; its column
// partial sums take about n^2 / 64 bytes (4.3 GB at the limit).  Above it
// the product sums whole rows.
constexpr int64_t kFusedSymMaxN = 1 << 19;

bool fused_sym(int64_t n, int d) { return use_mfma(d) && n <= kFusedSymMaxN; }

// Column partial sums of the symmetric product for row groups of G rows:
// the smaller G (256 rows, above 64 coordinates) needs the most entries,
// so the workspace is sized for it whatever d the product gets.
int64_t colpart_entries_for(int64_t n, int64_t G)
{
    const int64_t groups = (n + G - 1) / G;
    return colpart_offset(groups - 1, n, G);
}
int64_t colpart_entries(int64_t n)
{
    const int64_t a = colpart_entries_for(n, rows_per_group(kApplySym, 1));
    const int64_t b = colpart_entries_for(n, rows_per_group(kApplySym, kMaxNch));
    return a > b ? a : b;
}

// Column chunks of the symmetric product: kMaxChunks chunks, so that the
// triangle of (row group, chunk) pieces spreads over many workgroups.
void sym_chunking(int64_t n, int64_t *chunk_cols, int *nchunks)
{
    int64_t cols = (n + kMaxChunks - 1) / kMaxChunks;
    cols = (cols + kColAlign - 1) / kColAlign * kColAlign;
    *chunk_cols = cols;
    *nchunks = (int)((n + cols - 1) / cols);
}

int64_t al256(int64_t x) { return (x + 255) & ~(int64_t)255; }

struct Ws {
    half8 *xh;          // split operands, kMaxNch * 8 slots of np half8
    float *cn;          // [np] c |x|^2
    float *gam;         // [np] c |x|^2 2^-S
    float *sc;          // [np] 2^S
    float *mr;          // [np] -2 c 2^S
    double *mu;         // the centre [32 kMaxNch]
    double *part;       // per-chunk row sums, kMaxChunks * n
};

Ws carve(void *ws, int64_t n)
{
    char *b = static_cast<char *>(ws);
    const int64_t np = padded_points(n);
    Ws w;
    w.xh = reinterpret_cast<half8 *>(b);
    b += al256(np * kMaxNch * 8 * (int64_t)sizeof(half8));
    w.cn = reinterpret_cast<float *>(b);
    b += al256(np * 4);
    w.gam = reinterpret_cast<float *>(b);
    b += al256(np * 4);
    w.sc = reinterpret_cast<float *>(b);
    b += al256(np * 4);
    w.mr = reinterpret_cast<float *>(b);
    b += al256(np * 4);
    w.mu = reinterpret_cast<double *>(b);
    b += al256(32 * kMaxNch * 8);
    w.part = reinterpret_cast<double *>(b);
    return w;
}

hipError_t launch_split(const float *X, int64_t n, int d, float c, const Ws &w,
                        hipStream_t s)
{
    const int64_t np = padded_points(n);
    hipLaunchKernelGGL(centre_kernel, dim3((unsigned)d), dim3(kThreads), 0, s, X, n, d, w.mu);
    hipLaunchKernelGGL(split_kernel, dim3((unsigned)((np + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, X, w.mu, n, np, d, nch_for(d), c, w.xh, w.cn,
                       w.gam, w.sc, w.mr);
    return hipGetLastError();
}

template <int NCH, int MODE>
void launch_engine(const Ws &w, int64_t n, int64_t chunk_cols, int nchunks, float *A,
                   int64_t lda, const double *v, const double *degree_in, double *out,
                   double *part, double *partial, StopCtl ctl, int use_ctl, hipStream_t s,
                   double *colpart = nullptr)
{
    constexpr int RB = rb_for(MODE, NCH);
    constexpr int W = waves_for(MODE);
    constexpr int TC = tc_for(MODE, NCH);
    static_assert(kColAlign % TC == 0, "tiles start and end on the padding grain");
    const dim3 grid((unsigned)row_groups(n, MODE, NCH), (unsigned)nchunks);
    hipLaunchKernelGGL((affinity_mfma_kernel<NCH, RB, TC, MODE, W>), grid, dim3(W * 64), 0,
                       s, w.xh, padded_points(n), w.cn, w.gam, w.sc, w.mr, n, chunk_cols, A,
                       lda, v, degree_in, out, part, colpart, partial, ctl, use_ctl);
}

template <int MODE>
hipError_t dispatch(const float *X, int64_t n, int d, float c, float *A,
                    int64_t lda, const double *v, const double *degree_in,
                    double *out, double *partial, StopCtl ctl, int use_ctl,
                    void *ws, hipStream_t s, bool operands_ready = false)
{
    if (use_mfma(d)) {
        const Ws w = carve(ws, n);
        if (!operands_ready) {
            const hipError_t e = launch_split(X, n, d, c, w, s);
            if (e != hipSuccess)
                return e;
        }
        int64_t chunk_cols;
        int nchunks;
        chunking(n, &chunk_cols, &nchunks);
        const bool sums = (MODE != kStoreW) && (MODE != kStoreSym) &&
                          (MODE != kStore || out != nullptr);
        double *part = (sums && nchunks > 1) ? w.part : nullptr;
#define GPIC_MFMA(NCH)                                                          \
    launch_engine<NCH, MODE>(w, n, chunk_cols, nchunks, A, lda, v, degree_in, out, \
                             part, partial, ctl, use_ctl, s)
        switch (nch_for(d)) {
        case 1: GPIC_MFMA(1); break;
        case 2: GPIC_MFMA(2); break;
        case 3: GPIC_MFMA(3); break;
        default: GPIC_MFMA(4); break;
        }
#undef GPIC_MFMA
        if (part != nullptr) {
            const dim3 rg((unsigned)((n + kThreads - 1) / kThreads));
            if (MODE == kApply)
                hipLaunchKernelGGL(chunk_reduce_kernel<kApply>, rg, dim3(kThreads), 0, s,
                                   part, nchunks, n, degree_in, out, partial, ctl,
                                   use_ctl);
            else
                hipLaunchKernelGGL(chunk_reduce_kernel<kDegree>, rg, dim3(kThreads), 0,
                                   s, part, nchunks, n, degree_in, out, partial, ctl,
                                   use_ctl);
        }
        return hipGetLastError();
    }
    const dim3 block(kThreads);
    constexpr int RB = 8;
    const dim3 grid((unsigned)((n + RB - 1) / RB));
#define GPIC_VALU(D)                                                           \
    case D:                                                                    \
        hipLaunchKernelGGL((affinity_valu_kernel<D, RB, MODE>), grid, block, 0, \
                           s, X, n, d, c, A, lda, v, degree_in, out, partial,  \
                           ctl, use_ctl);                                      \
        break;
    switch (d) {
        GPIC_VALU(1) GPIC_VALU(2) GPIC_VALU(3) GPIC_VALU(4) GPIC_VALU(5)
        GPIC_VALU(6) GPIC_VALU(7) GPIC_VALU(8) GPIC_VALU(9) GPIC_VALU(10)
        GPIC_VALU(11) GPIC_VALU(12) GPIC_VALU(13) GPIC_VALU(14) GPIC_VALU(15)
    default:
        hipLaunchKernelGGL((affinity_valu_kernel<0, RB, MODE>), grid, block, 0,
                           s, X, n, d, c, A, lda, v, degree_in, out, partial,
                           ctl, use_ctl);
    }
#undef GPIC_VALU
    return hipGetLastError();
}

template <int MODE>
hipError_t dispatch_cosine(const float *X, int64_t n, int d, float *A, int64_t lda,
                           const double *degree_in, double *out, float *rinv,
                           hipStream_t s)
{
    hipLaunchKernelGGL(inv_norm_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, X, n, d, rinv);
    const dim3 block(kThreads);
    constexpr int RB = 8;
    const dim3 grid((unsigned)((n + RB - 1) / RB));
    StopCtl none{};
#define GPIC_COS(D)                                                             \
    case D:                                                                    \
        hipLaunchKernelGGL((affinity_valu_kernel<D, RB, MODE, kCosine>), grid, block, \
                           0, s, X, n, d, 0.0f, A, lda, nullptr, degree_in, out, \
                           nullptr, none, 0, rinv);                            \
        break;
    switch (d) {
        GPIC_COS(1) GPIC_COS(2) GPIC_COS(3) GPIC_COS(4) GPIC_COS(5)
        GPIC_COS(6) GPIC_COS(7) GPIC_COS(8) GPIC_COS(9) GPIC_COS(10)
        GPIC_COS(11) GPIC_COS(12) GPIC_COS(13) GPIC_COS(14) GPIC_COS(15)
        GPIC_COS(16)
    default:
        hipLaunchKernelGGL((affinity_valu_kernel<0, RB, MODE, kCosine>), grid, block, 0,
                           s, X, n, d, 0.0f, A, lda, nullptr, degree_in, out, nullptr,
                           none, 0, rinv);
    }
#undef GPIC_COS
    return hipGetLastError();
}

} // namespace

size_t cosine_ws(int64_t n) { return (size_t)al256(n * 4); }

hipError_t launch_affinity_cosine(const float *X, int64_t n, int d, float *A,
                                  int64_t lda, double *degree, void *ws, hipStream_t s)
{
    return dispatch_cosine<kStore>(X, n, d, A, lda, nullptr, degree,
                                   static_cast<float *>(ws), s);
}

hipError_t launch_cosine_degree(const float *X, int64_t n, int d, double *degree,
                                void *ws, hipStream_t s)
{
    return dispatch_cosine<kDegree>(X, n, d, nullptr, 0, nullptr, degree,
                                    static_cast<float *>(ws), s);
}

hipError_t launch_cosine_w(const float *X, int64_t n, int d, float *W, int64_t ldw,
                           const double *degree, void *ws, hipStream_t s)
{
    return dispatch_cosine<kStoreW>(X, n, d, W, ldw, degree, nullptr,
                                    static_cast<float *>(ws), s);
}

size_t affinity_ws(int64_t n)
{
    const int64_t np = padded_points(n);
    return (size_t)(al256(np * kMaxNch * 8 * (int64_t)sizeof(half8)) +
                    4 * al256(np * 4) + al256(32 * kMaxNch * 8) +
                    al256((int64_t)kMaxChunks * n * 8));
}

int64_t fused_blocks(int64_t n, int d)
{
    if (!use_mfma(d))
        return (n + 7) / 8;
    if (fused_sym(n, d))
        return (n + kThreads - 1) / kThreads;        // fused_sym_reduce workgroups
    int64_t chunk_cols;
    int nchunks;
    chunking(n, &chunk_cols, &nchunks);
    if (nchunks > 1)
        return (n + kThreads - 1) / kThreads;        // chunk_reduce workgroups
    return row_groups(n, kApply, nch_for(d));        // tile workgroups
}

hipError_t launch_affinity(const float *X, int64_t n, int d, float c, float *A,
                           int64_t lda, double *degree, void *ws, hipStream_t s)
{
    StopCtl none{};
    return dispatch<kStore>(X, n, d, c, A, lda, nullptr, nullptr, degree,
                            nullptr, none, 0, ws, s);
}

hipError_t launch_affinity_w(const float *X, int64_t n, int d, float c,
                             float *W, int64_t ldw, const double *degree,
                             void *ws, hipStream_t s)
{
    StopCtl none{};
    return dispatch<kStoreW>(X, n, d, c, W, ldw, nullptr, degree, nullptr,
                             nullptr, none, 0, ws, s);
}

hipError_t launch_affinity_sym(const float *X, int64_t n, int d, float c, float *As,
                               void *ws, hipStream_t s)
{
    StopCtl none{};
    const int64_t nb = (n + 255) / 256;            // tiles per block row (see sym.hip)
    return dispatch<kStoreSym>(X, n, d, c, As, nb, nullptr, nullptr, nullptr, nullptr,
                               none, 0, ws, s);
}

hipError_t launch_fused_degree(const float *X, int64_t n, int d, float c,
                               double *degree, void *ws, hipStream_t s)
{
    StopCtl none{};
    return dispatch<kDegree>(X, n, d, c, nullptr, 0, nullptr, nullptr, degree,
                             nullptr, none, 0, ws, s);
}

hipError_t launch_fused_prepare(const float *X, int64_t n, int d, float c, void *ws,
                                hipStream_t s)
{
    if (!use_mfma(d))
        return hipSuccess;
    return launch_split(X, n, d, c, carve(ws, n), s);
}

hipError_t launch_fused_apply(const float *X, int64_t n, int d, float c,
                              const double *v, const double *degree, double *y,
                              double *partial, StopCtl ctl, bool use_ctl,
                              void *ws, hipStream_t s, bool operands_ready)
{
    if (!fused_sym(n, d))
        return dispatch<kApply>(X, n, d, c, nullptr, 0, v, degree, y, partial, ctl,
                                use_ctl ? 1 : 0, ws, s, operands_ready);
    const Ws w = carve(ws, n);
    if (!operands_ready) {
        const hipError_t e = launch_split(X, n, d, c, w, s);
        if (e != hipSuccess)
            return e;
    }
    double *colpart = reinterpret_cast<double *>(static_cast<char *>(ws) + affinity_ws(n));
    int64_t chunk_cols;
    int nchunks;
    sym_chunking(n, &chunk_cols, &nchunks);
    const int uc = use_ctl ? 1 : 0;
#define GPIC_MFMA(NCH)                                                                \
    launch_engine<NCH, kApplySym>(w, n, chunk_cols, nchunks, nullptr, 0, v, degree,   \
                                  nullptr, w.part, nullptr, ctl, uc, s, colpart)
    switch (nch_for(d)) {
    case 1: GPIC_MFMA(1); break;
    case 2: GPIC_MFMA(2); break;
    case 3: GPIC_MFMA(3); break;
    default: GPIC_MFMA(4); break;
    }
#undef GPIC_MFMA
    const int64_t G = rows_per_group(kApplySym, nch_for(d));
    hipLaunchKernelGGL(fused_sym_reduce_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, w.part, nchunks, chunk_cols, colpart, n, G, degree,
                       y, partial, ctl, uc);
    return hipGetLastError();
}

hipError_t launch_fused_operator_degree(const float *X, int64_t n, int d, float c,
                                       double *degree, void *ws, hipStream_t s)
{
    if (!fused_sym(n, d))
        return launch_fused_degree(X, n, d, c, degree, ws, s);
    // the symmetric product with v = 1 and no division: the degrees of the
    // same symmetric A the products use, so W's rows sum to 1 up to rounding
    StopCtl none{};
    return launch_fused_apply(X, n, d, c, nullptr, nullptr, degree, nullptr, none, false,
                              ws, s, false);
}

size_t fused_ws(int64_t n)
{
    size_t b = affinity_ws(n);
    if (n <= kFusedSymMaxN)                          // whatever d the product gets
        b += (size_t)colpart_entries(n) * sizeof(double);
    return b;
}

} // namespace gpic
