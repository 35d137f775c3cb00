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
//   * MFMA, 16 <= d <= 128.  The matrix cores produce c * dist2 directly:
//     column operands are the augmented points [x_j, |x_j|^2, 1] and row
//     operands [-2c x_i, c, c |x_i|^2], so one fp32 Gram product gives
//     c (|x_i|^2 + |x_j|^2 - 2 x_i.x_j); it is clamped at 0 before exp2.
//     A prologue kernel writes both augmented operand arrays once per call
//     (squared norms as float64 sums rounded to float32, points padded with
//     zeros to a multiple of 64); the column operand is stored coordinate-
//     major, so a column tile is staged into LDS by contiguous 16-byte
//     copies and every wave reads its matrix-core operands for four column
//     blocks with one conflict-free 16-byte LDS read.
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
//   kDegree: d_i = sum_j A_ij with nothing of size n^2 written.
// Every mode evaluates the same float32 A_ij and sums rows in the same
// order, so kDegree reproduces kStore's degrees bit for bit and kStoreW
// writes exactly what kStore followed by the row scaling writes.
#include "common.h"

namespace gpic {
namespace {

enum { kStore = 0, kApply = 1, kDegree = 2, kStoreW = 3 };
enum { kGauss = 0, kCosine = 1 };             // affinity kind (VALU engine)

constexpr int kThreads = 256;
constexpr int kMaxChunks = 16;

typedef float floatx4 __attribute__((ext_vector_type(4)));

// exp2 on the transcendental unit (1 ulp; results below the smallest
// normal float flush to zero, far below anything a row sum can notice)
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Plain (cached) stores: measured on MI355X, non-temporal stores of this
// 16-rows-by-64-bytes pattern reach only about 60 % of the bandwidth of
// ordinary ones.
__device__ __forceinline__ void store4(float *dst, float a, float b, float c, float d)
{
    floatx4 t = {a, b, c, d};
    *reinterpret_cast<floatx4 *>(dst) = t;
}

// ------------------------------------------------------------ prologue

// Augmented operands, KP floats per point (KP = 4 KS >= d + 2):
//   column operand, coordinate-major: xa[k * np + p] = [x_p, |x_p|^2, 1, 0...]_k
//   row operand, point-major:         xb[p * KP + k] = [-2c x_p, c, c |x_p|^2, 0...]_k
// |x_p|^2 is a float64 sum rounded once to float32.  Points n .. np-1
// (padding up to a multiple of the column tile) are all zeros.
__global__ __launch_bounds__(kThreads) void augment_kernel(
    const float *__restrict__ X, int64_t n, int64_t np, int d, int KP, float c,
    float *__restrict__ xa, float *__restrict__ xb)
{
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= np)
        return;
    float *a = xa + p;                            // stride np
    float *b = xb + p * KP;
    if (p >= n) {
        for (int k = 0; k < KP; ++k) {
            a[k * np] = 0.0f;
            b[k] = 0.0f;
        }
        return;
    }
    double s = 0.0;
    for (int k = 0; k < d; ++k) {
        const double x = (double)X[p * d + k];
        s = fma(x, x, s);
    }
    const float nrm = (float)s;
    for (int k = 0; k < KP; ++k) {
        if (k < d) {
            const float x = X[p * d + k];
            a[k * np] = x;
            b[k] = -2.0f * c * x;
        } else if (k == d) {
            a[k * np] = nrm;
            b[k] = c;
        } else if (k == d + 1) {
            a[k * np] = 1.0f;
            b[k] = c * nrm;
        } else {
            a[k * np] = 0.0f;
            b[k] = 0.0f;
        }
    }
}

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

// ------------------------------------------------------------------ MFMA

// Workgroup: kMfmaWaves waves x 16 rows; columns [c0, c1) of its chunk in
// tiles of 64 staged through double-buffered LDS, coordinate-major: tile
// column c of coordinate k sits at xs[k][c ^ (16 (k % 4))].  The XOR
// swizzle spreads the four coordinates a wave reads at once over all 64
// banks (conflict-free 4-byte reads) and keeps 4-column groups contiguous
// for 16-byte staging writes.
//
// v_mfma_f32_16x16x4f32 operand layout (lane l, g = l / 16, m = l % 16):
//   A operand : element (row m,  k = g)
//   B operand : element (k = g,  column m)
//   result    : elements (row 4g + r, column m), r = 0..3
// The A operand of block q (q = 0..3) carries tile columns 16 q + a and
// the B operand the wave's 16 rows i.  Lane (m, g) ends with row i and
// columns 16 q + 4 g + r.  When A or W is written, the wave's 16 x 64
// tile goes through LDS first and is stored as 4 rows x 256 contiguous
// bytes per instruction (measured 10 % faster than 16 rows x 64 bytes).
constexpr int kMfmaWaves = 4;                 // waves (16 rows each) per workgroup
constexpr int kMfmaThreads = kMfmaWaves * 64;
constexpr int kRowsPerWave = 16;
constexpr int kRowsPerGroup = kMfmaWaves * kRowsPerWave;
constexpr int kTileCols = 64;

template <int KS, int MODE>
__global__ __launch_bounds__(kMfmaThreads) void affinity_mfma_kernel(
    const float *__restrict__ xa, int64_t np, const float *__restrict__ xb, int64_t n,
    int64_t chunk_cols, float *__restrict__ A, int64_t lda,
    const double *__restrict__ v, const double *__restrict__ degree_in,
    double *__restrict__ out, double *__restrict__ part,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    constexpr int KP = 4 * KS;               // augmented, padded dimension
    constexpr int kRow4 = kTileCols / 4;     // 16-byte pieces per coordinate
    __shared__ floatx4 xs[2][KP * kRow4];
    __shared__ double vs[2][kTileCols];
    __shared__ double red[kMfmaThreads / kWave];
    constexpr int kOutStride = kTileCols + 4;
    __shared__ float ot[(MODE == kStore || MODE == kStoreW) ? kMfmaWaves : 1][16 * kOutStride];

    if (MODE == kApply && use_ctl) {
        if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int g = lane >> 4;
    const int m = lane & 15;
    const int64_t wrow0 = (int64_t)blockIdx.x * kRowsPerGroup + wave * kRowsPerWave;
    const int64_t i = wrow0 + m;
    const bool row_ok = i < n;
    const int64_t ic = row_ok ? i : n - 1;
    const int64_t c0 = (int64_t)blockIdx.y * chunk_cols;
    const int64_t c1 = (c0 + chunk_cols < n) ? c0 + chunk_cols : n;

    // B operand: augmented row coordinates 4 s + g of [-2c x_i, c, c |x_i|^2]
    float bop[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s)
        bop[s] = xb[ic * KP + 4 * s + g];
    float rs = 0.0f;
    if (MODE == kStoreW) {
        const double di = degree_in[ic];
        rs = (di == 0.0) ? 0.0f : (float)(1.0 / di);
    }

    // staging: piece f = k * 16 + cg holds columns 4 cg .. 4 cg + 3 of
    // coordinate k (tiles start at multiples of 64 <= np - 64)
    constexpr int kPieces = KP * kRow4;
    constexpr int kPer = (kPieces + kMfmaThreads - 1) / kMfmaThreads;
    floatx4 stage[kPer];
    double vstage = 0.0;
    auto fetch = [&](int64_t jt) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = threadIdx.x + u * kMfmaThreads;
            if (kPieces % kMfmaThreads == 0 || f < kPieces)
                stage[u] = *reinterpret_cast<const floatx4 *>(
                    xa + (int64_t)(f / kRow4) * np + jt + 4 * (f % kRow4));
        }
        if (MODE == kApply && threadIdx.x < kTileCols) {
            const int64_t j = jt + threadIdx.x;
            vstage = (j < c1) ? v[j] : 0.0;
        }
    };
    auto commit = [&](int buf) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int f = threadIdx.x + u * kMfmaThreads;
            if (kPieces % kMfmaThreads == 0 || f < kPieces) {
                const int k = f / kRow4;
                xs[buf][k * kRow4 + ((f % kRow4) ^ (4 * (k & 3)))] = stage[u];
            }
        }
        if (MODE == kApply && threadIdx.x < kTileCols)
            vs[buf][threadIdx.x] = vstage;
    };

    double acc = 0.0;
    const int64_t ntiles = (c1 - c0 + kTileCols - 1) / kTileCols;
    fetch(c0);
    commit(0);
    __syncthreads();
    for (int64_t t = 0; t < ntiles; ++t) {
        const int buf = (int)(t & 1);
        const int64_t jt = c0 + t * kTileCols;
        if (t + 1 < ntiles)
            fetch(jt + kTileCols);                  // in flight during compute
        const bool diag = (wrow0 >= jt) && (wrow0 < jt + kTileCols);
        const bool tail = jt + kTileCols > c1;
        // coordinate 4 s + g, tile column 16 q + m, swizzled by 16 g
        const float *tile = reinterpret_cast<const float *>(xs[buf]) + g * kTileCols;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            floatx4 cacc = {0.0f, 0.0f, 0.0f, 0.0f};
            const float *ap = tile + ((16 * q + m) ^ (16 * g));
#pragma unroll
            for (int s = 0; s < KS; ++s)
                cacc = __builtin_amdgcn_mfma_f32_16x16x4f32(ap[4 * s * kTileCols], bop[s],
                                                            cacc, 0, 0, 0);
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r)
                a[r] = exp2_fast(-fmaxf(cacc[r], 0.0f));
            const int64_t j0 = jt + 16 * q + 4 * g;    // this lane's columns
            if (diag || tail) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (j0 + r == i || j0 + r >= c1)
                        a[r] = 0.0f;
            }
            if (MODE == kStore || MODE == kStoreW) {
                float *ow = ot[wave] + m * kOutStride + 16 * q + 4 * g;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ow[r] = (MODE == kStoreW) ? a[r] * rs : a[r];
            }
            if (MODE == kStore || MODE == kDegree) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc += (double)a[r];
            } else if (MODE == kApply) {
                const double *vp = vs[buf] + 16 * q + 4 * g;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc = fma((double)a[r], vp[r], acc);
            }
        }
        if (MODE == kStore || MODE == kStoreW) {
            // the wave's 16 x 64 tile, 4 rows x 256 contiguous bytes per store
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int rr = 4 * u + (lane >> 4);
                const int cc = 4 * (lane & 15);
                const int64_t ii = wrow0 + rr;
                const int64_t jj = jt + cc;
                const float *src = ot[wave] + rr * kOutStride + cc;
                if (ii < n) {
                    float *dst = A + ii * lda + jj;
                    if (!tail || jj + 3 < c1) {
                        store4(dst, src[0], src[1], src[2], src[3]);
                    } else {
                        for (int e = 0; e < 4 && jj + e < c1; ++e)
                            dst[e] = src[e];
                    }
                }
            }
        }
        if (t + 1 < ntiles) {
            // the barrier ending the previous iteration ordered every wave's
            // reads of buffer buf ^ 1 before this write; this one orders the
            // write before the next tile's reads
            commit(buf ^ 1);
            __syncthreads();
        }
    }

    if (MODE == kStoreW)
        return;
    // the four lanes sharing a row (g = 0..3) hold disjoint columns
    acc += __shfl_xor(acc, 16, kWave);
    acc += __shfl_xor(acc, 32, kWave);
    if (part != nullptr) {
        // chunk partial, reduced in chunk order by chunk_reduce_kernel
        if (g == 0 && row_ok)
            part[(int64_t)blockIdx.y * n + i] = acc;
        return;
    }
    double yabs = 0.0;
    if (g == 0 && row_ok) {
        if (MODE == kApply) {
            const double di = degree_in[i];
            const double yi = (di == 0.0) ? 0.0 : acc / di;
            out[i] = yi;
            yabs = fabs(yi);
        } else if (out != nullptr) {
            out[i] = acc;
        }
    }
    if (MODE == kApply && partial != nullptr) {
        const double sum = block_sum<kMfmaThreads>(yabs, red);
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
    for (int64_t gi = threadIdx.x; gi < ngroups; gi += kThreads) {
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
            if ((MODE == kStore || MODE == kStoreW) && i < n) {
                float o[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    o[q] = (MODE == kStoreW) ? a[r][q] * rs[r] : a[r][q];
                float *dst = A + i * lda + j0;
                if (j0 + 3 < n) {
                    store4(dst, o[0], o[1], o[2], o[3]);
                } else {
                    for (int q = 0; q < 4 && j0 + q < n; ++q)
                        dst[q] = o[q];
                }
            }
            if (MODE != kStoreW) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    acc[r] = fma((double)a[r][q], vj[q], acc[r]);
            }
        }
    }

    if (MODE == kStoreW)
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

int ks_for(int d)
{
    const int need = (d + 2 + 3) / 4;          // augmented dimension / 4
    static const int sizes[] = {5, 6, 8, 10, 12, 14, 17, 20, 24, 28, 33};
    for (int s : sizes)
        if (s >= need)
            return s;
    return 33;
}

// Column chunks: enough workgroups to fill the chip when rows are few.
void chunking(int64_t n, int64_t *chunk_cols, int *nchunks)
{
    const int64_t groups = (n + kRowsPerGroup - 1) / kRowsPerGroup;
    int64_t want = (4096 + groups - 1) / groups;     // >= 4 workgroups per CU
    if (want < 1)
        want = 1;
    if (want > kMaxChunks)
        want = kMaxChunks;
    int64_t cols = (n + want - 1) / want;
    cols = (cols + kTileCols - 1) / kTileCols * kTileCols;
    *chunk_cols = cols;
    *nchunks = (int)((n + cols - 1) / cols);
}

constexpr int kMaxKP = 4 * 33;               // largest augmented dimension

int64_t padded_points(int64_t n) { return (n + kTileCols - 1) / kTileCols * kTileCols; }

int64_t al256(int64_t x) { return (x + 255) & ~(int64_t)255; }

struct Ws {
    float *xa;
    float *xb;
    double *part;
};

// [xa: np * kMaxKP floats][xb: same][per-chunk row sums: kMaxChunks * n]
Ws carve(void *ws, int64_t n)
{
    char *b = static_cast<char *>(ws);
    const int64_t ob = al256(padded_points(n) * kMaxKP * 4);
    Ws w;
    w.xa = reinterpret_cast<float *>(b);
    w.xb = reinterpret_cast<float *>(b + ob);
    w.part = reinterpret_cast<double *>(b + 2 * ob);
    return w;
}

template <int MODE>
hipError_t dispatch(const float *X, int64_t n, int d, float c, float *A,
                    int64_t lda, const double *v, const double *degree_in,
                    double *out, double *partial, StopCtl ctl, int use_ctl,
                    void *ws, hipStream_t s, bool operands_ready = false)
{
    if (use_mfma(d)) {
        const Ws w = carve(ws, n);
        const int ks = ks_for(d);
        const int64_t np = padded_points(n);
        if (!operands_ready)
            hipLaunchKernelGGL(augment_kernel,
                               dim3((unsigned)((np + kThreads - 1) / kThreads)),
                               dim3(kThreads), 0, s, X, n, np, d, 4 * ks, c, w.xa, w.xb);
        int64_t chunk_cols;
        int nchunks;
        chunking(n, &chunk_cols, &nchunks);
        const bool sums = (MODE != kStoreW) && (MODE != kStore || out != nullptr);
        double *part = (sums && nchunks > 1) ? w.part : nullptr;
        const dim3 grid((unsigned)((n + kRowsPerGroup - 1) / kRowsPerGroup),
                        (unsigned)nchunks);
#define GPIC_MFMA(KS)                                                          \
    hipLaunchKernelGGL((affinity_mfma_kernel<KS, MODE>), grid, dim3(kMfmaThreads), 0, \
                       s, w.xa, np, w.xb, n, chunk_cols, A, lda, v, degree_in,   \
                       out, part, partial, ctl, use_ctl)
        switch (ks) {
        case 5: GPIC_MFMA(5); break;
        case 6: GPIC_MFMA(6); break;
        case 8: GPIC_MFMA(8); break;
        case 10: GPIC_MFMA(10); break;
        case 12: GPIC_MFMA(12); break;
        case 14: GPIC_MFMA(14); break;
        case 17: GPIC_MFMA(17); break;
        case 20: GPIC_MFMA(20); break;
        case 24: GPIC_MFMA(24); break;
        case 28: GPIC_MFMA(28); break;
        default: GPIC_MFMA(33); break;
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
    return (size_t)(2 * al256(padded_points(n) * kMaxKP * 4) +
                    al256((int64_t)kMaxChunks * n * 8));
}

int64_t fused_blocks(int64_t n, int d)
{
    if (!use_mfma(d))
        return (n + 7) / 8;
    int64_t chunk_cols;
    int nchunks;
    chunking(n, &chunk_cols, &nchunks);
    if (nchunks > 1)
        return (n + kThreads - 1) / kThreads;        // chunk_reduce workgroups
    return (n + kRowsPerGroup - 1) / kRowsPerGroup;  // tile workgroups
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
    const Ws w = carve(ws, n);
    const int64_t np = padded_points(n);
    hipLaunchKernelGGL(augment_kernel, dim3((unsigned)((np + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, s, X, n, np, d, 4 * ks_for(d), c, w.xa, w.xb);
    return hipGetLastError();
}

hipError_t launch_fused_apply(const float *X, int64_t n, int d, float c,
                              const double *v, const double *degree, double *y,
                              double *partial, StopCtl ctl, bool use_ctl,
                              void *ws, hipStream_t s, bool operands_ready)
{
    return dispatch<kApply>(X, n, d, c, nullptr, 0, v, degree, y, partial, ctl,
                            use_ctl ? 1 : 0, ws, s, operands_ready);
}

} // namespace gpic
