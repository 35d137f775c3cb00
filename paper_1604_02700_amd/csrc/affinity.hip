// Gaussian affinity tiles for gfx950, and the fused operator built on them.
//
// A_ij = exp(-||x_i - x_j||^2 / (2 sigma^2)) for i != j, A_ii = 0: the
// affinity matrix of section "Spectral Cluster" (AffinityMatrix step of
// Algorithm 2) with the Gaussian kernel read in for it.  The exponential is
// evaluated as exp2(-c * dist2) with c = log2(e) / (2 sigma^2), formed in
// float64 on the host and rounded once to float32.
//
// Two tile engines share one outer structure (a workgroup owns a block of
// rows and walks every column, so row sums are complete inside it):
//   * VALU, d < 16: squared distances from coordinate differences.
//   * MFMA, d >= 16: dist2 = |x_i|^2 + |x_j|^2 - 2 x_i.x_j with the Gram
//     product on the fp32 matrix cores (v_mfma_f32_16x16x4f32), clamped at 0.
// Three epilogues (template MODE):
//   kStore : write A (float32) and optionally the float64 row sums,
//   kApply : y_i = (sum_j A_ij v_j) / d_i, W = D^-1 A never stored (the
//            Multiply step with the affinity recomputed), plus per-block
//            partial sums of |y_i| for the L1 norm,
//   kDegree: d_i = sum_j A_ij with nothing of size n^2 written.
#include "common.h"

namespace gpic {
namespace {

enum { kStore = 0, kApply = 1, kDegree = 2 };

constexpr int kThreads = 256;

typedef float floatx4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ VALU

// Block: 256 threads, RB rows; each thread takes groups of 4 consecutive
// columns (one float4 store per row), stepping by 1024 columns.
template <int D, int RB, int MODE>
__global__ __launch_bounds__(kThreads) void affinity_valu_kernel(
    const float *__restrict__ X, int64_t n, int dyn_d, float c,
    float *__restrict__ A, int64_t lda, const double *__restrict__ v,
    const double *__restrict__ degree_in, double *__restrict__ out,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
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
#pragma unroll
    for (int r = 0; r < RB; ++r)
        acc[r] = 0.0;

    const int64_t ngroups = (n + 3) >> 2;
    for (int64_t g = threadIdx.x; g < ngroups; g += kThreads) {
        const int64_t j0 = g << 2;
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
#pragma unroll
            for (int r = 0; r < RB; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float s = 0.0f;
#pragma unroll
                    for (int k = 0; k < DR; ++k) {
                        const float df = xi[r][k] - xj[q][k];
                        s = fmaf(df, df, s);
                    }
                    a[r][q] = exp2f(-c * s);
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
                    for (int k = 0; k < d; ++k) {
                        const float df = X[i * d + k] - X[j * d + k];
                        s = fmaf(df, df, s);
                    }
                    a[r][q] = exp2f(-c * s);
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
            if (MODE == kStore && i < n) {
                float *dst = A + i * lda + j0;
                if (j0 + 3 < n) {
                    *reinterpret_cast<float4 *>(dst) =
                        make_float4(a[r][0], a[r][1], a[r][2], a[r][3]);
                } else {
                    for (int q = 0; q < 4 && j0 + q < n; ++q)
                        dst[q] = a[r][q];
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[r] = fma((double)a[r][q], vj[q], acc[r]);
        }
    }

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

// ------------------------------------------------------------------ MFMA

// Block: 4 waves x 16 rows = 64 rows.  The block walks the columns in
// tiles of 64 staged in LDS (points, their squared norms and, for kApply,
// v); every wave forms four 16x16 Gram sub-tiles per column tile.
//
// v_mfma_f32_16x16x4f32 operand layout (lane l, g = l / 16):
//   A operand : element (m = l % 16, k = g)
//   B operand : element (k = g,      n = l % 16)
//   result    : elements (m = 4 g + r, n = l % 16), r = 0..3
// The A operand carries 16 columns j of the affinity and the B operand the
// wave's 16 rows i, so the result gives every lane one row i and four
// consecutive columns: one float4 store per lane.  The k slot g of K-step s
// holds coordinate g * KS + s, so each lane reads KS consecutive
// coordinates of a point (vector loads from LDS and HBM).
constexpr int kRowsPerWave = 16;
constexpr int kTileCols = 64;

template <int KS, int MODE>
__global__ __launch_bounds__(kThreads) void affinity_mfma_kernel(
    const float *__restrict__ X, int64_t n, int d, float c,
    float *__restrict__ A, int64_t lda, const double *__restrict__ v,
    const double *__restrict__ degree_in, double *__restrict__ out,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    constexpr int DP = 4 * KS;       // padded dimension
    constexpr int LS = DP + 4;       // LDS row stride (floats), 16 B aligned
    __shared__ __attribute__((aligned(16))) float xs[kTileCols * LS];
    __shared__ __attribute__((aligned(16))) float ns[kTileCols];
    __shared__ __attribute__((aligned(16))) double vs[kTileCols];
    __shared__ double red[kThreads / kWave];

    if (MODE == kApply && use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int g = lane >> 4;
    const int m = lane & 15;
    const int64_t i = (int64_t)blockIdx.x * (4 * kRowsPerWave) +
                      wave * kRowsPerWave + m;
    const int64_t ic = (i < n) ? i : n - 1;

    // B operand: the row's coordinates g*KS .. g*KS+KS-1 (zero padded) and
    // the row's squared norm (sequential float32 sum, same order as ns[]).
    float bop[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int k = g * KS + s;
        bop[s] = (k < d) ? X[ic * d + k] : 0.0f;
    }
    float ni = 0.0f;
    for (int k = 0; k < d; ++k) {
        const float x = X[ic * d + k];
        ni = fmaf(x, x, ni);
    }

    double acc = 0.0;
    const int64_t ntiles = (n + kTileCols - 1) / kTileCols;
    for (int64_t t = 0; t < ntiles; ++t) {
        const int64_t jt = t * kTileCols;
        __syncthreads();
        // stage the column tile: 64 points x DP coordinates
        for (int e = threadIdx.x; e < kTileCols * DP; e += kThreads) {
            const int cj = e / DP, k = e % DP;
            const int64_t j = (jt + cj < n) ? jt + cj : n - 1;
            xs[cj * LS + k] = (k < d) ? X[j * d + k] : 0.0f;
        }
        if (MODE == kApply && threadIdx.x < kTileCols) {
            const int64_t j = jt + threadIdx.x;
            vs[threadIdx.x] = (j < n) ? v[j] : 0.0;
        }
        __syncthreads();
        if (threadIdx.x < kTileCols) {
            float s = 0.0f;
            for (int k = 0; k < d; ++k) {
                const float x = xs[threadIdx.x * LS + k];
                s = fmaf(x, x, s);
            }
            ns[threadIdx.x] = s;
        }
        __syncthreads();

#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float *ap = xs + (q * 16 + m) * LS + g * KS;
            floatx4 cacc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int s = 0; s < KS; ++s)
                cacc = __builtin_amdgcn_mfma_f32_16x16x4f32(ap[s], bop[s], cacc,
                                                            0, 0, 0);
            const int cbase = q * 16 + 4 * g;           // column within tile
            const float4 nj = *reinterpret_cast<const float4 *>(ns + cbase);
            const float njr[4] = {nj.x, nj.y, nj.z, nj.w};
            float a[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float d2 = ni + njr[r] - 2.0f * cacc[r];
                d2 = fmaxf(d2, 0.0f);
                const int64_t j = jt + cbase + r;
                a[r] = (j == i || j >= n) ? 0.0f : exp2f(-c * d2);
            }
            const int64_t j0 = jt + cbase;
            if (MODE == kStore) {
                if (i < n) {
                    float *dst = A + i * lda + j0;
                    if (j0 + 3 < n) {
                        *reinterpret_cast<float4 *>(dst) =
                            make_float4(a[0], a[1], a[2], a[3]);
                    } else {
                        for (int r = 0; r < 4 && j0 + r < n; ++r)
                            dst[r] = a[r];
                    }
                }
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc += (double)a[r];
            } else if (MODE == kDegree) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc += (double)a[r];
            } else {
                const double2 v01 = *reinterpret_cast<const double2 *>(vs + cbase);
                const double2 v23 = *reinterpret_cast<const double2 *>(vs + cbase + 2);
                acc = fma((double)a[0], v01.x, acc);
                acc = fma((double)a[1], v01.y, acc);
                acc = fma((double)a[2], v23.x, acc);
                acc = fma((double)a[3], v23.y, acc);
            }
        }
    }

    // the four lanes sharing a row (g = 0..3) hold disjoint columns
    acc += __shfl_xor(acc, 16, kWave);
    acc += __shfl_xor(acc, 32, kWave);
    double yabs = 0.0;
    if (g == 0 && i < n) {
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
        // rows of the block in ascending order: lanes 0..15 of each wave,
        // then the waves in order
        const double s = block_sum<kThreads>(yabs, red);
        if (threadIdx.x == 0)
            partial[blockIdx.x] = s;
    }
}

template <int MODE>
hipError_t dispatch(const float *X, int64_t n, int d, float c, float *A,
                    int64_t lda, const double *v, const double *degree_in,
                    double *out, double *partial, StopCtl ctl, int use_ctl,
                    hipStream_t s)
{
    const dim3 block(kThreads);
    if (d >= 16 && d <= 128) {
        const dim3 grid((unsigned)((n + 63) / 64));
        const int ks = (d + 3) / 4;
#define GPIC_MFMA(KS)                                                          \
    hipLaunchKernelGGL((affinity_mfma_kernel<KS, MODE>), grid, block, 0, s, X, \
                       n, d, c, A, lda, v, degree_in, out, partial, ctl,      \
                       use_ctl)
        if (ks <= 4) GPIC_MFMA(4);
        else if (ks <= 8) GPIC_MFMA(8);
        else if (ks <= 16) GPIC_MFMA(16);
        else GPIC_MFMA(32);
#undef GPIC_MFMA
        return hipGetLastError();
    }
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

} // namespace

int64_t fused_blocks(int64_t n, int d)
{
    if (d >= 16 && d <= 128)
        return (n + 63) / 64;
    return (n + 7) / 8;
}

hipError_t launch_affinity(const float *X, int64_t n, int d, float c, float *A,
                           int64_t lda, double *degree, hipStream_t s)
{
    StopCtl none{};
    return dispatch<kStore>(X, n, d, c, A, lda, nullptr, nullptr, degree,
                            nullptr, none, 0, s);
}

hipError_t launch_fused_degree(const float *X, int64_t n, int d, float c,
                               double *degree, hipStream_t s)
{
    StopCtl none{};
    return dispatch<kDegree>(X, n, d, c, nullptr, 0, nullptr, nullptr, degree,
                             nullptr, none, 0, s);
}

hipError_t launch_fused_apply(const float *X, int64_t n, int d, float c,
                              const double *v, const double *degree, double *y,
                              double *partial, StopCtl ctl, bool use_ctl,
                              hipStream_t s)
{
    return dispatch<kApply>(X, n, d, c, nullptr, 0, v, degree, y, partial, ctl,
                            use_ctl ? 1 : 0, s);
}

} // namespace gpic
