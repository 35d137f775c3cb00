// Dense product over symmetric tile storage for gfx950: y = D^-1 (A v),
// the Multiply step of Algorithm 2's loop with W = D^-1 A and the
// affinity A of section "Spectral Cluster", which is symmetric.  Only the
// upper block triangle of A is stored, so a product streams 2 n^2 bytes
// instead of the 4 n^2 bytes of a dense W.
//
// Storage ("packed upper tiles"): the indices 0 .. n-1 are cut into
// nb = ceil(n / 256) blocks of 256; tile (I, J), I <= J, holds
// A[256 I + r][256 J + c] at r * 256 + c, and the tiles follow each other
// in the order (0,0), (0,1), .., (0,nb-1), (1,1), .., so tile (I, J)
// starts at entry 65536 (I nb - I (I - 1) / 2 + J - I).  Diagonal tiles
// hold the whole block.  Entries outside [0, n)^2 (the last block row and
// column when 256 does not divide n) are never written by the affinity
// and may hold anything, NaN included: the product of the last block row
// or column still loads whole tile rows, but replaces every value outside
// [0, n)^2 by 0 with a select (never a multiply by a mask) before it is
// used, so such padding cannot reach a sum.
//
// One workgroup per super-tile of 2 x 2 tiles: super-tile (R, S), R <= S,
// covers the blocks 2R, 2R + 1 (rows) and 2S, 2S + 1 (columns), and takes
// its stored tiles one after another.  Tile (I, J) gives the row sums
// A_IJ v_J to the rows of block I and, when I < J, the column sums
// A_IJ^T v_I to the rows of block J (A_JI = A_IJ^T); the workgroup adds
// them per row in LDS (tiles in the order (2R, 2S), (2R, 2S + 1),
// (2R + 1, 2S), (2R + 1, 2S + 1)) and writes 512 sums for the rows of
// super-row R to part[(R ns + S) 512 + .] and, when R < S, 512 for those of
// super-row S to part[(S ns + R) 512 + .] -- half the partial sums of one
// workgroup per tile.  A second launch adds, for every row i, the ns
// partials of its super-row (four slices summed in ascending order, then
// added in slice order), divides by d_i and writes per-workgroup partial
// sums of |y_i| for the L1 norm.  Every sum runs in a fixed order: bitwise
// reproducible.
#include "common.h"

namespace gpic {
namespace {

constexpr int kTile = 256;                 // tile edge (indices per block)
constexpr int kThreads = 256;              // four waves; a thread covers 32 rows x 8 columns
constexpr int64_t kTileEntries = (int64_t)kTile * kTile;
constexpr int kSuper = 2 * kTile;          // rows (and columns) of a super-tile

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __host__ __forceinline__ int64_t tile_start(int64_t I, int64_t nb)
{
    return I * nb - I * (I - 1) / 2;
}

// (I, J) of the t-th pair I <= J in the order (0,0), (0,1), .., (0,nb-1),
// (1,1), ..: I from the quadratic formula, corrected by at most a step
// either way against rounding.
__device__ __forceinline__ void tile_of(int64_t t, int64_t nb, int64_t *I, int64_t *J)
{
    const double b = (double)(2 * nb + 1);
    int64_t i = (int64_t)((b - sqrt(b * b - 8.0 * (double)t)) * 0.5);
    if (i < 0)
        i = 0;
    if (i > nb - 1)
        i = nb - 1;
    while (i > 0 && tile_start(i, nb) > t)
        --i;
    while (i + 1 < nb && tile_start(i + 1, nb) <= t)
        ++i;
    *I = i;
    *J = i + (t - tile_start(i, nb));
}

// The float64 of lane (lane xor K), K < 32: data-parallel moves for K = 1,
// 2, 8 (quad permutations, a rotation by 8 within a row of 16), swizzles for
// K = 4, 16, on the two halves of the value.
template <int K>
__device__ __forceinline__ double dxor(double x)
{
    const long long b = __double_as_longlong(x);
    int lo = (int)(b & 0xffffffffll), hi = (int)(b >> 32);
    if (K == 1) {
        lo = __builtin_amdgcn_mov_dpp(lo, 0xb1, 0xf, 0xf, false);
        hi = __builtin_amdgcn_mov_dpp(hi, 0xb1, 0xf, 0xf, false);
    } else if (K == 2) {
        lo = __builtin_amdgcn_mov_dpp(lo, 0x4e, 0xf, 0xf, false);
        hi = __builtin_amdgcn_mov_dpp(hi, 0x4e, 0xf, 0xf, false);
    } else if (K == 4) {
        lo = __builtin_amdgcn_ds_swizzle(lo, 0x101f);
        hi = __builtin_amdgcn_ds_swizzle(hi, 0x101f);
    } else if (K == 8) {
        lo = __builtin_amdgcn_mov_dpp(lo, 0x128, 0xf, 0xf, false);
        hi = __builtin_amdgcn_mov_dpp(hi, 0x128, 0xf, 0xf, false);
    } else {
        lo = __builtin_amdgcn_ds_swizzle(lo, 0x401f);
        hi = __builtin_amdgcn_ds_swizzle(hi, 0x401f);
    }
    return __longlong_as_double(((long long)(unsigned)hi << 32) | (long long)(unsigned)lo);
}

// Thread (ty, tx) = (t / 32, t % 32) owns the columns 128 q + 4 tx + e
// (q = 0, 1; e = 0..3) of the tile and, in pass p = 0..3, the rows
// 64 p + 8 ty + k (k = 0..7): per row and q the 32 lanes of a row group
// read 512 contiguous bytes.  Row partials (over the thread's 8 columns,
// q then e ascending) are reduce-scattered over the 32 lanes after each
// pass; column partials (over the thread's 32 rows, ascending) are carried
// over the passes and reduced once at the end, over the wave's two row
// groups and through LDS over the 4 waves.  v is read from global memory
// (it stays in the caches), so the first loads of the tile issue at once.
// All eight rows of a pass are loaded before any is used (16 loads of 16
// bytes in flight per thread): at 236 registers, two workgroups per compute
// unit, this streams faster than two rows in flight at 116 registers and
// four workgroups (measured, n = 50,000: 799 against 831 us per product).
template <bool EDGE>
__device__ __forceinline__ void sym_tile(const float *__restrict__ T, int64_t I, int64_t J,
                                         int64_t n, const double *__restrict__ v,
                                         double (*cred)[kTile], double *__restrict__ racc_l,
                                         double *__restrict__ cacc_l)
{
    const int tid = threadIdx.x;
    const int tx = tid & 31;
    const int ty = tid >> 5;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int64_t cI = kTile * I, cJ = kTile * J;
    double vj[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        const int64_t col = cJ + 128 * (c >> 2) + 4 * tx + (c & 3);
        vj[c] = (!EDGE || col < n) ? (v != nullptr ? v[col] : 1.0) : 0.0;
    }
    double cacc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
        cacc[c] = 0.0;
    const floatx4 *base = reinterpret_cast<const floatx4 *>(T) + (8 * ty) * (kTile / 4) + tx;
#pragma unroll 1
    for (int p = 0; p < 4; ++p) {
        double racc[8];
#pragma unroll
        for (int k = 0; k < 8; ++k)
            racc[k] = 0.0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const floatx4 *rp = base + (64 * p + k) * (kTile / 4);
            const floatx4 w0 = __builtin_nontemporal_load(rp);
            const floatx4 w1 = __builtin_nontemporal_load(rp + 32);
            const int64_t row = cI + 64 * p + 8 * ty + k;
            const bool rowok = !EDGE || row < n;
            const double vi = rowok ? (v != nullptr ? v[row] : 1.0) : 0.0;
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                float af = (c < 4) ? w0[c & 3] : w1[c & 3];
                if (EDGE && !(rowok && cJ + 128 * (c >> 2) + 4 * tx + (c & 3) < n))
                    af = 0.0f;
                const double a = (double)af;
                racc[k] = fma(a, vj[c], racc[k]);
                cacc[c] = fma(a, vi, cacc[c]);
            }
        }
        // rows: after m = 16, 8, 4 lane tx holds row 4 b4 + 2 b3 + b2 of the
        // group (b = the bits of tx), summed over the 8 lanes sharing those
        // bits; m = 2, 1 add the remaining 4 lanes
        {
            const bool up = (tx & 16) != 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const double send = up ? racc[q] : racc[q + 4];
                const double keep = up ? racc[q + 4] : racc[q];
                racc[q] = keep + dxor<16>(send);
            }
        }
        {
            const bool up = (tx & 8) != 0;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const double send = up ? racc[q] : racc[q + 2];
                const double keep = up ? racc[q + 2] : racc[q];
                racc[q] = keep + dxor<8>(send);
            }
        }
        {
            const bool up = (tx & 4) != 0;
            const double send = up ? racc[0] : racc[1];
            const double keep = up ? racc[1] : racc[0];
            racc[0] = keep + dxor<4>(send);
        }
        double rs = racc[0];
        rs = rs + dxor<2>(rs);
        rs = rs + dxor<1>(rs);
        if ((tx & 3) == 0) {
            const int r = 4 * ((tx >> 4) & 1) + 2 * ((tx >> 3) & 1) + ((tx >> 2) & 1);
            racc_l[64 * p + 8 * ty + r] += rs;       // this lane's slot in every tile
        }
    }
    if (I == J)
        return;                                  // uniform over the workgroup

    // columns: over the wave's two row groups (lanes 32 apart) ...
    const int b1 = (lane >> 5) & 1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const double send = b1 ? cacc[q] : cacc[q + 4];
        const double keep = b1 ? cacc[q + 4] : cacc[q];
        cacc[q] = keep + __shfl_xor(send, 32, kWave);
    }
    // ... this lane now holds the columns 128 b1 + 4 tx + e
#pragma unroll
    for (int e = 0; e < 4; ++e)
        cred[wave][128 * b1 + 4 * tx + e] = cacc[e];
    __syncthreads();
    // ... then over the four waves, in wave order
    const double s = ((cred[0][tid] + cred[1][tid]) + cred[2][tid]) + cred[3][tid];
    cacc_l[tid] += s;
    __syncthreads();                             // cred is reused by the next tile
}

__global__ __launch_bounds__(kThreads) void sym_gemv_kernel(
    const float *__restrict__ As, int64_t n, int64_t nb, const double *__restrict__ v,
    double *__restrict__ part, StopCtl ctl, int use_ctl)
{
    __shared__ double cred[kThreads / kWave][kTile];
    __shared__ double acc[4][kTile];              // rows of blocks 2R, 2R+1, 2S, 2S+1
    if (use_ctl) {
        if (blockIdx.x == 0 && threadIdx.x == 0)
            *ctl.cur_stat = 0.0;
        if (stop_reached(ctl))
            return;
    }
    const int64_t ns = (nb + 1) / 2;
    int64_t R, S;
    tile_of((int64_t)blockIdx.x, ns, &R, &S);
    for (int q = 0; q < 4; ++q)
        acc[q][threadIdx.x] = 0.0;
    __syncthreads();
    // the stored tiles of the super-tile, in a fixed order; on the diagonal
    // (R = S) the tile (2R + 1, 2R) is not stored, and the column sums of
    // (2R, 2R + 1) go to block 2R + 1, whose rows sit in acc[1]
#pragma unroll 1
    for (int u = 0; u < 4; ++u) {
        const int64_t I = 2 * R + (u >> 1), J = 2 * S + (u & 1);
        if (I >= nb || J >= nb || I > J)
            continue;                            // uniform over the workgroup
        const float *T = As + (tile_start(I, nb) + (J - I)) * kTileEntries;
        double *ra = acc[u >> 1];
        double *ca = (R == S) ? acc[1] : acc[2 + (u & 1)];
        if (kTile * (J + 1) > n)                 // J >= I: the last block column
            sym_tile<true>(T, I, J, n, v, cred, ra, ca);
        else
            sym_tile<false>(T, I, J, n, v, cred, ra, ca);
    }
    __syncthreads();
    for (int q = 0; q < 2; ++q)
        part[(R * ns + S) * kSuper + q * kTile + threadIdx.x] = acc[q][threadIdx.x];
    if (R < S)
        for (int q = 0; q < 2; ++q)
            part[(S * ns + R) * kSuper + q * kTile + threadIdx.x] = acc[2 + q][threadIdx.x];
}

// y_i = (sum over K of part[(R ns + K) 512 + 256 (I - 2R) + r]) / d_i for
// row i = 256 I + r of super-row R = I / 2; one workgroup of 4 x 256
// threads per block of 256 rows: slice s sums K = s, s + 4, .. (eight loads
// in flight), then the four slices are added in slice order.
constexpr int kSlices = 4;

__global__ __launch_bounds__(kThreads * kSlices) void sym_finalize_kernel(
    const double *__restrict__ part, int64_t n, int64_t nb,
    const double *__restrict__ degree, double *__restrict__ y,
    double *__restrict__ partial, StopCtl ctl, int use_ctl)
{
    __shared__ double sl[kSlices][kThreads];
    __shared__ double red[kThreads * kSlices / kWave];
    if (use_ctl && stop_reached(ctl))
        return;
    const int r = threadIdx.x % kThreads;
    const int sidx = threadIdx.x / kThreads;
    const int64_t I = blockIdx.x;
    const int64_t ns = (nb + 1) / 2;
    const double *p = part + (I / 2) * ns * kSuper + (I % 2) * kTile + r;
    double s = 0.0;
    int64_t K = sidx;
    for (; K + 7 * kSlices < ns; K += 8 * kSlices) {
        double x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            x[u] = p[(K + u * kSlices) * kSuper];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            s += x[u];
    }
    for (; K < ns; K += kSlices)
        s += p[K * kSuper];
    sl[sidx][r] = s;
    __syncthreads();
    const int64_t i = kTile * I + r;
    double yabs = 0.0;
    if (sidx == 0 && i < n) {
        const double t = ((sl[0][r] + sl[1][r]) + sl[2][r]) + sl[3][r];
        if (degree == nullptr) {
            y[i] = t;                            // the row sums themselves
        } else {
            const double di = degree[i];
            const double yi = (di == 0.0) ? 0.0 : t / di;
            y[i] = yi;
            yabs = fabs(yi);
        }
    }
    // every wave takes part; those of slices 1..3 add zeros
    const double sum = block_sum<kThreads * kSlices>(yabs, red);
    if (threadIdx.x == 0 && partial != nullptr)
        partial[blockIdx.x] = sum;
}

} // namespace

int64_t sym_blocks(int64_t n) { return (n + kTile - 1) / kTile; }

size_t sym_storage_bytes(int64_t n)
{
    const int64_t nb = sym_blocks(n);
    return (size_t)(nb * (nb + 1) / 2) * (size_t)kTileEntries * sizeof(float);
}

size_t sym_part_bytes(int64_t n)
{
    const int64_t ns = (sym_blocks(n) + 1) / 2;
    return (size_t)(ns * ns * kSuper) * sizeof(double);
}

hipError_t launch_sym_gemv(const float *As, int64_t n, const double *degree,
                           const double *v, double *y, double *part, double *partial,
                           StopCtl ctl, bool use_ctl, hipStream_t s)
{
    const int64_t nb = sym_blocks(n);
    const int64_t ns = (nb + 1) / 2;
    hipLaunchKernelGGL(sym_gemv_kernel, dim3((unsigned)(ns * (ns + 1) / 2)), dim3(kThreads),
                       0, s, As, n, nb, v, part, ctl, use_ctl ? 1 : 0);
    hipLaunchKernelGGL(sym_finalize_kernel, dim3((unsigned)nb), dim3(kThreads * kSlices), 0,
                       s, part,
                       n, nb, degree, y, partial, ctl, use_ctl ? 1 : 0);
    return hipGetLastError();
}

} // namespace gpic
