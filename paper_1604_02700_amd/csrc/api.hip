// libgpic C ABI: host-side validation, workspace layout and the
// power-iteration driver (Algorithm 1's loop) over the kernels of the other
// translation units.  Nothing here computes on the host; every step of the
// method runs in the HIP kernels.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>

#include "../../include/gpic.h"
#include "common.h"

namespace gpic {

namespace {
thread_local std::string g_last_error;
} // namespace

const char *last_error_text() { return g_last_error.c_str(); }

void set_error(const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

} // namespace gpic

using namespace gpic;

namespace {

constexpr int64_t kMaxN = 2147483647LL;     // indices are int32 in places
constexpr int64_t kMaxKmeansN = 1LL << 30;  // the split-point recursion indexes nodes in 32 bits
constexpr int64_t kRing = 1024;             // statistic slots on the device
constexpr int64_t kMaxSymN = 1LL << 24;     // one workgroup per stored tile: < 2^31 tiles
constexpr size_t kCtlBytes = 256;           // err @0, tau @8, csr flag @16

inline size_t al(size_t x) { return (x + 255) & ~(size_t)255; }

inline bool aligned(const void *p, size_t a)
{
    return ((uintptr_t)p % a) == 0;
}

gpic_status fail(gpic_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    set_error("%s", buf);
    return st;
}

gpic_status hip_fail(hipError_t e, const char *where)
{
    return fail(GPIC_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

#define CHECK_ARG(cond, ...)                                                   \
    do {                                                                       \
        if (!(cond))                                                           \
            return fail(GPIC_ERR_INVALID_ARG, __VA_ARGS__);                    \
    } while (0)

#define CHECK_HIP(expr, where)                                                 \
    do {                                                                       \
        hipError_t e_ = (expr);                                                \
        if (e_ != hipSuccess)                                                  \
            return hip_fail(e_, where);                                        \
    } while (0)

size_t start_ws(int64_t n) { return al(start_vector_ws(n)); }
size_t aff_ws(int64_t n) { return al(affinity_ws(n)); }

// [ctl][statistic ring][|y| partials nb][y n][delta n], and for the
// one-launch dense update (small n) a second partials and y buffer
size_t pi_ws(int64_t n, int64_t nb)
{
    const size_t pipe = gemv_pipe_applies(n) ? al((size_t)nb * 8) + al((size_t)n * 8) : 0;
    return kCtlBytes + al(kRing * 8) + al((size_t)nb * 8) + 2 * al((size_t)n * 8) + pipe;
}

int64_t fused_nb_bound(int64_t n) { return (n + 7) / 8; }

// the column-blocked copy of a CSR W follows the power-iteration layout
size_t pi_csr_ws(int64_t n, int64_t nnz)
{
    return pi_ws(n, spmv_blocks(n)) + al(csr_blocked_ws(n, nnz));
}

// the fused product's own scratch follows the power-iteration layout
size_t pi_fused_ws(int64_t n) { return pi_ws(n, fused_nb_bound(n)) + al(fused_ws(n)); }

// A into the symmetric storage, then its row sums by the symmetric product:
// the affinity scratch, reused for the product's partial sums
size_t sym_aff_ws(int64_t n)
{
    const size_t a = aff_ws(n), b = al(sym_part_bytes(n));
    return a > b ? a : b;
}

// the symmetric product's partial sums follow the power-iteration layout
size_t pi_sym_ws(int64_t n) { return pi_ws(n, sym_blocks(n)) + al(sym_part_bytes(n)); }

// Out-of-core dense path: two staging buffers of P rows (P a multiple of
// 4, the dense product's rows per workgroup) with a row pitch of n rounded
// up to 4 floats follow the power-iteration layout.
constexpr int64_t kHostPanelBytes = 64ll << 20;     // default panel: 64 MiB
int64_t host_pitch(int64_t n) { return (n + 3) & ~(int64_t)3; }
size_t host_panel_bytes(int64_t n, int64_t P) { return al((size_t)(P * host_pitch(n)) * 4); }
int64_t host_default_rows(int64_t n)
{
    int64_t P = kHostPanelBytes / (host_pitch(n) * 4) / 4 * 4;
    const int64_t all = (n + 3) & ~(int64_t)3;
    if (P < 4)
        P = 4;
    return P < all ? P : all;
}
size_t pi_host_base(int64_t n) { return pi_ws(n, gemv_blocks(n)); }
size_t pi_host_ws(int64_t n)
{
    return pi_host_base(n) + 2 * host_panel_bytes(n, host_default_rows(n));
}

// exp(-x / (2 sigma^2)) = exp2(-c x) with c = log2(e) / (2 sigma^2)
bool gauss_coefficient(float sigma, float *c)
{
    const double s = (double)sigma;
    const double cc = 1.4426950408889634074 / (2.0 * s * s);
    *c = (float)cc;
    return isfinite(*c) && *c > 0.0f;
}

gpic_status check_coords(const float *X, int64_t n, int32_t d)
{
    CHECK_ARG(X != nullptr, "X is null");
    CHECK_ARG(aligned(X, 4), "X must be 4-byte aligned");
    CHECK_ARG(n >= 2 && n <= kMaxN, "n = %lld out of range [2, 2^31-1]", (long long)n);
    CHECK_ARG(d >= 1, "d = %d must be >= 1", d);
    return GPIC_OK;
}

gpic_status check_points(const float *X, int64_t n, int32_t d, float sigma)
{
    gpic_status st = check_coords(X, n, d);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(isfinite(sigma) && sigma > 0.0f, "sigma must be finite and > 0");
    float c;
    CHECK_ARG(gauss_coefficient(sigma, &c), "sigma too small (1/(2 sigma^2) overflows)");
    return GPIC_OK;
}

gpic_status check_vec(const void *p, const char *name, bool nullable = false)
{
    if (p == nullptr) {
        if (nullable)
            return GPIC_OK;
        return fail(GPIC_ERR_INVALID_ARG, "%s is null", name);
    }
    if (!aligned(p, 16))
        return fail(GPIC_ERR_INVALID_ARG, "%s must be 16-byte aligned", name);
    return GPIC_OK;
}

gpic_status check_ws(void *ws, size_t have, size_t need)
{
    if (need == 0)
        return GPIC_OK;
    if (ws == nullptr || have < need)
        return fail(GPIC_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given",
                    need, ws == nullptr ? (size_t)0 : have);
    if (!aligned(ws, 256))
        return fail(GPIC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    return GPIC_OK;
}

gpic_status check_params(const gpic_pi_params *p)
{
    CHECK_ARG(p != nullptr, "params is null");
    CHECK_ARG(p->mode == GPIC_MODE_FIXED || p->mode == GPIC_MODE_CONVERGE,
              "mode %d is not FIXED (0) or CONVERGE (1)", p->mode);
    CHECK_ARG(p->max_iter >= 0, "max_iter must be >= 0");
    CHECK_ARG(!(p->eps < 0.0) && !isnan(p->eps), "eps must be >= 0");
    CHECK_ARG(p->check_every >= 0, "check_every must be >= 0");
    CHECK_ARG(p->reserved == 0, "reserved must be 0");
    return GPIC_OK;
}

gpic_status check_csr(const int64_t *row_ptr, const int32_t *col,
                      const void *val, int64_t n, int64_t nnz)
{
    CHECK_ARG(row_ptr != nullptr && col != nullptr && val != nullptr,
              "CSR arrays must not be null");
    CHECK_ARG(aligned(row_ptr, 8) && aligned(col, 4) && aligned(val, 4),
              "CSR arrays misaligned");
    CHECK_ARG(n >= 2 && n <= kMaxN, "n = %lld out of range", (long long)n);
    CHECK_ARG(nnz >= 0, "nnz must be >= 0");
    return GPIC_OK;
}

// Device-side structural check of a CSR graph (row_ptr monotone from 0 to
// nnz, columns in range) before any kernel indexes through it.
gpic_status verify_csr(const int64_t *row_ptr, const int32_t *col, int64_t n,
                       int64_t nnz, void *ws, hipStream_t s)
{
    int *flag = reinterpret_cast<int *>(static_cast<char *>(ws) + 16);
    int bad = 0;
    CHECK_HIP(launch_csr_check(row_ptr, col, n, nnz, flag, s, &bad), "csr check");
    if (bad)
        return fail(GPIC_ERR_INVALID_ARG,
                    "CSR structure invalid (row_ptr not monotone from 0 to nnz, "
                    "or a column outside [0, n))");
    return GPIC_OK;
}

// The product of one update: y = W v, with per-block partial |y| sums.
struct Product {
    virtual ~Product() {}
    virtual int64_t blocks() const = 0;
    virtual hipError_t launch(const double *v, double *y, double *partial,
                              StopCtl ctl, hipStream_t s) const = 0;
    // one launch per update (the previous iteration's tau and update, then
    // this iteration's product), where the operator offers it
    virtual bool pipelined() const { return false; }
    virtual hipError_t launch_pipe(double *, double *, const double *, const double *,
                                   double *, double *, bool, bool, double *, StopCtl,
                                   hipStream_t) const
    {
        return hipErrorNotSupported;
    }
};

struct DenseProduct : Product {
    const float *W;
    int64_t n, ldw;
    int64_t blocks() const override { return gemv_blocks(n); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        return launch_gemv(W, n, ldw, v, y, partial, ctl, true, s);
    }
    bool pipelined() const override { return gemv_pipe_applies(n); }
    hipError_t launch_pipe(double *v, double *delta, const double *y_prev,
                           const double *part_prev, double *y_cur, double *part_cur,
                           bool update, bool product, double *zero_slot, StopCtl ctl,
                           hipStream_t s) const override
    {
        return launch_gemv_pipe(W, n, ldw, v, delta, y_prev, part_prev, y_cur, part_cur, update,
                                product, zero_slot, ctl, s);
    }
};

struct CsrProduct : Product {
    const int64_t *row_ptr;
    const int32_t *col;
    const float *val;
    int64_t n, nnz;
    int64_t blocks() const override { return spmv_partials(n, nnz); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        return launch_spmv(row_ptr, col, val, n, nnz, v, y, partial, ctl, true, s);
    }
};

struct BlockedCsrProduct : Product {
    CsrBlocked B;
    int64_t blocks() const override { return csr_blocked_partials(B.n); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        return launch_spmv_blocked(B, v, y, partial, ctl, s);
    }
};

struct FusedProduct : Product {
    const float *X;
    int64_t n;
    int d;
    float c;
    const double *degree;
    void *scratch;
    int64_t blocks() const override { return fused_blocks(n, d); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        return launch_fused_apply(X, n, d, c, v, degree, y, partial, ctl, true,
                                  scratch, s, true);
    }
};

struct SymProduct : Product {
    const float *As;
    int64_t n;
    const double *degree;
    double *part;
    int64_t blocks() const override { return sym_blocks(n); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        return launch_sym_gemv(As, n, degree, v, y, part, partial, ctl, true, s);
    }
};

// Out-of-core product: W stays in host memory and every product streams it
// to the device in panels of P rows, alternating between two staging
// buffers: panel k is copied on a copy stream (waiting until the product
// that last read its buffer is done) and multiplied on the caller's stream
// (waiting for its copy), so the copy of one panel overlaps the product of
// the previous one.  Each panel's product writes its rows of y and its
// workgroups' |y| partials at their whole-matrix positions, so the results
// are bitwise those of the device-resident dense product.
struct HostDenseProduct : Product {
    const float *Wh;                 // host
    int64_t n, ldw, P, pitch;
    float *buf[2];
    hipStream_t cs;
    hipEvent_t copied[2], consumed[2];
    mutable int64_t seq = 0;         // panels issued so far
    int64_t blocks() const override { return gemv_blocks(n); }
    hipError_t launch(const double *v, double *y, double *partial, StopCtl ctl,
                      hipStream_t s) const override
    {
        for (int64_t r0 = 0; r0 < n; r0 += P) {
            const int64_t rows = (r0 + P < n) ? P : n - r0;
            const int b = (int)(seq & 1);
            hipError_t e;
            if (seq >= 2 && (e = hipStreamWaitEvent(cs, consumed[b], 0)) != hipSuccess)
                return e;
            if ((e = hipMemcpy2DAsync(buf[b], (size_t)pitch * 4, Wh + r0 * ldw,
                                      (size_t)ldw * 4, (size_t)n * 4, (size_t)rows,
                                      hipMemcpyHostToDevice, cs)) != hipSuccess ||
                (e = hipEventRecord(copied[b], cs)) != hipSuccess ||
                (e = hipStreamWaitEvent(s, copied[b], 0)) != hipSuccess ||
                (e = launch_gemv_panel(buf[b], rows, n, pitch, v, y + r0, partial + r0 / 4,
                                       ctl, true, s)) != hipSuccess ||
                (e = hipEventRecord(consumed[b], s)) != hipSuccess)
                return e;
            ++seq;
        }
        return hipSuccess;
    }
};

// the copy stream and events of one out-of-core call, released on return
struct HostStreams {
    hipStream_t cs = nullptr;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    hipError_t create()
    {
        hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        for (int i = 0; i < 4 && e == hipSuccess; ++i)
            e = hipEventCreateWithFlags(&ev[i], hipEventDisableTiming);
        return e;
    }
    ~HostStreams()
    {
        if (cs != nullptr)
            (void)hipStreamSynchronize(cs);
        for (hipEvent_t e : ev)
            if (e != nullptr)
                (void)hipEventDestroy(e);
        if (cs != nullptr)
            (void)hipStreamDestroy(cs);
    }
};

// Algorithm 1's loop on the device; the host only batches launches and
// reads the statistic slots back every chunk.
gpic_status run_power_iteration(const Product &op, int64_t n,
                                const gpic_pi_params *p, double *v,
                                double *delta_user, void *ws,
                                gpic_pi_result *res, hipStream_t s)
{
    char *w = static_cast<char *>(ws);
    int *err = reinterpret_cast<int *>(w);
    double *tau = reinterpret_cast<double *>(w + 8);
    size_t o = kCtlBytes;
    double *ring = reinterpret_cast<double *>(w + o);
    o += al(kRing * 8);
    double *partial = reinterpret_cast<double *>(w + o);
    o += al((size_t)op.blocks() * 8);
    double *y = reinterpret_cast<double *>(w + o);
    o += al((size_t)n * 8);
    double *delta = delta_user ? delta_user : reinterpret_cast<double *>(w + o);
    o += al((size_t)n * 8);
    const bool pipe = op.pipelined();
    double *partial2 = pipe ? reinterpret_cast<double *>(w + o) : nullptr;
    if (pipe)
        o += al((size_t)op.blocks() * 8);
    double *y2 = pipe ? reinterpret_cast<double *>(w + o) : nullptr;

    res->iterations = 0;
    res->converged = 0;
    res->last_stat = 0.0;
    CHECK_HIP(launch_init_state(ring, kRing, err, v, delta, n, delta_user == nullptr, s),
              "init");
    const bool conv = p->mode == GPIC_MODE_CONVERGE;
    const double eps = conv ? p->eps : -1.0;
    int64_t chunk = kRing;
    if (conv)
        chunk = p->check_every > 0 ? (p->check_every < kRing ? p->check_every : kRing)
                                   : 16;
    double hstat[kRing];                       // chunk <= kRing; no heap use
    const int64_t T = p->max_iter;
    int64_t t = 0;
    bool stopped = false;
    // one launch per update: launch u takes iteration u - 1's tau and update
    // (statistic u - 1, skipped once statistic u - 2 met eps) and, for u < T,
    // iteration u's product; the partials and y alternate between two
    // buffers by the parity of u
    double *pbuf[2] = {partial, partial2};
    double *ybuf[2] = {y, y2};
    auto launch_u = [&](int64_t u) {
        StopCtl ctl;
        ctl.prev_stat = (conv && u >= 2) ? ring + ((u - 2) % kRing) : nullptr;
        ctl.cur_stat = (u >= 1) ? ring + ((u - 1) % kRing) : nullptr;
        ctl.eps = eps;
        ctl.err = err;
        const bool prod = u < T;
        return op.launch_pipe(v, delta, ybuf[(u + 1) & 1], pbuf[(u + 1) & 1], ybuf[u & 1],
                              pbuf[u & 1], u >= 1, prod, prod ? ring + (u % kRing) : nullptr,
                              ctl, s);
    };
    if (pipe && T > 0)
        CHECK_HIP(launch_u(0), "product");
    while (t < T && !stopped) {
        const int64_t te = (t + chunk < T) ? t + chunk : T;
        for (int64_t u = t; u < te && pipe; ++u)
            CHECK_HIP(launch_u(u + 1), "update and product");
        for (int64_t u = t; u < te && !pipe; ++u) {
            StopCtl ctl;
            ctl.prev_stat = (conv && u > 0) ? ring + ((u - 1) % kRing) : nullptr;
            ctl.cur_stat = ring + (u % kRing);
            ctl.eps = eps;
            ctl.err = err;
            CHECK_HIP(op.launch(v, y, partial, ctl, s), "product");
            CHECK_HIP(launch_tau_update(partial, op.blocks(), tau, y, v, delta, n, ctl, s),
                      "tau and update");
        }
        const int64_t m = te - t;
        const int64_t a = t % kRing;
        const int64_t first = (a + m <= kRing) ? m : kRing - a;
        CHECK_HIP(hipMemcpyAsync(hstat, ring + a, first * 8,
                                 hipMemcpyDeviceToHost, s), "stat copy");
        if (first < m)
            CHECK_HIP(hipMemcpyAsync(hstat + first, ring, (m - first) * 8,
                                     hipMemcpyDeviceToHost, s), "stat copy");
        int herr = 0;
        CHECK_HIP(hipMemcpyAsync(&herr, err, sizeof(int), hipMemcpyDeviceToHost, s),
                  "flag copy");
        CHECK_HIP(hipStreamSynchronize(s), "synchronize");
        if (herr)
            return fail(GPIC_ERR_NUMERIC, "||W v||_1 is zero or not finite");
        for (int64_t u = t; u < te; ++u) {
            const double su = hstat[u - t];
            if (p->stats_host)
                p->stats_host[u] = su;
            res->last_stat = su;
            res->iterations = (int32_t)(u + 1);
            if (conv && su <= p->eps) {
                res->converged = 1;
                stopped = true;
                break;
            }
        }
        t = te;
    }
    if (T == 0)
        CHECK_HIP(hipStreamSynchronize(s), "synchronize");
    return GPIC_OK;
}

} // namespace

// Scratch of gpic_power_iterate_dense_noalloc: the power-iteration state
// (control words, statistic ring, per-workgroup |y| partials, y and delta)
// in a library-owned device array instead of a caller workspace, for
// callers that cannot allocate device memory.  Every GPU the library runs
// on holds its own copy until the process ends.  In host code `scratch`
// is only a stand-in for the symbol: its device address, one per device,
// comes from hipGetSymbolAddress with that device current, and only that
// address is ever handed to kernels.
static __device__ __align__(256) unsigned char scratch[GPIC_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];            // per device, set on first use

// the device address of `scratch` on the device `s` belongs to
gpic_status noalloc_scratch(hipStream_t s, void **out)
{
    int dev = -1;
    if (s != nullptr)
        CHECK_HIP(hipStreamGetDevice(s, &dev), "stream device");
    else
        CHECK_HIP(hipGetDevice(&dev), "current device");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(GPIC_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        int cur = -1;
        CHECK_HIP(hipGetDevice(&cur), "current device");
        if (cur != dev)
            CHECK_HIP(hipSetDevice(dev), "set device");
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev)
            (void)hipSetDevice(cur);
        if (e != hipSuccess)
            return hip_fail(e, "scratch address");
        if (ptr == nullptr || !aligned(ptr, 256))
            return fail(GPIC_ERR_HIP, "scratch address null or misaligned");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return GPIC_OK;
}

} // namespace

extern "C" {

int32_t gpic_abi_version(void) { return GPIC_ABI_VERSION; }

const char *gpic_status_string(gpic_status st)
{
    switch (st) {
    case GPIC_OK: return "GPIC_OK";
    case GPIC_ERR_INVALID_ARG: return "GPIC_ERR_INVALID_ARG";
    case GPIC_ERR_WORKSPACE: return "GPIC_ERR_WORKSPACE";
    case GPIC_ERR_HIP: return "GPIC_ERR_HIP";
    case GPIC_ERR_NUMERIC: return "GPIC_ERR_NUMERIC";
    case GPIC_ERR_UNSUPPORTED: return "GPIC_ERR_UNSUPPORTED";
    }
    return "unknown gpic_status";
}

const char *gpic_last_error(void) { return gpic::last_error_text(); }

size_t gpic_workspace_bytes(int32_t op, int64_t n, int64_t nnz, int32_t k)
{
    if (n < 0 || nnz < 0 || k < 0)
        return 0;
    switch (op) {
    case GPIC_OP_AFFINITY: return aff_ws(n);
    case GPIC_OP_DEGREE_NORMALIZE: return start_ws(n);
    case GPIC_OP_DEGREE_NORMALIZE_CSR: return kCtlBytes + start_ws(n);
    case GPIC_OP_DEGREE_FUSED: return start_ws(n) + al(fused_ws(n));
    case GPIC_OP_PI_DENSE: return pi_ws(n, gemv_blocks(n));
    case GPIC_OP_PI_FUSED: return pi_fused_ws(n);
    case GPIC_OP_PI_CSR: return pi_csr_ws(n, nnz);
    case GPIC_OP_KMEANS1D: return kmeans_ws(n, k < 1 ? 1 : k);
    case GPIC_OP_AFFINITY_NORMALIZED: return start_ws(n) + aff_ws(n);
    case GPIC_OP_MATVEC_FUSED: return al(fused_ws(n));
    case GPIC_OP_AFFINITY_COSINE: return al(cosine_ws(n));
    case GPIC_OP_AFFINITY_COSINE_NORMALIZED: return start_ws(n) + al(cosine_ws(n));
    case GPIC_OP_KNN_GRAPH:
        return (k >= 1 && k <= 64 && n >= 2) ? al(knn_graph_ws(n, k)) : 0;
    case GPIC_OP_AFFINITY_SYM: return start_ws(n) + sym_aff_ws(n);
    case GPIC_OP_MATVEC_SYM: return al(sym_part_bytes(n));
    case GPIC_OP_PI_SYM: return pi_sym_ws(n);
    case GPIC_OP_PI_DENSE_HOST: return (n >= 2 && n <= kMaxN) ? pi_host_ws(n) : 0;
    default: return 0;
    }
}

gpic_status gpic_affinity(const float *X, int64_t n, int32_t d, float sigma,
                          float *A, int64_t lda, double *degree, void *ws,
                          size_t ws_bytes, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(A != nullptr, "A is null");
    CHECK_ARG(aligned(A, 16), "A must be 16-byte aligned");
    CHECK_ARG(lda >= n && lda % 4 == 0, "lda = %lld must be >= n and a multiple of 4",
              (long long)lda);
    if ((st = check_vec(degree, "degree", true)) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, aff_ws(n))) != GPIC_OK)
        return st;
    float c;
    gauss_coefficient(sigma, &c);
    CHECK_HIP(launch_affinity(X, n, d, c, A, lda, degree, ws, (hipStream_t)stream),
              "affinity");
    return GPIC_OK;
}

gpic_status gpic_affinity_normalized(const float *X, int64_t n, int32_t d,
                                     float sigma, float *W, int64_t ldw,
                                     double *degree, double *v0,
                                     int64_t *n_zero_rows, void *ws,
                                     size_t ws_bytes, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(W != nullptr, "W is null");
    CHECK_ARG(aligned(W, 16), "W must be 16-byte aligned");
    CHECK_ARG(ldw >= n && ldw % 4 == 0, "ldw = %lld must be >= n and a multiple of 4",
              (long long)ldw);
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, start_ws(n) + aff_ws(n))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    float c;
    gauss_coefficient(sigma, &c);
    void *aws = static_cast<char *>(ws) + start_ws(n);
    CHECK_HIP(launch_fused_degree(X, n, d, c, degree, aws, s), "degree sweep");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows, ws, s, &bad), "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    CHECK_HIP(launch_affinity_w(X, n, d, c, W, ldw, degree, aws, s), "W sweep");
    return GPIC_OK;
}

size_t gpic_sym_bytes(int64_t n)
{
    if (n < 2 || n > kMaxSymN)
        return 0;
    return sym_storage_bytes(n);
}

gpic_status gpic_affinity_sym(const float *X, int64_t n, int32_t d, float sigma,
                              float *As, double *degree, double *v0, int64_t *n_zero_rows,
                              void *ws, size_t ws_bytes, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(n <= kMaxSymN, "n = %lld exceeds the symmetric storage's limit 2^24",
              (long long)n);
    CHECK_ARG(As != nullptr, "As is null");
    CHECK_ARG(aligned(As, 16), "As must be 16-byte aligned");
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, start_ws(n) + sym_aff_ws(n))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    float c;
    gauss_coefficient(sigma, &c);
    void *aws = static_cast<char *>(ws) + start_ws(n);
    CHECK_HIP(launch_affinity_sym(X, n, d, c, As, aws, s), "symmetric A sweep");
    // the degrees are the row sums of the stored symmetric A (the product
    // with v = 1, no division), so the rows of D^-1 A sum to 1
    StopCtl none{};
    CHECK_HIP(launch_sym_gemv(As, n, nullptr, nullptr, degree, static_cast<double *>(aws),
                              nullptr, none, false, s),
              "degrees");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows, ws, s, &bad), "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    return GPIC_OK;
}

gpic_status gpic_affinity_cosine(const float *X, int64_t n, int32_t d, float *A,
                                 int64_t lda, double *degree, void *ws, size_t ws_bytes,
                                 void *stream)
{
    gpic_status st = check_coords(X, n, d);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(A != nullptr, "A is null");
    CHECK_ARG(aligned(A, 16), "A must be 16-byte aligned");
    CHECK_ARG(lda >= n && lda % 4 == 0, "lda = %lld must be >= n and a multiple of 4",
              (long long)lda);
    if ((st = check_vec(degree, "degree", true)) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, al(cosine_ws(n)))) != GPIC_OK)
        return st;
    CHECK_HIP(launch_affinity_cosine(X, n, d, A, lda, degree, ws, (hipStream_t)stream),
              "cosine affinity");
    return GPIC_OK;
}

gpic_status gpic_affinity_cosine_normalized(const float *X, int64_t n, int32_t d,
                                            float *W, int64_t ldw, double *degree,
                                            double *v0, int64_t *n_zero_rows, void *ws,
                                            size_t ws_bytes, void *stream)
{
    gpic_status st = check_coords(X, n, d);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(W != nullptr, "W is null");
    CHECK_ARG(aligned(W, 16), "W must be 16-byte aligned");
    CHECK_ARG(ldw >= n && ldw % 4 == 0, "ldw = %lld must be >= n and a multiple of 4",
              (long long)ldw);
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, start_ws(n) + al(cosine_ws(n)))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    void *cws = static_cast<char *>(ws) + start_ws(n);
    CHECK_HIP(launch_cosine_degree(X, n, d, degree, cws, s), "degree sweep");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows, ws, s, &bad), "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    CHECK_HIP(launch_cosine_w(X, n, d, W, ldw, degree, cws, s), "W sweep");
    return GPIC_OK;
}

static gpic_status knn_graph_common(const float *X, int64_t n, int32_t d, int32_t k,
                                    float sigma, int64_t *row_ptr, int32_t *col, float *val,
                                    int64_t *nnz, int32_t *perm, void *ws, size_t ws_bytes,
                                    void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    if (d > 16)
        return fail(GPIC_ERR_UNSUPPORTED, "the kNN graph builder supports d <= 16 (d = %d)", d);
    CHECK_ARG(k >= 1 && k <= 64 && (int64_t)k <= n - 1, "k = %d must be in [1, min(64, n-1)]",
              k);
    CHECK_ARG(2 * n * (int64_t)k < ((int64_t)1 << 32), "2 n k must be below 2^32");
    CHECK_ARG(row_ptr != nullptr && aligned(row_ptr, 8), "row_ptr null or misaligned");
    CHECK_ARG(col != nullptr && aligned(col, 4) && val != nullptr && aligned(val, 4),
              "col / val null or misaligned");
    CHECK_ARG(nnz != nullptr, "nnz is null");
    if ((st = check_ws(ws, ws_bytes, al(knn_graph_ws(n, k)))) != GPIC_OK)
        return st;
    int status = 0;
    CHECK_HIP(run_knn_graph(X, n, d, k, sigma, row_ptr, col, val, nnz, &status, ws,
                            (hipStream_t)stream, perm),
              "kNN graph");
    if (status != 0)
        return fail(GPIC_ERR_NUMERIC, "kNN candidate bounds did not converge");
    return GPIC_OK;
}

gpic_status gpic_knn_graph(const float *X, int64_t n, int32_t d, int32_t k, float sigma,
                           int64_t *row_ptr, int32_t *col, float *val, int64_t *nnz,
                           void *ws, size_t ws_bytes, void *stream)
{
    return knn_graph_common(X, n, d, k, sigma, row_ptr, col, val, nnz, nullptr, ws, ws_bytes,
                            stream);
}

gpic_status gpic_knn_graph_local(const float *X, int64_t n, int32_t d, int32_t k,
                                 float sigma, int64_t *row_ptr, int32_t *col, float *val,
                                 int64_t *nnz, int32_t *perm, void *ws, size_t ws_bytes,
                                 void *stream)
{
    CHECK_ARG(perm != nullptr && aligned(perm, 4), "perm null or misaligned");
    return knn_graph_common(X, n, d, k, sigma, row_ptr, col, val, nnz, perm, ws, ws_bytes,
                            stream);
}

gpic_status gpic_degree_normalize(float *A, int64_t n, int64_t lda, double *degree,
                                  int32_t degree_given, double *v0,
                                  int64_t *n_zero_rows, void *ws, size_t ws_bytes,
                                  void *stream)
{
    CHECK_ARG(A != nullptr && aligned(A, 16), "A is null or not 16-byte aligned");
    CHECK_ARG(n >= 2 && n <= kMaxN, "n = %lld out of range", (long long)n);
    CHECK_ARG(lda >= n && lda % 4 == 0, "lda must be >= n and a multiple of 4");
    gpic_status st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, start_ws(n))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    if (!degree_given)
        CHECK_HIP(launch_dense_degree(A, n, lda, degree, s), "degree");
    CHECK_HIP(launch_dense_scale(A, n, lda, degree, s), "normalise");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows, ws, s, &bad), "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    return GPIC_OK;
}

gpic_status gpic_degree_normalize_csr(const int64_t *row_ptr, const int32_t *col,
                                      float *val, int64_t n, int64_t nnz,
                                      double *degree, double *v0,
                                      int64_t *n_zero_rows, void *ws,
                                      size_t ws_bytes, void *stream)
{
    gpic_status st = check_csr(row_ptr, col, val, n, nnz);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, kCtlBytes + start_ws(n))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    if ((st = verify_csr(row_ptr, col, n, nnz, ws, s)) != GPIC_OK)
        return st;
    CHECK_HIP(launch_csr_degree_scale(row_ptr, val, n, degree, s), "csr normalise");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows,
                                  static_cast<char *>(ws) + kCtlBytes, s, &bad),
              "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    return GPIC_OK;
}

gpic_status gpic_degree_fused(const float *X, int64_t n, int32_t d, float sigma,
                              double *degree, double *v0, int64_t *n_zero_rows,
                              void *ws, size_t ws_bytes, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v0, "v0")) != GPIC_OK)
        return st;
    CHECK_ARG(n_zero_rows == nullptr || aligned(n_zero_rows, 8),
              "n_zero_rows misaligned");
    if ((st = check_ws(ws, ws_bytes, start_ws(n) + al(fused_ws(n)))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    float c;
    gauss_coefficient(sigma, &c);
    CHECK_HIP(launch_fused_operator_degree(X, n, d, c, degree,
                                           static_cast<char *>(ws) + start_ws(n), s),
              "fused degree");
    int bad = 0;
    CHECK_HIP(launch_start_vector(degree, n, v0, n_zero_rows, ws, s, &bad), "v0");
    if (bad)
        return fail(GPIC_ERR_NUMERIC, "sum of degrees is zero or not finite");
    return GPIC_OK;
}

gpic_status gpic_matvec_dense(const float *W, int64_t n, int64_t ldw,
                              const double *v, double *y, void *stream)
{
    CHECK_ARG(W != nullptr && aligned(W, 16), "W is null or not 16-byte aligned");
    CHECK_ARG(n >= 2 && n <= kMaxN, "n = %lld out of range", (long long)n);
    CHECK_ARG(ldw >= n && ldw % 4 == 0, "ldw must be >= n and a multiple of 4");
    gpic_status st;
    if ((st = check_vec(v, "v")) != GPIC_OK || (st = check_vec(y, "y")) != GPIC_OK)
        return st;
    StopCtl none{};
    CHECK_HIP(launch_gemv(W, n, ldw, v, y, nullptr, none, false, (hipStream_t)stream),
              "gemv");
    return GPIC_OK;
}

gpic_status gpic_matvec_sym(const float *As, int64_t n, const double *degree,
                            const double *v, double *y, void *ws, size_t ws_bytes,
                            void *stream)
{
    CHECK_ARG(As != nullptr && aligned(As, 16), "As is null or not 16-byte aligned");
    CHECK_ARG(n >= 2 && n <= kMaxSymN, "n = %lld out of range [2, 2^24]", (long long)n);
    gpic_status st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v, "v")) != GPIC_OK || (st = check_vec(y, "y")) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, al(sym_part_bytes(n)))) != GPIC_OK)
        return st;
    StopCtl none{};
    CHECK_HIP(launch_sym_gemv(As, n, degree, v, y, static_cast<double *>(ws), nullptr, none,
                              false, (hipStream_t)stream),
              "symmetric product");
    return GPIC_OK;
}

gpic_status gpic_matvec_csr(const int64_t *row_ptr, const int32_t *col,
                            const float *val, int64_t n, int64_t nnz,
                            const double *v, double *y, void *stream)
{
    gpic_status st = check_csr(row_ptr, col, val, n, nnz);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(v, "v")) != GPIC_OK || (st = check_vec(y, "y")) != GPIC_OK)
        return st;
    StopCtl none{};
    CHECK_HIP(launch_spmv(row_ptr, col, val, n, nnz, v, y, nullptr, none, false,
                          (hipStream_t)stream),
              "spmv");
    return GPIC_OK;
}

gpic_status gpic_matvec_fused(const float *X, int64_t n, int32_t d, float sigma,
                              const double *degree, const double *v, double *y,
                              void *ws, size_t ws_bytes, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK ||
        (st = check_vec(v, "v")) != GPIC_OK || (st = check_vec(y, "y")) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, al(fused_ws(n)))) != GPIC_OK)
        return st;
    float c;
    gauss_coefficient(sigma, &c);
    StopCtl none{};
    CHECK_HIP(launch_fused_apply(X, n, d, c, v, degree, y, nullptr, none, false, ws,
                                 (hipStream_t)stream),
              "fused product");
    return GPIC_OK;
}

static gpic_status check_pi_common(int64_t n, const gpic_pi_params *params,
                                   double *v, double *delta, gpic_pi_result *res)
{
    CHECK_ARG(n >= 2 && n <= kMaxN, "n = %lld out of range", (long long)n);
    gpic_status st;
    if ((st = check_params(params)) != GPIC_OK)
        return st;
    if ((st = check_vec(v, "v")) != GPIC_OK ||
        (st = check_vec(delta, "delta", true)) != GPIC_OK)
        return st;
    CHECK_ARG(res != nullptr, "res is null");
    return GPIC_OK;
}

gpic_status gpic_power_iterate_dense(const float *W, int64_t n, int64_t ldw,
                                     const gpic_pi_params *params, double *v,
                                     double *delta, void *ws, size_t ws_bytes,
                                     gpic_pi_result *res, void *stream)
{
    CHECK_ARG(W != nullptr && aligned(W, 16), "W is null or not 16-byte aligned");
    gpic_status st = check_pi_common(n, params, v, delta, res);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(ldw >= n && ldw % 4 == 0, "ldw must be >= n and a multiple of 4");
    if ((st = check_ws(ws, ws_bytes, pi_ws(n, gemv_blocks(n)))) != GPIC_OK)
        return st;
    DenseProduct op;
    op.W = W;
    op.n = n;
    op.ldw = ldw;
    return run_power_iteration(op, n, params, v, delta, ws, res, (hipStream_t)stream);
}

gpic_status gpic_power_iterate_dense_noalloc(const float *W, int64_t n, int64_t ldw,
                                             const gpic_pi_params *params, double *v,
                                             double *delta, gpic_pi_result *res,
                                             void *stream)
{
    CHECK_ARG(W != nullptr && aligned(W, 16), "W is null or not 16-byte aligned");
    gpic_status st = check_pi_common(n, params, v, delta, res);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(ldw >= n && ldw % 4 == 0, "ldw must be >= n and a multiple of 4");
    const size_t need = pi_ws(n, gemv_blocks(n));
    if (need > (size_t)GPIC_NOALLOC_SCRATCH_BYTES)
        return fail(GPIC_ERR_WORKSPACE,
                    "n = %lld needs %zu bytes of scratch; the static scratch holds %zu "
                    "(n <= %lld)",
                    (long long)n, need, (size_t)GPIC_NOALLOC_SCRATCH_BYTES,
                    (long long)GPIC_NOALLOC_MAX_N);
    hipStream_t s = (hipStream_t)stream;
    void *ws = nullptr;
    if ((st = noalloc_scratch(s, &ws)) != GPIC_OK)
        return st;
    DenseProduct op;
    op.W = W;
    op.n = n;
    op.ldw = ldw;
    return run_power_iteration(op, n, params, v, delta, ws, res, s);
}

gpic_status gpic_power_iterate_dense_host(const float *W_host, int64_t n, int64_t ldw,
                                          const gpic_pi_params *params, double *v,
                                          double *delta, void *ws, size_t ws_bytes,
                                          gpic_pi_result *res, void *stream)
{
    CHECK_ARG(W_host != nullptr && aligned(W_host, 4), "W_host is null or misaligned");
    gpic_status st = check_pi_common(n, params, v, delta, res);
    if (st != GPIC_OK)
        return st;
    CHECK_ARG(ldw >= n, "ldw must be >= n");
    const size_t base = pi_host_base(n);
    CHECK_ARG(ws != nullptr && aligned(ws, 256), "workspace is null or not 256-byte aligned");
    if (ws_bytes < base + 2 * host_panel_bytes(n, 4))
        return fail(GPIC_ERR_WORKSPACE, "workspace of %zu bytes holds no two 4-row panels "
                    "(need at least %zu)", ws_bytes, base + 2 * host_panel_bytes(n, 4));
    // the panel: the largest multiple of 4 rows whose two buffers fit
    int64_t P = (int64_t)((ws_bytes - base) / 2 / 256 * 256 / 4) / host_pitch(n) / 4 * 4;
    const int64_t all = (n + 3) & ~(int64_t)3;
    if (P > all)
        P = all;
    while (P > 4 && base + 2 * host_panel_bytes(n, P) > ws_bytes)
        P -= 4;
    if (P < 4)
        P = 4;                                   // the size check above allows 4
    HostStreams hs;
    CHECK_HIP(hs.create(), "copy stream");
    HostDenseProduct op;
    op.Wh = W_host;
    op.n = n;
    op.ldw = ldw;
    op.P = P;
    op.pitch = host_pitch(n);
    char *w = static_cast<char *>(ws) + base;
    op.buf[0] = reinterpret_cast<float *>(w);
    op.buf[1] = reinterpret_cast<float *>(w + host_panel_bytes(n, P));
    op.cs = hs.cs;
    op.copied[0] = hs.ev[0];
    op.copied[1] = hs.ev[1];
    op.consumed[0] = hs.ev[2];
    op.consumed[1] = hs.ev[3];
    // in CONVERGE mode the stop state is read after every update unless the
    // caller asks otherwise: each update queued past a stop costs a full
    // pass of W over PCIe
    gpic_pi_params p = *params;
    if (p.mode == GPIC_MODE_CONVERGE && p.check_every == 0)
        p.check_every = 1;
    return run_power_iteration(op, n, &p, v, delta, ws, res, (hipStream_t)stream);
}

gpic_status gpic_power_iterate_sym(const float *As, int64_t n, const double *degree,
                                   const gpic_pi_params *params, double *v, double *delta,
                                   void *ws, size_t ws_bytes, gpic_pi_result *res,
                                   void *stream)
{
    CHECK_ARG(As != nullptr && aligned(As, 16), "As is null or not 16-byte aligned");
    CHECK_ARG(n <= kMaxSymN, "n = %lld exceeds the symmetric storage's limit 2^24",
              (long long)n);
    gpic_status st = check_pi_common(n, params, v, delta, res);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, pi_sym_ws(n))) != GPIC_OK)
        return st;
    SymProduct op;
    op.As = As;
    op.n = n;
    op.degree = degree;
    op.part = reinterpret_cast<double *>(static_cast<char *>(ws) + pi_ws(n, sym_blocks(n)));
    return run_power_iteration(op, n, params, v, delta, ws, res, (hipStream_t)stream);
}

gpic_status gpic_power_iterate_fused(const float *X, int64_t n, int32_t d,
                                     float sigma, const double *degree,
                                     const gpic_pi_params *params, double *v,
                                     double *delta, void *ws, size_t ws_bytes,
                                     gpic_pi_result *res, void *stream)
{
    gpic_status st = check_points(X, n, d, sigma);
    if (st != GPIC_OK)
        return st;
    if ((st = check_vec(degree, "degree")) != GPIC_OK)
        return st;
    if ((st = check_pi_common(n, params, v, delta, res)) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, pi_fused_ws(n))) != GPIC_OK)
        return st;
    FusedProduct op;
    op.X = X;
    op.n = n;
    op.d = d;
    gauss_coefficient(sigma, &op.c);
    op.degree = degree;
    op.scratch = static_cast<char *>(ws) + pi_ws(n, fused_nb_bound(n));
    // the augmented operands are the same for every product of the run
    CHECK_HIP(launch_fused_prepare(X, n, d, op.c, op.scratch, (hipStream_t)stream),
              "operands");
    return run_power_iteration(op, n, params, v, delta, ws, res, (hipStream_t)stream);
}

gpic_status gpic_power_iterate_csr(const int64_t *row_ptr, const int32_t *col,
                                   const float *val, int64_t n, int64_t nnz,
                                   const gpic_pi_params *params, double *v,
                                   double *delta, void *ws, size_t ws_bytes,
                                   gpic_pi_result *res, void *stream)
{
    gpic_status st = check_csr(row_ptr, col, val, n, nnz);
    if (st != GPIC_OK)
        return st;
    if ((st = check_pi_common(n, params, v, delta, res)) != GPIC_OK)
        return st;
    if ((st = check_ws(ws, ws_bytes, pi_csr_ws(n, nnz))) != GPIC_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    if ((st = verify_csr(row_ptr, col, n, nnz, ws, s)) != GPIC_OK)
        return st;
    if (csr_blocked_applies(n) && nnz > 0) {
        BlockedCsrProduct bop;
        int usable = 0;
        CHECK_HIP(build_csr_blocked(row_ptr, col, val, n, nnz,
                                    static_cast<char *>(ws) + pi_ws(n, spmv_blocks(n)),
                                    &bop.B, s, &usable),
                  "blocked CSR copy");
        if (usable)
            return run_power_iteration(bop, n, params, v, delta, ws, res, s);
    }
    CsrProduct op;
    op.row_ptr = row_ptr;
    op.col = col;
    op.val = val;
    op.n = n;
    op.nnz = nnz;
    return run_power_iteration(op, n, params, v, delta, ws, res, s);
}

gpic_status gpic_read_stream(const float *x, int64_t n, double *sink, void *stream)
{
    CHECK_ARG(x != nullptr && aligned(x, 16), "x is null or not 16-byte aligned");
    CHECK_ARG(n >= 4 && n % 4 == 0, "n = %lld must be a positive multiple of 4", (long long)n);
    gpic_status st;
    if ((st = check_vec(sink, "sink")) != GPIC_OK)
        return st;
    static_assert(kReadStreamBlocks == GPIC_READ_STREAM_SINK, "sink length");
    CHECK_HIP(launch_read_stream(x, n, sink, (hipStream_t)stream), "read stream");
    return GPIC_OK;
}

gpic_status gpic_kmeans1d(const double *v, int64_t n, int32_t k, int32_t *labels,
                          double *centroids, int32_t *k_eff, double *cost, void *ws,
                          size_t ws_bytes, void *stream)
{
    CHECK_ARG(n >= 1 && n <= kMaxKmeansN, "n = %lld out of range [1, 2^30]", (long long)n);
    CHECK_ARG(k >= 1 && (int64_t)k <= n, "k = %d must be in [1, n]", k);
    gpic_status st;
    if ((st = check_vec(v, "v")) != GPIC_OK ||
        (st = check_vec(centroids, "centroids")) != GPIC_OK)
        return st;
    CHECK_ARG(labels != nullptr && aligned(labels, 4), "labels null or misaligned");
    CHECK_ARG(k_eff != nullptr, "k_eff is null");
    if ((st = check_ws(ws, ws_bytes, kmeans_ws(n, k))) != GPIC_OK)
        return st;
    CHECK_HIP(run_kmeans1d(v, n, k, labels, centroids, k_eff, cost, ws,
                           (hipStream_t)stream),
              "kmeans1d");
    return GPIC_OK;
}

} // extern "C"
