"""Python binding of libgpic: Power Iteration Clustering on an MI355X.

A thin ctypes layer over the C ABI declared in include/gpic.h.  Every
function here has the name of a C entry point and only marshals arguments:
it checks dtypes and devices, allocates caller-owned outputs and workspace
as torch tensors (PyTorch is used for device memory and streams only),
passes raw pointers and the current HIP stream, and raises GpicError on a
non-OK status.  All computation happens in the library's HIP kernels.

There is no fallback: if libgpic.so is missing or cannot be loaded, every
call raises.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgpic.so")

GPIC_OK = 0
STATUS = {0: "GPIC_OK", 1: "GPIC_ERR_INVALID_ARG", 2: "GPIC_ERR_WORKSPACE",
          3: "GPIC_ERR_HIP", 4: "GPIC_ERR_NUMERIC", 5: "GPIC_ERR_UNSUPPORTED"}
OP = {"affinity": 0, "degree_normalize": 1, "degree_normalize_csr": 2,
      "degree_fused": 3, "pi_dense": 4, "pi_fused": 5, "pi_csr": 6,
      "kmeans1d": 7, "affinity_normalized": 8, "matvec_fused": 9,
      "affinity_cosine": 10, "affinity_cosine_normalized": 11, "knn_graph": 12,
      "affinity_sym": 13, "matvec_sym": 14, "pi_sym": 15, "pi_dense_host": 16}
MODES = {"fixed": 0, "converge": 1}

# C entry points declared in include/gpic.h (checked by the tests)
EXPORTS = (
    "gpic_abi_version", "gpic_status_string", "gpic_last_error",
    "gpic_workspace_bytes", "gpic_affinity", "gpic_affinity_normalized",
    "gpic_degree_normalize",
    "gpic_degree_normalize_csr", "gpic_degree_fused", "gpic_matvec_dense",
    "gpic_matvec_csr", "gpic_matvec_fused", "gpic_power_iterate_dense",
    "gpic_power_iterate_fused", "gpic_power_iterate_csr", "gpic_kmeans1d",
    "gpic_affinity_cosine", "gpic_affinity_cosine_normalized", "gpic_knn_graph",
    "gpic_sym_bytes", "gpic_affinity_sym", "gpic_matvec_sym", "gpic_power_iterate_sym",
    "gpic_power_iterate_dense_host", "gpic_read_stream",
    "gpic_power_iterate_dense_noalloc", "gpic_knn_graph_local",
)

# the static scratch of gpic_power_iterate_dense_noalloc (include/gpic.h)
NOALLOC_SCRATCH_BYTES = 8 << 20
NOALLOC_MAX_N = 465536


class GpicError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class PiParams(C.Structure):
    _fields_ = [("mode", C.c_int32), ("max_iter", C.c_int32), ("eps", C.c_double),
                ("check_every", C.c_int32), ("reserved", C.c_int32),
                ("stats_host", C.POINTER(C.c_double))]


class PiResult(C.Structure):
    _fields_ = [("iterations", C.c_int32), ("converged", C.c_int32),
                ("last_stat", C.c_double)]


_lib = None


def lib() -> C.CDLL:
    """The loaded libgpic (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                              "or python paper_1604_02700_amd/build.py")
        L = C.CDLL(LIB_PATH)
        p, i64, i32, f32, sz = C.c_void_p, C.c_int64, C.c_int32, C.c_float, C.c_size_t
        L.gpic_abi_version.restype = i32
        L.gpic_status_string.restype = C.c_char_p
        L.gpic_status_string.argtypes = [C.c_int]
        L.gpic_last_error.restype = C.c_char_p
        L.gpic_workspace_bytes.restype = sz
        L.gpic_workspace_bytes.argtypes = [i32, i64, i64, i32]
        L.gpic_sym_bytes.restype = sz
        L.gpic_sym_bytes.argtypes = [i64]
        sigs = {
            "gpic_affinity": [p, i64, i32, f32, p, i64, p, p, sz, p],
            "gpic_affinity_normalized": [p, i64, i32, f32, p, i64, p, p, p, p, sz, p],
            "gpic_affinity_cosine": [p, i64, i32, p, i64, p, p, sz, p],
            "gpic_affinity_cosine_normalized": [p, i64, i32, p, i64, p, p, p, p, sz, p],
            "gpic_knn_graph": [p, i64, i32, i32, f32, p, p, p, C.POINTER(i64), p, sz, p],
            "gpic_knn_graph_local": [p, i64, i32, i32, f32, p, p, p, C.POINTER(i64), p, p, sz,
                                     p],
            "gpic_degree_normalize": [p, i64, i64, p, i32, p, p, p, sz, p],
            "gpic_degree_normalize_csr": [p, p, p, i64, i64, p, p, p, p, sz, p],
            "gpic_degree_fused": [p, i64, i32, f32, p, p, p, p, sz, p],
            "gpic_matvec_dense": [p, i64, i64, p, p, p],
            "gpic_matvec_csr": [p, p, p, i64, i64, p, p, p],
            "gpic_matvec_fused": [p, i64, i32, f32, p, p, p, p, sz, p],
            "gpic_affinity_sym": [p, i64, i32, f32, p, p, p, p, p, sz, p],
            "gpic_matvec_sym": [p, i64, p, p, p, p, sz, p],
            "gpic_power_iterate_sym": [p, i64, p, C.POINTER(PiParams), p, p, p, sz,
                                       C.POINTER(PiResult), p],
            "gpic_power_iterate_dense_host": [p, i64, i64, C.POINTER(PiParams), p, p, p,
                                              sz, C.POINTER(PiResult), p],
            "gpic_power_iterate_dense": [p, i64, i64, C.POINTER(PiParams), p, p, p,
                                         sz, C.POINTER(PiResult), p],
            "gpic_power_iterate_dense_noalloc": [p, i64, i64, C.POINTER(PiParams), p, p,
                                                 C.POINTER(PiResult), p],
            "gpic_power_iterate_fused": [p, i64, i32, f32, p, C.POINTER(PiParams),
                                         p, p, p, sz, C.POINTER(PiResult), p],
            "gpic_power_iterate_csr": [p, p, p, i64, i64, C.POINTER(PiParams), p, p,
                                       p, sz, C.POINTER(PiResult), p],
            "gpic_kmeans1d": [p, i64, i32, p, p, C.POINTER(i32), C.POINTER(C.c_double),
                              p, sz, p],
            "gpic_read_stream": [p, i64, p, p],
        }
        for name, args in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = C.c_int
        _lib = L
    return _lib


def _check(st: int):
    if st != GPIC_OK:
        raise GpicError(st, lib().gpic_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(device) -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dev(t: torch.Tensor, dtype, name):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")


def _vec(t, n, name, device):
    if t is None:
        return torch.empty(n, dtype=torch.float64, device=device)
    _dev(t, torch.float64, name)
    if not t.is_contiguous() or t.numel() != n:
        raise ValueError(f"{name} must be contiguous with {n} elements")
    return t


def workspace_bytes(op: str, n: int, nnz: int = 0, k: int = 0) -> int:
    return int(lib().gpic_workspace_bytes(OP[op], int(n), int(nnz), int(k)))


def workspace(op: str, n: int, nnz: int = 0, k: int = 0, device="cuda"):
    """A 256-byte aligned uint8 workspace tensor for `op` (plus its size)."""
    nbytes = workspace_bytes(op, n, nnz, k)
    if nbytes == 0:
        return None, 0
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + nbytes], nbytes


def padded_ld(n: int) -> int:
    """Row stride (in floats) used for dense n x n storage: 128-byte rows."""
    return (n + 31) // 32 * 32


# ------------------------------------------------------------- 1. affinity
def gpic_affinity(X: torch.Tensor, sigma: float, A: Optional[torch.Tensor] = None,
                  want_degree: bool = True):
    """A (float32 [n, lda], first n columns valid) and optional float64 degrees."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    if A is None:
        A = torch.empty((n, padded_ld(n)), dtype=torch.float32, device=X.device)
    _dev(A, torch.float32, "A")
    if A.dim() != 2 or A.shape[0] != n or A.stride(1) != 1 or A.shape[1] < n:
        raise ValueError("A must be [n, >= n] with unit column stride")
    deg = torch.empty(n, dtype=torch.float64, device=X.device) if want_degree else None
    ws, nb = workspace("affinity", n, device=X.device)
    _check(lib().gpic_affinity(_ptr(X), n, d, float(sigma), _ptr(A), A.stride(0),
                               _ptr(deg), _ptr(ws), nb, _stream(X.device)))
    return A, deg


def gpic_affinity_normalized(X: torch.Tensor, sigma: float,
                             W: Optional[torch.Tensor] = None):
    """W = D^-1 A written directly (A never stored); returns
    (W, degree, v0, n_zero_rows tensor)."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    if W is None:
        W = torch.empty((n, padded_ld(n)), dtype=torch.float32, device=dev)
    _dev(W, torch.float32, "W")
    if W.dim() != 2 or W.shape[0] != n or W.stride(1) != 1 or W.shape[1] < n:
        raise ValueError("W must be [n, >= n] with unit column stride")
    degree = torch.empty(n, dtype=torch.float64, device=dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("affinity_normalized", n, device=dev)
    _check(lib().gpic_affinity_normalized(_ptr(X), n, d, float(sigma), _ptr(W),
                                          W.stride(0), _ptr(degree), _ptr(v0),
                                          _ptr(nz), _ptr(ws), nb, _stream(dev)))
    return W, degree, v0, nz


def _square(M, n, name, dev):
    if M is None:
        M = torch.empty((n, padded_ld(n)), dtype=torch.float32, device=dev)
    _dev(M, torch.float32, name)
    if M.dim() != 2 or M.shape[0] != n or M.stride(1) != 1 or M.shape[1] < n:
        raise ValueError(f"{name} must be [n, >= n] with unit column stride")
    return M


def gpic_affinity_cosine(X: torch.Tensor, A: Optional[torch.Tensor] = None,
                         want_degree: bool = True):
    """Cosine affinity (1 + cos) / 2 (float32 [n, lda]) and optional degrees."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    A = _square(A, n, "A", X.device)
    deg = torch.empty(n, dtype=torch.float64, device=X.device) if want_degree else None
    ws, nb = workspace("affinity_cosine", n, device=X.device)
    _check(lib().gpic_affinity_cosine(_ptr(X), n, d, _ptr(A), A.stride(0), _ptr(deg),
                                      _ptr(ws), nb, _stream(X.device)))
    return A, deg


def gpic_affinity_cosine_normalized(X: torch.Tensor, W: Optional[torch.Tensor] = None):
    """W = D^-1 A for the cosine affinity, written directly; returns
    (W, degree, v0, n_zero_rows tensor)."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    W = _square(W, n, "W", dev)
    degree = torch.empty(n, dtype=torch.float64, device=dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("affinity_cosine_normalized", n, device=dev)
    _check(lib().gpic_affinity_cosine_normalized(_ptr(X), n, d, _ptr(W), W.stride(0),
                                                 _ptr(degree), _ptr(v0), _ptr(nz),
                                                 _ptr(ws), nb, _stream(dev)))
    return W, degree, v0, nz


def gpic_knn_graph(X: torch.Tensor, k: int, sigma: float):
    """Exact kNN graph (union symmetrised, Gaussian weights) as device CSR:
    (row_ptr int64 [n+1], col int32 [nnz], val float32 [nnz])."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    rp = torch.empty(n + 1, dtype=torch.int64, device=dev)
    col = torch.empty(2 * n * k, dtype=torch.int32, device=dev)
    val = torch.empty(2 * n * k, dtype=torch.float32, device=dev)
    nnz = C.c_int64(0)
    ws, nb = workspace("knn_graph", n, 0, k, device=dev)
    _check(lib().gpic_knn_graph(_ptr(X), n, d, int(k), float(sigma), _ptr(rp), _ptr(col),
                                _ptr(val), C.byref(nnz), _ptr(ws), nb, _stream(dev)))
    m = int(nnz.value)
    return rp, col[:m], val[:m]


def gpic_knn_graph_local(X: torch.Tensor, k: int, sigma: float):
    """The same graph with its nodes numbered in the Morton order of the
    points: (row_ptr, col, val, perm), node p being point perm[p] (int32)."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    rp = torch.empty(n + 1, dtype=torch.int64, device=dev)
    col = torch.empty(2 * n * k, dtype=torch.int32, device=dev)
    val = torch.empty(2 * n * k, dtype=torch.float32, device=dev)
    perm = torch.empty(n, dtype=torch.int32, device=dev)
    nnz = C.c_int64(0)
    ws, nb = workspace("knn_graph", n, 0, k, device=dev)
    _check(lib().gpic_knn_graph_local(_ptr(X), n, d, int(k), float(sigma), _ptr(rp),
                                      _ptr(col), _ptr(val), C.byref(nnz), _ptr(perm),
                                      _ptr(ws), nb, _stream(dev)))
    m = int(nnz.value)
    return rp, col[:m], val[:m], perm


# ----------------------------------------------- 2. degrees, W and v0
def gpic_degree_normalize(A: torch.Tensor, n: Optional[int] = None,
                          degree: Optional[torch.Tensor] = None,
                          degree_given: bool = False):
    """A -> W in place; returns (A, degree, v0, n_zero_rows tensor)."""
    _dev(A, torch.float32, "A")
    n = A.shape[0] if n is None else n
    dev = A.device
    degree = _vec(degree, n, "degree", dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("degree_normalize", n, device=dev)
    _check(lib().gpic_degree_normalize(_ptr(A), n, A.stride(0), _ptr(degree),
                                       1 if degree_given else 0, _ptr(v0), _ptr(nz),
                                       _ptr(ws), nb, _stream(dev)))
    return A, degree, v0, nz


def gpic_degree_normalize_csr(row_ptr, col, val):
    """val -> normalised in place; returns (val, degree, v0, n_zero_rows)."""
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col, torch.int32, "col")
    _dev(val, torch.float32, "val")
    n = row_ptr.numel() - 1
    nnz = val.numel()
    dev = val.device
    degree = torch.empty(n, dtype=torch.float64, device=dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("degree_normalize_csr", n, nnz, device=dev)
    _check(lib().gpic_degree_normalize_csr(_ptr(row_ptr), _ptr(col), _ptr(val), n, nnz,
                                           _ptr(degree), _ptr(v0), _ptr(nz), _ptr(ws),
                                           nb, _stream(dev)))
    return val, degree, v0, nz


def gpic_degree_fused(X: torch.Tensor, sigma: float):
    """Degrees and v0 with A recomputed and never stored."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    degree = torch.empty(n, dtype=torch.float64, device=dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("degree_fused", n, device=dev)
    _check(lib().gpic_degree_fused(_ptr(X), n, d, float(sigma), _ptr(degree), _ptr(v0),
                                   _ptr(nz), _ptr(ws), nb, _stream(dev)))
    return degree, v0, nz


# --------------------------------------------------- 3. one product y = W v
def gpic_matvec_dense(W: torch.Tensor, v: torch.Tensor, y=None, n=None):
    _dev(W, torch.float32, "W")
    n = W.shape[0] if n is None else n
    y = _vec(y, n, "y", W.device)
    _dev(v, torch.float64, "v")
    _check(lib().gpic_matvec_dense(_ptr(W), n, W.stride(0), _ptr(v), _ptr(y),
                                   _stream(W.device)))
    return y


def gpic_matvec_csr(row_ptr, col, val, v, y=None):
    n = row_ptr.numel() - 1
    y = _vec(y, n, "y", val.device)
    _dev(v, torch.float64, "v")
    _check(lib().gpic_matvec_csr(_ptr(row_ptr), _ptr(col), _ptr(val), n, val.numel(),
                                 _ptr(v), _ptr(y), _stream(val.device)))
    return y


# ------------------------------------------- symmetric (packed upper tiles)
def sym_bytes(n: int) -> int:
    """Bytes of the symmetric tile storage of an n x n affinity."""
    return int(lib().gpic_sym_bytes(int(n)))


def gpic_affinity_sym(X: torch.Tensor, sigma: float, As: Optional[torch.Tensor] = None):
    """A into the packed upper tiles (a flat float32 tensor of sym_bytes(n) / 4
    entries); returns (As, degree, v0, n_zero_rows tensor)."""
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    dev = X.device
    m = sym_bytes(n) // 4
    if As is None:
        As = torch.empty(m, dtype=torch.float32, device=dev)
    _dev(As, torch.float32, "As")
    if not As.is_contiguous() or As.numel() < m:
        raise ValueError(f"As must be contiguous with at least {m} entries")
    degree = torch.empty(n, dtype=torch.float64, device=dev)
    v0 = torch.empty(n, dtype=torch.float64, device=dev)
    nz = torch.zeros(1, dtype=torch.int64, device=dev)
    ws, nb = workspace("affinity_sym", n, device=dev)
    _check(lib().gpic_affinity_sym(_ptr(X), n, d, float(sigma), _ptr(As), _ptr(degree),
                                   _ptr(v0), _ptr(nz), _ptr(ws), nb, _stream(dev)))
    return As, degree, v0, nz


def gpic_matvec_sym(As, n, degree, v, y=None):
    """y = D^-1 (A v) over the symmetric storage."""
    _dev(As, torch.float32, "As")
    dev = As.device
    y = _vec(y, n, "y", dev)
    ws, nb = workspace("matvec_sym", n, device=dev)
    _check(lib().gpic_matvec_sym(_ptr(As), int(n), _ptr(degree), _ptr(v), _ptr(y),
                                 _ptr(ws), nb, _stream(dev)))
    return y


def gpic_matvec_fused(X, sigma, degree, v, y=None):
    _dev(X, torch.float32, "X")
    n, d = X.shape
    y = _vec(y, n, "y", X.device)
    ws, nb = workspace("matvec_fused", n, device=X.device)
    _check(lib().gpic_matvec_fused(_ptr(X), n, d, float(sigma), _ptr(degree), _ptr(v),
                                   _ptr(y), _ptr(ws), nb, _stream(X.device)))
    return y


# ------------------------------------------------------- 3+4. iteration
@dataclasses.dataclass
class PIOut:
    v: torch.Tensor
    delta: Optional[torch.Tensor]
    iterations: int
    converged: bool
    last_stat: float
    stats: np.ndarray


def _params(mode, max_iter, eps, check_every, stats_buf):
    p = PiParams()
    p.mode = MODES[mode]
    p.max_iter = int(max_iter)
    p.eps = float(eps)
    p.check_every = int(check_every)
    p.reserved = 0
    p.stats_host = (stats_buf.ctypes.data_as(C.POINTER(C.c_double))
                    if stats_buf is not None else None)
    return p


def _run_pi(fn, head, n, dev, v, delta, mode, max_iter, eps, check_every,
            record_stats, op, nnz=0):
    stats = np.zeros(max(int(max_iter), 1)) if record_stats else None
    p = _params(mode, max_iter, eps, check_every, stats)
    r = PiResult()
    ws, nb = workspace(op, n, nnz, device=dev)
    _check(fn(*head, C.byref(p), _ptr(v), _ptr(delta), _ptr(ws), nb, C.byref(r),
              _stream(dev)))
    st = stats[: r.iterations].copy() if record_stats else np.zeros(0)
    return PIOut(v, delta, int(r.iterations), bool(r.converged), float(r.last_stat), st)


def gpic_power_iterate_dense(W, v, delta=None, mode="converge", max_iter=1000, eps=0.0,
                             check_every=0, record_stats=True, n=None):
    """Algorithm 1's loop over dense W; v (and delta, if given) are updated in place."""
    _dev(W, torch.float32, "W")
    n = W.shape[0] if n is None else n
    _vec(v, n, "v", W.device)
    if delta is not None:
        _vec(delta, n, "delta", W.device)
    return _run_pi(lib().gpic_power_iterate_dense, (_ptr(W), n, W.stride(0)), n,
                   W.device, v, delta, mode, max_iter, eps, check_every, record_stats,
                   "pi_dense")


def gpic_power_iterate_dense_noalloc(W, v, delta=None, mode="converge", max_iter=1000,
                                     eps=0.0, check_every=0, record_stats=True, n=None):
    """gpic_power_iterate_dense with the library's static device scratch in
    place of a workspace: nothing is allocated on the device (n <=
    NOALLOC_MAX_N; calls that overlap on one GPU race)."""
    _dev(W, torch.float32, "W")
    n = W.shape[0] if n is None else n
    _vec(v, n, "v", W.device)
    if delta is not None:
        _vec(delta, n, "delta", W.device)
    stats = np.zeros(max(int(max_iter), 1)) if record_stats else None
    p = _params(mode, max_iter, eps, check_every, stats)
    r = PiResult()
    _check(lib().gpic_power_iterate_dense_noalloc(_ptr(W), n, W.stride(0), C.byref(p),
                                                  _ptr(v), _ptr(delta), C.byref(r),
                                                  _stream(W.device)))
    st = stats[: r.iterations].copy() if record_stats else np.zeros(0)
    return PIOut(v, delta, int(r.iterations), bool(r.converged), float(r.last_stat), st)


def gpic_power_iterate_dense_host(W_host, v, delta=None, mode="converge", max_iter=1000,
                                  eps=0.0, check_every=0, record_stats=True, n=None,
                                  ws_bytes=None):
    """Algorithm 1's loop over a dense W kept in host memory (a pinned CPU
    float32 tensor [n, >= n]), streamed to the device in row panels every
    update; ws_bytes (default: two 64 MiB panels) sets the panel size."""
    if not isinstance(W_host, torch.Tensor) or W_host.is_cuda or W_host.dtype != torch.float32:
        raise TypeError("W_host must be a float32 CPU tensor")
    if W_host.dim() != 2 or W_host.stride(1) != 1:
        raise ValueError("W_host must be 2-D with unit column stride")
    dev = v.device
    n = W_host.shape[0] if n is None else n
    _vec(v, n, "v", dev)
    if delta is not None:
        _vec(delta, n, "delta", dev)
    stats = np.zeros(max(int(max_iter), 1)) if record_stats else None
    p = _params(mode, max_iter, eps, check_every, stats)
    r = PiResult()
    nb = workspace_bytes("pi_dense_host", n) if ws_bytes is None else int(ws_bytes)
    buf = torch.empty(nb + 256, dtype=torch.uint8, device=dev)
    off = (-buf.data_ptr()) % 256
    ws = buf[off:off + nb]
    _check(lib().gpic_power_iterate_dense_host(C.c_void_p(W_host.data_ptr()), n,
                                               W_host.stride(0), C.byref(p), _ptr(v),
                                               _ptr(delta), _ptr(ws), nb, C.byref(r),
                                               _stream(dev)))
    st = stats[: r.iterations].copy() if record_stats else np.zeros(0)
    return PIOut(v, delta, int(r.iterations), bool(r.converged), float(r.last_stat), st)


def gpic_power_iterate_sym(As, n, degree, v, delta=None, mode="converge", max_iter=1000,
                           eps=0.0, check_every=0, record_stats=True):
    """Algorithm 1's loop over the symmetric storage (y = D^-1 (A v))."""
    _dev(As, torch.float32, "As")
    dev = As.device
    _vec(v, n, "v", dev)
    _vec(degree, n, "degree", dev)
    if delta is not None:
        _vec(delta, n, "delta", dev)
    return _run_pi(lib().gpic_power_iterate_sym, (_ptr(As), int(n), _ptr(degree)), n, dev,
                   v, delta, mode, max_iter, eps, check_every, record_stats, "pi_sym")


def gpic_power_iterate_fused(X, sigma, degree, v, delta=None, mode="fixed", max_iter=30,
                             eps=0.0, check_every=0, record_stats=True):
    _dev(X, torch.float32, "X")
    X = X.contiguous()
    n, d = X.shape
    _vec(v, n, "v", X.device)
    _vec(degree, n, "degree", X.device)
    if delta is not None:
        _vec(delta, n, "delta", X.device)
    return _run_pi(lib().gpic_power_iterate_fused,
                   (_ptr(X), n, d, float(sigma), _ptr(degree)), n, X.device, v, delta,
                   mode, max_iter, eps, check_every, record_stats, "pi_fused")


def gpic_power_iterate_csr(row_ptr, col, val, v, delta=None, mode="converge",
                           max_iter=1000, eps=0.0, check_every=0, record_stats=True):
    _dev(row_ptr, torch.int64, "row_ptr")
    _dev(col, torch.int32, "col")
    _dev(val, torch.float32, "val")
    n = row_ptr.numel() - 1
    nnz = val.numel()
    _vec(v, n, "v", val.device)
    if delta is not None:
        _vec(delta, n, "delta", val.device)
    return _run_pi(lib().gpic_power_iterate_csr,
                   (_ptr(row_ptr), _ptr(col), _ptr(val), n, nnz), n, val.device, v,
                   delta, mode, max_iter, eps, check_every, record_stats, "pi_csr",
                   nnz)


# ------------------------------------------------------------ 5. k-means
@dataclasses.dataclass
class KMOut:
    labels: torch.Tensor        # int32 [n]
    centroids: torch.Tensor     # float64 [k_eff]
    k_eff: int
    cost: float


READ_STREAM_SINK = 1536


def gpic_read_stream(x: torch.Tensor, n: Optional[int] = None,
                     sink: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Read the first n floats of x once (a bandwidth reference, not a step
    of the method); returns the per-workgroup float64 sums."""
    _dev(x, torch.float32, "x")
    n = x.numel() if n is None else n
    if n > x.numel() or not x.is_contiguous():
        raise ValueError("x must be contiguous and hold n floats")
    if sink is None:
        sink = torch.empty(READ_STREAM_SINK, dtype=torch.float64, device=x.device)
    _check(lib().gpic_read_stream(_ptr(x), n, _ptr(sink), _stream(x.device)))
    return sink


def gpic_kmeans1d(v: torch.Tensor, k: int) -> KMOut:
    _dev(v, torch.float64, "v")
    n = v.numel()
    dev = v.device
    labels = torch.empty(n, dtype=torch.int32, device=dev)
    cent = torch.empty(max(int(k), 1), dtype=torch.float64, device=dev)
    ke = C.c_int32(0)
    cost = C.c_double(0.0)
    ws, nb = workspace("kmeans1d", n, 0, k, device=dev)
    _check(lib().gpic_kmeans1d(_ptr(v), n, int(k), _ptr(labels), _ptr(cent),
                               C.byref(ke), C.byref(cost), _ptr(ws), nb, _stream(dev)))
    return KMOut(labels, cent[: ke.value], int(ke.value), float(cost.value))


# ----------------------------------------------- whole paths (call chains)
@dataclasses.dataclass
class PICOut:
    degree: torch.Tensor
    v0: torch.Tensor
    pi: PIOut
    km: KMOut
    n_zero_rows: int


def pic_dense(X, sigma, k, mode="converge", max_iter=1000, eps=0.0, check_every=0,
              A: Optional[torch.Tensor] = None, fused_normalize: bool = True) -> PICOut:
    """Affinity, degrees, W = D^-1 A, v0, the power iteration and k-means,
    over a materialised dense W (n^2 float32).  fused_normalize writes W in
    one call (gpic_affinity_normalized); otherwise A is written, then scaled
    in place (gpic_affinity + gpic_degree_normalize)."""
    n = X.shape[0]
    if fused_normalize:
        W, deg, v0, nz = gpic_affinity_normalized(X, sigma, A)
    else:
        A, deg = gpic_affinity(X, sigma, A)
        W, deg, v0, nz = gpic_degree_normalize(A, n, deg, degree_given=True)
    v = v0.clone()
    pi = gpic_power_iterate_dense(W, v, None, mode, max_iter, eps, check_every, n=n)
    km = gpic_kmeans1d(pi.v, k)
    return PICOut(deg, v0, pi, km, int(nz.item()))


def pic_sym(X, sigma, k, mode="converge", max_iter=1000, eps=0.0, check_every=0,
            As: Optional[torch.Tensor] = None) -> PICOut:
    """The dense path over the symmetric storage: A's upper tiles, the
    degrees and v0, the power iteration with y = D^-1 (A v), k-means."""
    n = X.shape[0]
    As, deg, v0, nz = gpic_affinity_sym(X, sigma, As)
    v = v0.clone()
    pi = gpic_power_iterate_sym(As, n, deg, v, None, mode, max_iter, eps, check_every)
    km = gpic_kmeans1d(pi.v, k)
    return PICOut(deg, v0, pi, km, int(nz.item()))


def pic_cosine(X, k, mode="converge", max_iter=3, eps=0.0, check_every=0,
               W: Optional[torch.Tensor] = None) -> PICOut:
    """The dense path with the cosine affinity of the paper's Experiment I
    (its runs stop after at most 3 updates)."""
    n = X.shape[0]
    W, deg, v0, nz = gpic_affinity_cosine_normalized(X, W)
    v = v0.clone()
    pi = gpic_power_iterate_dense(W, v, None, mode, max_iter, eps, check_every, n=n)
    km = gpic_kmeans1d(pi.v, k)
    return PICOut(deg, v0, pi, km, int(nz.item()))


def pic_fused(X, sigma, k, mode="fixed", max_iter=30, eps=0.0, check_every=0) -> PICOut:
    """The same path with W never stored (affinity recomputed every sweep)."""
    deg, v0, nz = gpic_degree_fused(X, sigma)
    v = v0.clone()
    pi = gpic_power_iterate_fused(X, sigma, deg, v, None, mode, max_iter, eps, check_every)
    km = gpic_kmeans1d(pi.v, k)
    return PICOut(deg, v0, pi, km, int(nz.item()))


def pic_csr(row_ptr, col, val, k, mode="converge", max_iter=1000, eps=0.0,
            check_every=0) -> PICOut:
    """The same path over a CSR affinity graph (val normalised in place)."""
    val, deg, v0, nz = gpic_degree_normalize_csr(row_ptr, col, val)
    v = v0.clone()
    pi = gpic_power_iterate_csr(row_ptr, col, val, v, None, mode, max_iter, eps,
                                check_every)
    km = gpic_kmeans1d(pi.v, k)
    return PICOut(deg, v0, pi, km, int(nz.item()))
