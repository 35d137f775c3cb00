"""Python face of the oracle (plain float64 CPU Power Iteration Clustering).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check and
the benchmark's CPU-baseline leg import this package.  It wraps the C file
``gpic_oracle.c`` in this directory through ctypes and shares nothing with
the GPU library.  See that file's header for what each function follows in
the paper and how it is pinned.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gpic_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

FIXED, CONVERGE = 0, 1
_MODES = {"fixed": FIXED, "converge": CONVERGE, FIXED: FIXED, CONVERGE: CONVERGE}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-fPIC", "-shared", "-Wall", "-o", tmp,
               _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        _lib = _declare(C.CDLL(_LIB_PATH))
    return _lib


class use_library:
    """Temporarily route every oracle call through another build of the
    oracle source (the mutation tests load deliberately broken copies)."""

    def __init__(self, path):
        self.path = path

    def __enter__(self):
        global _lib
        self.saved = _L()
        _lib = _declare(C.CDLL(self.path))
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def compile_source(src_path, out_path):
    """Compile an oracle source file with the oracle's own flags."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-fPIC", "-shared", "-w", "-o", out_path,
           src_path, "-lm"]
    subprocess.run(cmd, check=True)
    return out_path


def _declare(lib):
    """Declare the argument and return types of every oracle function."""
    p = C.c_void_p
    i64, i32, f64 = C.c_int64, C.c_int32, C.c_double
    lib.orc_num_threads.restype = i32
    lib.orc_affinity_rows.argtypes = [p, i64, i32, f64, i64, i64, p]
    lib.orc_affinity_cosine_rows.argtypes = [p, i64, i32, i64, i64, p]
    lib.orc_knn_graph.argtypes = [p, i64, i32, i32, f64, p, p, p]
    lib.orc_knn_graph.restype = i64
    lib.orc_knn_rows.argtypes = [p, i64, i32, i32, f64, p, i64, p, p, p]
    lib.orc_knn_rows.restype = i32
    lib.orc_degree_rows.argtypes = [p, i64, i32, f64, p, i64, p]
    lib.orc_degree_normalize.argtypes = [p, i64, p, p]
    lib.orc_degree_normalize.restype = i64
    lib.orc_degree_normalize_csr.argtypes = [p, p, p, i64, p, p, p]
    lib.orc_degree_normalize_csr.restype = i64
    lib.orc_degree_onthefly.argtypes = [p, i64, i32, f64, p, p]
    lib.orc_degree_onthefly.restype = i64
    lib.orc_power_iterate_dense.argtypes = [p, i64, i32, i32, f64, p, p, p, p]
    lib.orc_power_iterate_dense.restype = i32
    lib.orc_power_iterate_csr.argtypes = [p, p, p, i64, i32, i32, f64, p, p, p, p]
    lib.orc_power_iterate_csr.restype = i32
    lib.orc_power_iterate_onthefly.argtypes = [p, i64, i32, f64, p, i32, i32,
                                               f64, p, p, p, p]
    lib.orc_power_iterate_onthefly.restype = i32
    lib.orc_matvec_onthefly_rows.argtypes = [p, i64, i32, f64, p, p, p, i64, p]
    lib.orc_kmeans1d.argtypes = [p, i64, i32, i32, p, p, p, p]
    lib.orc_kmeans1d.restype = i32
    return lib


def _ptr(a: np.ndarray):
    return C.c_void_p(a.ctypes.data)


def _f32(X):
    return np.ascontiguousarray(X, dtype=np.float32)


def _f64(x):
    return np.ascontiguousarray(x, dtype=np.float64)


def num_threads() -> int:
    return int(_L().orc_num_threads())


# ---------------------------------------------------------------- affinity
def affinity(X, sigma) -> np.ndarray:
    """Full n x n Gaussian affinity (zero diagonal), float64."""
    X = _f32(X)
    n, d = X.shape
    A = np.empty((n, n), dtype=np.float64)
    _L().orc_affinity_rows(_ptr(X), n, d, float(np.float32(sigma)), 0, n, _ptr(A))
    return A


def affinity_cosine(X) -> np.ndarray:
    """Full n x n cosine affinity (1 + cos) / 2 with a zero diagonal, float64."""
    X = _f32(X)
    n, d = X.shape
    A = np.empty((n, n), dtype=np.float64)
    _L().orc_affinity_cosine_rows(_ptr(X), n, d, 0, n, _ptr(A))
    return A


def affinity_cosine_rows(X, rows) -> np.ndarray:
    """Rows `rows` of the cosine A (recomputed), float64 [len(rows), n]."""
    X = _f32(X)
    n, d = X.shape
    out = np.empty((len(rows), n), dtype=np.float64)
    for r, i in enumerate(rows):
        _L().orc_affinity_cosine_rows(_ptr(X), n, d, int(i), 1,
                                      C.c_void_p(out.ctypes.data + r * n * 8))
    return out


def affinity_rows(X, sigma, rows) -> np.ndarray:
    """Rows `rows` of A (recomputed), float64 [len(rows), n]."""
    X = _f32(X)
    n, d = X.shape
    out = np.empty((len(rows), n), dtype=np.float64)
    for r, i in enumerate(rows):
        _L().orc_affinity_rows(_ptr(X), n, d, float(np.float32(sigma)), int(i), 1,
                               C.c_void_p(out.ctypes.data + r * n * 8))
    return out


def degree_rows(X, sigma, rows) -> np.ndarray:
    X = _f32(X)
    n, d = X.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty(rows.shape[0], dtype=np.float64)
    _L().orc_degree_rows(_ptr(X), n, d, float(np.float32(sigma)), _ptr(rows),
                         rows.shape[0], _ptr(out))
    return out


# ------------------------------------------------------- degree / normalise
def degree_normalize(A, copy=True):
    """Returns (W, degree, v0, n_zero_rows); with copy=False a float64
    C-contiguous A is overwritten by W."""
    W = np.array(A, dtype=np.float64, order="C", copy=copy)
    n = W.shape[0]
    deg = np.empty(n)
    v0 = np.empty(n)
    nz = _L().orc_degree_normalize(_ptr(W), n, _ptr(deg), _ptr(v0))
    if nz < 0:
        raise FloatingPointError("degrees sum to zero")
    return W, deg, v0, int(nz)


def degree_normalize_csr(row_ptr, col, val):
    rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
    cl = np.ascontiguousarray(col, dtype=np.int32)
    a = _f64(val)
    n = rp.shape[0] - 1
    w = np.empty_like(a)
    deg = np.empty(n)
    v0 = np.empty(n)
    nz = _L().orc_degree_normalize_csr(_ptr(rp), _ptr(cl), _ptr(a), n, _ptr(w),
                                       _ptr(deg), _ptr(v0))
    if nz < 0:
        raise FloatingPointError("degrees sum to zero")
    return w, deg, v0, int(nz)


def degree_onthefly(X, sigma):
    X = _f32(X)
    n, d = X.shape
    deg = np.empty(n)
    v0 = np.empty(n)
    nz = _L().orc_degree_onthefly(_ptr(X), n, d, float(np.float32(sigma)),
                                  _ptr(deg), _ptr(v0))
    if nz < 0:
        raise FloatingPointError("degrees sum to zero")
    return deg, v0, int(nz)


# ---------------------------------------------------------- power iteration
@dataclasses.dataclass
class PIResult:
    v: np.ndarray
    delta: np.ndarray
    stats: np.ndarray       # statistic of every update performed
    iterations: int         # matrix-vector products performed
    converged: bool


def _run(fn, args, v0, mode, max_iter, eps, delta):
    v = _f64(v0).copy()
    dl = v.copy() if delta is None else _f64(delta).copy()
    stats = np.zeros(max(int(max_iter), 1))
    conv = C.c_int32(0)
    it = fn(*args, _MODES[mode], int(max_iter), float(eps), _ptr(v), _ptr(dl),
            _ptr(stats), C.byref(conv))
    if it < 0:
        raise FloatingPointError("||W v||_1 is zero or not finite")
    return PIResult(v, dl, stats[:it].copy(), int(it), bool(conv.value))


def power_iterate_dense(W, v0, mode="fixed", max_iter=10, eps=0.0, delta=None):
    """Algorithm 1 on a dense float64 W.  delta=None means delta_0 = v_0."""
    W = _f64(W)
    n = W.shape[0]
    return _run(_L().orc_power_iterate_dense, (_ptr(W), n), v0, mode, max_iter,
                eps, delta)


def power_iterate_csr(row_ptr, col, w, v0, mode="fixed", max_iter=10, eps=0.0,
                      delta=None):
    rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
    cl = np.ascontiguousarray(col, dtype=np.int32)
    ww = _f64(w)
    n = rp.shape[0] - 1
    return _run(_L().orc_power_iterate_csr, (_ptr(rp), _ptr(cl), _ptr(ww), n),
                v0, mode, max_iter, eps, delta)


def power_iterate_onthefly(X, sigma, degree, v0, mode="fixed", max_iter=10,
                           eps=0.0, delta=None):
    X = _f32(X)
    n, d = X.shape
    deg = _f64(degree)
    return _run(_L().orc_power_iterate_onthefly,
                (_ptr(X), n, d, float(np.float32(sigma)), _ptr(deg)),
                v0, mode, max_iter, eps, delta)


def matvec_onthefly_rows(X, sigma, degree, v, rows) -> np.ndarray:
    X = _f32(X)
    n, d = X.shape
    deg = _f64(degree)
    vv = _f64(v)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    y = np.empty(rows.shape[0])
    _L().orc_matvec_onthefly_rows(_ptr(X), n, d, float(np.float32(sigma)),
                                  _ptr(deg), _ptr(vv), _ptr(rows), rows.shape[0],
                                  _ptr(y))
    return y


# ------------------------------------------------------------------ k-means
@dataclasses.dataclass
class KMeansResult:
    labels: np.ndarray      # int32, 0..k_eff-1 by ascending centroid
    centroids: np.ndarray   # float64 [k_eff]
    k_eff: int
    cost: float             # total within-cluster sum of squares


def knn_graph(X, k, sigma):
    """Exact kNN graph (self excluded, ties to the smaller index), union
    symmetrised, Gaussian weights: (row_ptr int64, col int32, val float32)."""
    X = _f32(X)
    n, d = X.shape
    rp = np.empty(n + 1, dtype=np.int64)
    col = np.empty(2 * n * int(k), dtype=np.int32)
    val = np.empty(2 * n * int(k), dtype=np.float32)
    nnz = _L().orc_knn_graph(_ptr(X), n, d, int(k), float(np.float32(sigma)), _ptr(rp),
                             _ptr(col), _ptr(val))
    if nnz < 0:
        raise ValueError("k must be in [1, n-1]")
    return rp, col[:nnz].copy(), val[:nnz].copy()


def knn_rows(X, k, sigma, rows):
    """The k nearest neighbours of the listed points, in order (self
    excluded, ties to the smaller index), as the kNN graph defines them:
    (nbr int64 [m, k], squared distances float64 [m, k], weights float32
    [m, k])."""
    X = _f32(X)
    n, d = X.shape
    r = np.ascontiguousarray(rows, dtype=np.int64)
    m = r.shape[0]
    nbr = np.empty((m, int(k)), dtype=np.int64)
    d2 = np.empty((m, int(k)))
    w = np.empty((m, int(k)), dtype=np.float32)
    st = _L().orc_knn_rows(_ptr(X), n, d, int(k), float(np.float32(sigma)), _ptr(r), m,
                           _ptr(nbr), _ptr(d2), _ptr(w))
    if st != 0:
        raise ValueError("k must be in [1, n-1] and rows in [0, n)")
    return nbr, d2, w


def kmeans1d(v, k, method="auto") -> KMeansResult:
    """Exact 1-D k-means; method "plain" (O(k n^2)), "dc" or "auto"."""
    vv = _f64(v)
    n = vv.shape[0]
    if method == "auto":
        method = "plain" if n <= 2000 else "dc"
    m = {"plain": 0, "dc": 1}[method]
    labels = np.empty(n, dtype=np.int32)
    cent = np.empty(max(int(k), 1))
    ke = C.c_int32(0)
    cost = C.c_double(0.0)
    st = _L().orc_kmeans1d(_ptr(vv), n, int(k), m, _ptr(labels), _ptr(cent),
                           C.byref(ke), C.byref(cost))
    if st != 0:
        raise ValueError("k-means failed")
    return KMeansResult(labels, cent[: ke.value].copy(), int(ke.value),
                        float(cost.value))


# --------------------------------------------------------------- end to end
@dataclasses.dataclass
class PICResult:
    A_degree: np.ndarray
    v0: np.ndarray
    pi: PIResult
    km: KMeansResult
    n_zero_rows: int


def pic_dense(X, sigma, k, mode="converge", max_iter=1000, eps=0.0) -> PICResult:
    """Affinity, W = D^-1 A, v0 = D / sum D, Algorithm 1, k-means."""
    A = affinity(X, sigma)
    W, deg, v0, nz = degree_normalize(A)
    del A
    pi = power_iterate_dense(W, v0, mode, max_iter, eps)
    km = kmeans1d(pi.v, k)
    return PICResult(deg, v0, pi, km, nz)
