"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/gpic.h declares, and rejects bad arguments on the
host before any launch."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    import paper_1604_02700_amd as g
    return g.lib()


def _declared():
    src = open(os.path.join(ROOT, "include", "gpic.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return set(re.findall(r"\b(gpic_[a-z0-9_]+)\s*\(", src))


def test_header_and_exports_agree(L):
    import paper_1604_02700_amd as g
    decl = _declared()
    assert decl == set(g.EXPORTS)
    for name in decl:
        assert hasattr(L, name), name
    assert L.gpic_abi_version() == 1


def test_status_strings(L):
    assert L.gpic_status_string(0) == b"GPIC_OK"
    assert L.gpic_status_string(4) == b"GPIC_ERR_NUMERIC"


def test_workspace_sizes(L):
    import paper_1604_02700_amd as g
    for op in ("affinity", "affinity_normalized", "degree_normalize", "degree_fused",
               "pi_dense", "pi_fused", "pi_csr", "kmeans1d", "matvec_fused",
               "affinity_cosine", "affinity_cosine_normalized", "knn_graph"):
        a = g.workspace_bytes(op, 1000, 5000, 3)
        b = g.workspace_bytes(op, 100000, 500000, 3)
        assert 0 < a < b
    assert g.workspace_bytes("kmeans1d", 10**6, 0, 50) > 50 * 4 * 10**6
    # above 2^18 rows the CSR power iteration also holds a column-blocked
    # copy of W (8 bytes per stored entry) and per-block row sums
    small = g.workspace_bytes("pi_csr", 1 << 18, 10**7, 0)
    assert small == g.workspace_bytes("pi_csr", 1 << 18, 0, 0)
    big, big0 = (g.workspace_bytes("pi_csr", 600_000, 10**7, 0),
                 g.workspace_bytes("pi_csr", 600_000, 0, 0))
    assert big - big0 >= 8 * 10**7 and big0 > 3 * 600_000 * 8
    assert L.gpic_workspace_bytes(99, 10, 0, 0) == 0
    assert L.gpic_workspace_bytes(4, -1, 0, 0) == 0


def test_argument_validation_before_launch(L):
    import paper_1604_02700_amd as g
    f = L.gpic_affinity
    dummy = C.c_void_p(4096)               # never dereferenced: checks fail first
    W = (dummy, 1 << 20)                   # workspace pointer and size
    assert f(None, 10, 2, 1.0, dummy, 12, None, *W, None) == 1
    assert f(dummy, 1, 2, 1.0, dummy, 12, None, *W, None) == 1        # n < 2
    assert f(dummy, 10, 0, 1.0, dummy, 12, None, *W, None) == 1       # d < 1
    assert f(dummy, 10, 2, 0.0, dummy, 12, None, *W, None) == 1       # sigma <= 0
    assert f(dummy, 10, 2, float("nan"), dummy, 12, None, *W, None) == 1
    assert f(dummy, 10, 2, 1e-30, dummy, 12, None, *W, None) == 1     # 1/sigma^2 overflows
    assert f(dummy, 10, 2, 1.0, dummy, 9, None, *W, None) == 1        # lda < n
    assert f(dummy, 10, 2, 1.0, dummy, 14, None, *W, None) == 1       # lda % 4
    assert f(dummy, 10, 2, 1.0, C.c_void_p(4100), 12, None, *W, None) == 1  # A misaligned
    assert b"lda" in L.gpic_last_error() or L.gpic_last_error()
    assert f(dummy, 10, 2, 1.0, dummy, 12, None, dummy, 8, None) == 2  # workspace
    fn = L.gpic_affinity_normalized
    assert fn(dummy, 10, 2, 1.0, dummy, 12, dummy, dummy, None, dummy, 8, None) == 2
    assert fn(dummy, 10, 2, 1.0, dummy, 12, None, dummy, None, *W, None) == 1
    fc = L.gpic_affinity_cosine
    assert fc(None, 10, 2, dummy, 12, None, *W, None) == 1
    assert fc(dummy, 1, 2, dummy, 12, None, *W, None) == 1               # n < 2
    assert fc(dummy, 10, 0, dummy, 12, None, *W, None) == 1              # d < 1
    assert fc(dummy, 10, 2, dummy, 9, None, *W, None) == 1               # lda < n
    assert fc(dummy, 10, 2, dummy, 12, None, dummy, 8, None) == 2        # workspace
    kg = L.gpic_knn_graph
    nz = C.c_int64()
    assert kg(dummy, 100, 17, 8, 1.0, dummy, dummy, dummy, C.byref(nz), *W, None) == 5  # d > 16
    assert kg(dummy, 100, 8, 0, 1.0, dummy, dummy, dummy, C.byref(nz), *W, None) == 1   # k < 1
    assert kg(dummy, 100, 8, 65, 1.0, dummy, dummy, dummy, C.byref(nz), *W, None) == 1  # k > 64
    assert kg(dummy, 10, 8, 10, 1.0, dummy, dummy, dummy, C.byref(nz), *W, None) == 1   # k > n-1
    assert kg(dummy, 100, 8, 8, 1.0, dummy, dummy, dummy, None, *W, None) == 1          # nnz null
    assert kg(dummy, 100, 8, 8, 1.0, dummy, dummy, dummy, C.byref(nz), dummy, 8, None) == 2
    fcn = L.gpic_affinity_cosine_normalized
    assert fcn(dummy, 10, 2, dummy, 12, None, dummy, None, *W, None) == 1   # degree null
    assert fcn(dummy, 10, 2, dummy, 12, dummy, dummy, None, dummy, 8, None) == 2
    p = g.PiParams()
    p.mode, p.max_iter, p.eps, p.check_every, p.reserved = 2, 10, 0.0, 0, 0
    r = g.PiResult()
    pi = L.gpic_power_iterate_dense
    assert pi(dummy, 10, 12, C.byref(p), dummy, None, dummy, 1 << 20, C.byref(r), None) == 1
    p.mode, p.eps = 1, -1.0
    assert pi(dummy, 10, 12, C.byref(p), dummy, None, dummy, 1 << 20, C.byref(r), None) == 1
    p.eps, p.reserved = 0.0, 3
    assert pi(dummy, 10, 12, C.byref(p), dummy, None, dummy, 1 << 20, C.byref(r), None) == 1
    p.reserved = 0
    assert pi(dummy, 10, 12, C.byref(p), dummy, None, dummy, 16, C.byref(r), None) == 2
    assert pi(dummy, 10, 12, C.byref(p), dummy, None, None, 0, C.byref(r), None) == 2
    km = L.gpic_kmeans1d
    ke = C.c_int32()
    assert km(dummy, 5, 6, dummy, dummy, C.byref(ke), None, dummy, 1 << 20, None) == 1
    assert km(dummy, 5, 0, dummy, dummy, C.byref(ke), None, dummy, 1 << 20, None) == 1
    assert km(dummy, 5, 2, dummy, dummy, None, None, dummy, 1 << 20, None) == 1
    assert km(dummy, 5, 2, dummy, dummy, C.byref(ke), None, dummy, 8, None) == 2
