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


def test_sym_bytes_limits():
    """The symmetric storage's size: nb(nb+1)/2 tiles of 256 x 256 float32,
    nb = ceil(n / 256); 0 outside 2 <= n <= 2^24."""
    import paper_1604_02700_amd as g
    for n in (2, 255, 256, 257, 50000):
        nb = (n + 255) // 256
        assert g.sym_bytes(n) == nb * (nb + 1) // 2 * 65536 * 4
    assert g.sym_bytes(1) == 0 and g.sym_bytes((1 << 24) + 1) == 0


def test_sym_and_host_validation(L):
    """The symmetric and out-of-core entry points reject bad arguments on
    the host before any launch."""
    import paper_1604_02700_amd as g
    for op in ("affinity_sym", "matvec_sym", "pi_sym", "pi_dense_host"):
        a = g.workspace_bytes(op, 1000)
        b = g.workspace_bytes(op, 100000)
        assert 0 < a < b
    dummy = C.c_void_p(4096)
    W = (dummy, 1 << 30)
    fa = L.gpic_affinity_sym
    assert fa(None, 10, 2, 1.0, dummy, dummy, dummy, None, *W, None) == 1      # X null
    assert fa(dummy, 10, 2, 1.0, None, dummy, dummy, None, *W, None) == 1      # As null
    assert fa(dummy, 10, 2, 1.0, C.c_void_p(4100), dummy, dummy, None, *W, None) == 1
    assert fa(dummy, 10, 2, 0.0, dummy, dummy, dummy, None, *W, None) == 1     # sigma
    assert fa(dummy, (1 << 24) + 1, 2, 1.0, dummy, dummy, dummy, None, *W, None) == 1
    assert fa(dummy, 10, 2, 1.0, dummy, dummy, dummy, None, dummy, 8, None) == 2
    mv = L.gpic_matvec_sym
    assert mv(dummy, 1, dummy, dummy, dummy, *W, None) == 1                   # n < 2
    assert mv(dummy, 10, None, dummy, dummy, *W, None) == 1                   # degree null
    assert mv(dummy, 10, dummy, dummy, dummy, dummy, 8, None) == 2            # workspace
    p = g.PiParams()
    p.mode, p.max_iter, p.eps, p.check_every, p.reserved = 0, 5, 0.0, 0, 0
    r = g.PiResult()
    ps = L.gpic_power_iterate_sym
    assert ps(dummy, 10, None, C.byref(p), dummy, None, *W, C.byref(r), None) == 1
    assert ps(dummy, 10, dummy, C.byref(p), dummy, None, dummy, 8, C.byref(r), None) == 2
    ph = L.gpic_power_iterate_dense_host
    assert ph(None, 10, 10, C.byref(p), dummy, None, *W, C.byref(r), None) == 1
    assert ph(dummy, 10, 9, C.byref(p), dummy, None, *W, C.byref(r), None) == 1   # ldw < n
    small = g.workspace_bytes("pi_dense", 10)
    assert ph(dummy, 10, 10, C.byref(p), dummy, None, dummy, small, C.byref(r), None) == 2


def test_read_stream_validation(L):
    """The read-bandwidth reference rejects bad buffers on the host."""
    dummy = C.c_void_p(4096)
    rs = L.gpic_read_stream
    assert rs(None, 16, dummy, None) == 1                      # x null
    assert rs(C.c_void_p(4100), 16, dummy, None) == 1          # x misaligned
    assert rs(dummy, 18, dummy, None) == 1                     # n % 4 != 0
    assert rs(dummy, 0, dummy, None) == 1                      # empty
    assert rs(dummy, 16, None, None) == 1                      # sink null


def test_noalloc_validation(L):
    """The no-allocation dense power iteration checks its arguments and its
    size limit on the host, before it looks up its static scratch or
    launches anything."""
    import paper_1604_02700_amd as g
    # the documented limit is the largest n whose power-iteration state fits
    assert (g.workspace_bytes("pi_dense", g.NOALLOC_MAX_N) <= g.NOALLOC_SCRATCH_BYTES
            < g.workspace_bytes("pi_dense", g.NOALLOC_MAX_N + 1))
    dummy = C.c_void_p(4096)
    p = g.PiParams()
    p.mode, p.max_iter, p.eps, p.check_every, p.reserved = 0, 5, 0.0, 0, 0
    r = g.PiResult()
    fn = L.gpic_power_iterate_dense_noalloc
    assert fn(None, 10, 12, C.byref(p), dummy, None, C.byref(r), None) == 1     # W null
    assert fn(dummy, 10, 9, C.byref(p), dummy, None, C.byref(r), None) == 1     # ldw < n
    assert fn(dummy, 10, 12, C.byref(p), None, None, C.byref(r), None) == 1     # v null
    assert fn(dummy, 10, 12, C.byref(p), dummy, None, None, None) == 1          # res null
    n = g.NOALLOC_MAX_N + 1
    assert fn(dummy, n, n + 3, C.byref(p), dummy, None, C.byref(r), None) == 2
    assert b"static scratch" in L.gpic_last_error()
