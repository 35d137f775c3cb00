"""The dense power iteration's no-allocation entry point
(gpic_power_iterate_dense_noalloc: its scratch in the library's static
device array) against the workspace entry point, through the C ABI: the
same kernels in the same order, so v, delta, the statistics and the stop
update must be identical, on two calls in a row (the second smaller, over
the scratch the first left behind)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"


@pytest.fixture(scope="module")
def g():
    import paper_1604_02700_amd as g
    g.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return g


@pytest.mark.parametrize("mode", ["fixed", "converge"])
def test_noalloc_equals_workspace_entry_point(g, mode):
    import workloads
    for n in (3001, 1203):
        w = workloads.make("blobs16d", n=n)
        eps = 1e-5 / n
        T = 30 if mode == "fixed" else 1000
        print(f"noalloc dense n={n} mode={mode}", flush=True)
        X = torch.from_numpy(w.X).to(DEV)
        W, deg, v0, _ = g.gpic_affinity_normalized(X, w.sigma)
        a = v0.clone()
        ra = g.gpic_power_iterate_dense(W, a, None, mode, T, eps, n=n)
        b = v0.clone()
        rb = g.gpic_power_iterate_dense_noalloc(W, b, None, mode, T, eps, n=n)
        torch.cuda.synchronize()
        assert ra.iterations == rb.iterations and ra.converged == rb.converged
        assert rb.iterations == (T if mode == "fixed" else rb.iterations) > 0
        assert torch.equal(a, b)
        assert np.array_equal(ra.stats, rb.stats)
        # the caller's own delta (resume form): a further 5 updates each
        da, db = a.clone(), b.clone()
        g.gpic_power_iterate_dense(W, a, da, "fixed", 5, n=n)
        g.gpic_power_iterate_dense_noalloc(W, b, db, "fixed", 5, n=n)
        torch.cuda.synchronize()
        assert torch.equal(a, b) and torch.equal(da, db)


def test_noalloc_rejects_too_large_n(g):
    """Above the scratch's limit the call fails before any launch (W is a
    single row with the row pitch of n: nothing is read)."""
    n = g.NOALLOC_MAX_N + 1
    W = torch.zeros((1, (n + 3) // 4 * 4), dtype=torch.float32, device=DEV)
    v = torch.zeros(n, dtype=torch.float64, device=DEV)
    with pytest.raises(g.GpicError) as ei:
        g.gpic_power_iterate_dense_noalloc(W, v, None, "fixed", 1, n=n)
    assert ei.value.status == 2
