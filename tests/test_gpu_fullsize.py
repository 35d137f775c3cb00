"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times.

* 16-D blobs, n = 50,000 (dense W of 2.5e9 entries): the oracle runs the
  whole path (20 GB of float64 W on the host), so v, the statistics, the
  stop iteration and the labels are compared element by element.
* 64-D blobs, n = 200,000 (fused operator): the oracle cannot run 31
  sweeps of 4e10 pairs, so sampled rows are recomputed one by one (degrees
  and one product from the GPU's own iterate), plus invariants of the whole
  vector; a reduced n runs end to end.
* kNN graph (CSR) at a reduced n, end to end, and at its full size
  (n = 2,000,000, the column-blocked product) to convergence.
* 1-D k-means at the kNN workload's full size (n = 2,000,000, k = 50).
* The paper's Experiment I shape at its largest size: two moons, n = 45,000,
  cosine affinity, at most 3 updates, end to end.
* The kNN input graph built on the GPU: against the oracle's brute force at
  n = 200,000 and against the scipy k-d tree graph of the kNN workload at
  n = 2,000,000.
"""
import numpy as np
import pytest

from gpu_helpers import check_kmeans, check_labels, rel_l1, stop_margin

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"


@pytest.fixture(scope="module")
def g():
    import paper_1604_02700_amd as g
    g.lib()
    assert torch.cuda.is_available()
    return g


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.fixture(scope="module")
def knn8d():
    """The full kNN workload (its scipy k-d tree graph takes minutes on the
    host), built once for the module."""
    import workloads
    return workloads.make("knn8d")


@pytest.fixture(scope="module")
def blobs16d():
    import workloads
    return workloads.make("blobs16d")


@pytest.fixture(scope="module")
def blobs16d_oracle(orc, blobs16d):
    w = blobs16d
    print(f"oracle: blobs16d n={w.n} (affinity, normalise, T=50)", flush=True)
    W = orc.affinity(w.X, w.sigma)
    W, deg, v0, nz = orc.degree_normalize(W, copy=False)
    fixed = orc.power_iterate_dense(W, v0, "fixed", 50)
    conv = orc.power_iterate_dense(W, v0, "converge", 1000, w.eps)
    del W
    km = orc.kmeans1d(fixed.v, w.k)
    return {"deg": deg, "v0": v0, "fixed": fixed, "conv": conv, "km": km}


def test_blobs16d_full_fixed_T(g, orc, blobs16d, blobs16d_oracle):
    w, ref = blobs16d, blobs16d_oracle
    print(f"gpu: blobs16d n={w.n} fixed T=50", flush=True)
    W, deg, v0, nz = g.gpic_affinity_normalized(_t(w.X), w.sigma)
    np.testing.assert_allclose(deg.cpu().numpy(), ref["deg"], rtol=1e-5)
    np.testing.assert_allclose(v0.cpu().numpy(), ref["v0"], rtol=1e-5)
    v = v0.clone()
    out = g.gpic_power_iterate_dense(W, v, None, "fixed", 50, n=w.n)
    vg = v.cpu().numpy()
    err = rel_l1(vg, ref["fixed"].v)
    print(f"  rel_l1 = {err:.3e}", flush=True)
    assert out.iterations == 50 and err <= 1e-4
    np.testing.assert_allclose(out.stats, ref["fixed"].stats, rtol=1e-3,
                               atol=1e-3 * w.eps)
    assert np.all(vg >= 0) and abs(vg.sum() - 1.0) < 1e-12
    km = g.gpic_kmeans1d(v, w.k)
    assert km.k_eff == ref["km"].k_eff == w.k
    check_labels(orc, f"blobs16d n={w.n} T=50", ref["fixed"].v, ref["km"].labels, vg, km,
                 w.k)
    # k-means parity on the same (GPU) embedding, whatever the guard: the
    # identical optimum
    kmo = orc.kmeans1d(vg, w.k, "dc")
    assert km.cost == pytest.approx(kmo.cost, rel=1e-9)
    # determinism at full size
    v2 = v0.clone()
    out2 = g.gpic_power_iterate_dense(W, v2, None, "fixed", 50, n=w.n)
    assert torch.equal(v, v2) and np.array_equal(out.stats, out2.stats)


def test_blobs16d_full_converge(g, blobs16d, blobs16d_oracle):
    w, ref = blobs16d, blobs16d_oracle
    out = g.pic_dense(_t(w.X), w.sigma, w.k, "converge", 1000, w.eps)
    conv = ref["conv"]
    mu = stop_margin(conv.stats, w.eps, conv.iterations)
    print(f"  iterations gpu={out.pi.iterations} oracle={conv.iterations} "
          f"margin={mu:.3g}", flush=True)
    assert conv.converged and out.pi.converged
    assert out.pi.iterations == conv.iterations
    assert rel_l1(out.pi.v.cpu().numpy(), conv.v) <= 1e-4


def test_blobs16d_full_sym(g, blobs16d, blobs16d_oracle):
    """The same workload over the symmetric storage (5.06 GB of tiles):
    T = 50 and to convergence against the oracle."""
    w, ref = blobs16d, blobs16d_oracle
    print(f"gpu: blobs16d n={w.n} symmetric storage", flush=True)
    out = g.pic_sym(_t(w.X), w.sigma, w.k, "fixed", 50)
    np.testing.assert_allclose(out.degree.cpu().numpy(), ref["deg"], rtol=1e-5)
    vg = out.pi.v.cpu().numpy()
    err = rel_l1(vg, ref["fixed"].v)
    print(f"  rel_l1 = {err:.3e}", flush=True)
    assert out.pi.iterations == 50 and err <= 1e-4
    np.testing.assert_allclose(out.pi.stats, ref["fixed"].stats, rtol=1e-3,
                               atol=1e-3 * w.eps)
    del out
    conv = g.pic_sym(_t(w.X), w.sigma, w.k, "converge", 1000, w.eps)
    assert conv.pi.converged and conv.pi.iterations == ref["conv"].iterations
    assert rel_l1(conv.pi.v.cpu().numpy(), ref["conv"].v) <= 1e-4


def test_blobs64d_full_size_sampled(g, orc):
    """n = 200,000, d = 64, fused operator, T = 30: sampled rows one by one."""
    import workloads
    w = workloads.make("blobs64d")
    X = _t(w.X)
    print(f"gpu: blobs64d n={w.n} fused T=30", flush=True)
    deg, v0, nz = g.gpic_degree_fused(X, w.sigma)
    v = v0.clone()
    out = g.gpic_power_iterate_fused(X, w.sigma, deg, v, None, "fixed", 29)
    v29 = v.clone()
    g.gpic_power_iterate_fused(X, w.sigma, deg, v, None, "fixed", 1)
    rng = np.random.default_rng(0)
    rows = np.concatenate([[0, 1, w.n // 2, w.n - 1],
                           rng.choice(w.n, 28, replace=False)]).astype(np.int64)
    dr = orc.degree_rows(w.X, w.sigma, rows)
    np.testing.assert_allclose(deg.cpu().numpy()[rows], dr, rtol=1e-4)
    # one product from the GPU's own iterate, against the oracle's rows
    y = g.gpic_matvec_fused(X, w.sigma, deg, v29).cpu().numpy()
    dfull = np.zeros(w.n)
    dfull[rows] = dr
    yr = orc.matvec_onthefly_rows(w.X, w.sigma, dfull, v29.cpu().numpy(), rows)
    np.testing.assert_allclose(y[rows], yr, rtol=1e-4)
    # the last update is y / ||y||_1 of that product
    vg = v.cpu().numpy()
    np.testing.assert_allclose(vg, y / np.abs(y).sum(), rtol=1e-12)
    assert np.all(vg >= 0) and abs(vg.sum() - 1) < 1e-12
    assert out.iterations == 29


def test_blobs64d_reduced_end_to_end(g, orc):
    """Same generator at n = 6,000: the whole fused path against the oracle."""
    import workloads
    w = workloads.make("blobs64d", n=6000)
    out = g.pic_fused(_t(w.X), w.sigma, w.k, "fixed", 30)
    dr, v0r, _ = orc.degree_onthefly(w.X, w.sigma)
    ref = orc.power_iterate_onthefly(w.X, w.sigma, dr, v0r, "fixed", 30)
    np.testing.assert_allclose(out.degree.cpu().numpy(), dr, rtol=1e-4)
    vg = out.pi.v.cpu().numpy()
    assert rel_l1(vg, ref.v) <= 1e-4
    km = orc.kmeans1d(ref.v, w.k)
    check_labels(orc, f"blobs64d fused n={w.n}", ref.v, km.labels, vg, out.km, w.k)


def test_knn_csr_relabelled_matches_original(g):
    """Renumbering the graph's nodes permutes v (up to summation order)."""
    import workloads
    w = workloads.make("knn8d", n=50000)
    r = workloads.relabel_rcm(w)
    outs = []
    for x in (w, r):
        outs.append(g.pic_csr(_t(x.row_ptr), _t(x.col), _t(x.val.copy()), x.k, "fixed",
                              20))
    perm = np.empty(w.n, dtype=np.int64)
    # r.X[i] == w.X[perm_i]: recover perm from the points
    order_w = np.lexsort(w.X.T[::-1])
    order_r = np.lexsort(r.X.T[::-1])
    perm[order_r] = order_w
    assert np.array_equal(r.X, w.X[perm])
    v0 = outs[0].pi.v.cpu().numpy()
    v1 = outs[1].pi.v.cpu().numpy()
    np.testing.assert_allclose(v1, v0[perm], rtol=1e-10)


def test_knn_csr_reduced_end_to_end(g, orc):
    """kNN graph path at n = 100,000 (same generator), to convergence."""
    import workloads
    w = workloads.make("knn8d", n=100000)
    print(f"gpu: knn8d n={w.n} nnz={w.val.shape[0]}", flush=True)
    out = g.pic_csr(_t(w.row_ptr), _t(w.col), _t(w.val.copy()), w.k, "converge",
                    1000, w.eps)
    wr, dr, v0r, _ = orc.degree_normalize_csr(w.row_ptr, w.col, w.val)
    ref = orc.power_iterate_csr(w.row_ptr, w.col, wr, v0r, "converge", 1000, w.eps)
    mu = stop_margin(ref.stats, w.eps, ref.iterations)
    print(f"  iterations gpu={out.pi.iterations} oracle={ref.iterations} "
          f"margin={mu:.3g}", flush=True)
    np.testing.assert_allclose(out.degree.cpu().numpy(), dr, rtol=1e-12)
    assert ref.converged == out.pi.converged
    assert out.pi.iterations == ref.iterations
    vg = out.pi.v.cpu().numpy()
    assert rel_l1(vg, ref.v) <= 1e-4
    check_labels(orc, f"knn8d csr n={w.n}", ref.v, orc.kmeans1d(ref.v, w.k, "dc").labels,
                 vg, out.km, w.k)


def test_kmeans1d_full_size(g, orc):
    """n = 2,000,000 scalars into k = 50 clusters: the exact optimum."""
    rng = np.random.default_rng(2_000_050)
    n, k = 2_000_000, 50
    centres = np.sort(rng.uniform(0, 100, size=k))
    v = centres[rng.integers(0, k, size=n)] + rng.standard_normal(n) * 0.5
    print(f"gpu: kmeans1d n={n} k={k}", flush=True)
    out = g.gpic_kmeans1d(_t(v), k)
    check_kmeans(v, out, orc.kmeans1d(v, k, "dc"))


def test_knn_csr_full_size_converge(g, orc, knn8d):
    """knn8d at n = 2,000,000 (90M stored entries, random node order): the
    column-blocked product to convergence against the oracle."""
    w = knn8d
    print(f"gpu: knn8d n={w.n} nnz={w.val.shape[0]}", flush=True)
    out = g.pic_csr(_t(w.row_ptr), _t(w.col), _t(w.val.copy()), w.k, "converge",
                    1000, w.eps)
    wr, dr, v0r, _ = orc.degree_normalize_csr(w.row_ptr, w.col, w.val)
    ref = orc.power_iterate_csr(w.row_ptr, w.col, wr, v0r, "converge", 1000, w.eps)
    mu = stop_margin(ref.stats, w.eps, ref.iterations)
    print(f"  iterations gpu={out.pi.iterations} oracle={ref.iterations} "
          f"margin={mu:.3g}", flush=True)
    np.testing.assert_allclose(out.degree.cpu().numpy(), dr, rtol=1e-12)
    assert ref.converged and out.pi.converged
    assert out.pi.iterations == ref.iterations
    vg = out.pi.v.cpu().numpy()
    assert rel_l1(vg, ref.v) <= 1e-4
    check_labels(orc, f"knn8d csr n={w.n}", ref.v, orc.kmeans1d(ref.v, w.k, "dc").labels,
                 vg, out.km, w.k)


def test_knn_csr_full_size_local_order(g, orc, knn8d):
    """knn8d at n = 2,000,000 with the graph built on the GPU in the Morton
    numbering of the points (the staged product, gathers near the row):
    to convergence against the oracle on that same graph, and the graph
    itself equal to the workload's k-d tree graph relabelled."""
    w = knn8d
    print(f"gpu: knn8d n={w.n} local numbering", flush=True)
    rp, col, val, perm = g.gpic_knn_graph_local(_t(w.X), 32, 1.0)
    perm = perm.cpu().numpy()
    rph, colh, valh = rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy()
    import scipy.sparse as sp
    S = sp.csr_matrix((w.val, w.col, w.row_ptr), shape=(w.n, w.n))[perm][:, perm].tocsr()
    S.sort_indices()
    assert np.array_equal(rph, S.indptr) and np.array_equal(colh, S.indices)
    assert np.all(np.abs(valh - S.data) <= np.spacing(S.data))
    del S
    out = g.pic_csr(rp, col, val, w.k, "converge", 1000, w.eps)
    wr, dr, v0r, _ = orc.degree_normalize_csr(rph, colh, valh)
    ref = orc.power_iterate_csr(rph, colh, wr, v0r, "converge", 1000, w.eps)
    mu = stop_margin(ref.stats, w.eps, ref.iterations)
    print(f"  iterations gpu={out.pi.iterations} oracle={ref.iterations} "
          f"margin={mu:.3g}", flush=True)
    np.testing.assert_allclose(out.degree.cpu().numpy(), dr, rtol=1e-12)
    assert ref.converged and out.pi.converged
    assert out.pi.iterations == ref.iterations
    vg = out.pi.v.cpu().numpy()
    assert rel_l1(vg, ref.v) <= 1e-4
    check_labels(orc, f"knn8d csr local n={w.n}", ref.v,
                 orc.kmeans1d(ref.v, w.k, "dc").labels, vg, out.km, w.k)


def test_moons_full_size_cosine(g, orc):
    """Two moons, n = 45,000, cosine affinity (dense W of 8.1 GB), at most 3
    updates with eps = 1e-5 / n: degrees, stop and v against the oracle."""
    import workloads
    w = workloads.make("moons")
    print(f"gpu: moons n={w.n} cosine, <= {w.max_iter} updates", flush=True)
    out = g.pic_cosine(_t(w.X), w.k, "converge", w.max_iter, w.eps)
    vg = out.pi.v.cpu().numpy()
    dg = out.degree.cpu().numpy()
    it, conv = out.pi.iterations, out.pi.converged
    km = out.km
    del out
    torch.cuda.empty_cache()
    print("oracle: moons n=45000 (cosine affinity, normalise, <= 3 updates)", flush=True)
    A = orc.affinity_cosine(w.X)
    W, deg, v0, _ = orc.degree_normalize(A, copy=False)
    ref = orc.power_iterate_dense(W, v0, "converge", w.max_iter, w.eps)
    del A, W
    np.testing.assert_allclose(dg, deg, rtol=1e-5)
    assert it == ref.iterations and conv == ref.converged
    assert rel_l1(vg, ref.v) <= 1e-4
    check_labels(orc, f"moons cosine n={w.n}", ref.v, orc.kmeans1d(ref.v, w.k).labels, vg,
                 km, w.k)


def test_knn_graph_200k(g, orc):
    """n = 200,000 points of the kNN workload's generator, k = 32."""
    import workloads
    w = workloads.make("knn8d", n=200000)
    print(f"gpu: knn graph n={w.n} d={w.d} k=32", flush=True)
    rp, col, val = g.gpic_knn_graph(_t(w.X), 32, 1.0)
    rp, col, val = rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy()
    print("oracle: brute-force kNN graph n=200000", flush=True)
    rpo, colo, valo = orc.knn_graph(w.X, 32, 1.0)
    assert np.array_equal(rp, rpo) and np.array_equal(col, colo)
    assert np.all(np.abs(val - valo) <= np.spacing(valo))


def test_knn_graph_full_size(g, knn8d):
    """n = 2,000,000: the same graph as the workload's (scipy k-d tree, exact
    kNN, union, float64 weights); weights within one float32 ulp."""
    w = knn8d
    print(f"gpu: knn graph n={w.n} d={w.d} k=32", flush=True)
    rp, col, val = g.gpic_knn_graph(_t(w.X), 32, 1.0)
    assert np.array_equal(rp.cpu().numpy(), w.row_ptr)
    assert np.array_equal(col.cpu().numpy(), w.col)
    vg = val.cpu().numpy()
    assert np.all(np.abs(vg - w.val) <= np.spacing(w.val))
