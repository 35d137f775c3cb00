"""GPU parity: the HIP path through the C ABI against the oracle.

Every comparison runs the same seeded inputs through both sides.  The GPU
stores X, A and W in float32 and keeps every accumulation and the iteration
state in float64; the oracle is float64 throughout.
"""
import numpy as np
import pytest

from gpu_helpers import (cosine_tolerance, EPS32, affinity_tolerance, check_kmeans,
                         check_labels, matched_agreement, rel_l1, stop_margin)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def g():
    import paper_1604_02700_amd as g
    g.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return g


DEV = "cuda:0"


def _pts(n, d, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return (scale * rng.standard_normal((n, d))).astype(np.float32)


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


# --------------------------------------------------------------- affinity
@pytest.mark.parametrize("n,d", [(2, 2), (3, 1), (63, 2), (64, 3), (65, 15),
                                 (1000, 2), (1023, 5), (130, 16), (257, 17),
                                 (200, 64), (129, 40), (77, 130), (150, 128),
                                 (4100, 16), (70, 110)])
def test_affinity_parity(g, orc, n, d):
    X = _pts(n, d, 1000 + n + d, scale=2.0)
    sigma = np.float32(1.5 * np.sqrt(d))
    print(f"affinity n={n} d={d}", flush=True)
    A, deg = g.gpic_affinity(_t(X), sigma)
    torch.cuda.synchronize()
    Ag = A[:, :n].cpu().numpy().astype(np.float64)
    Ar = orc.affinity(X, sigma)
    gram = 16 <= d <= 128
    tol = affinity_tolerance(X, sigma, Ar, gram)
    err = np.abs(Ag - Ar)
    assert np.all(np.diag(Ag) == 0.0)
    assert np.all(err <= tol), f"max err/tol {np.max(err / tol):.3g}"
    # degrees are the float64 sums of the stored float32 values
    np.testing.assert_allclose(deg.cpu().numpy(), Ag.sum(1), rtol=1e-13)


@pytest.mark.parametrize("n,d,offset", [(700, 16, 1.0e4), (300, 64, -3.0e3), (257, 33, 250.0)])
def test_affinity_offset_points(g, orc, n, d, offset):
    """Points far from the origin (a common offset much larger than their
    spread): the Gram form runs on centred coordinates, so its error scales
    with the spread; against the oracle's difference form, the same bound
    as for centred data, and the fused operator's degrees to 1e-5."""
    X = (_pts(n, d, 3000 + d, scale=1.0) + np.float32(offset)).astype(np.float32)
    sigma = np.float32(np.sqrt(d))
    print(f"affinity offset n={n} d={d} offset={offset}", flush=True)
    A, deg = g.gpic_affinity(_t(X), sigma)
    torch.cuda.synchronize()
    Ag = A[:, :n].cpu().numpy().astype(np.float64)
    Ar = orc.affinity(X, sigma)
    tol = affinity_tolerance(X, sigma, Ar, True)
    err = np.abs(Ag - Ar)
    assert np.all(err <= tol), f"max err/tol {np.max(err / tol):.3g}"
    assert np.max(err) <= 1e-5 * np.max(Ar)
    degf, _, _ = g.gpic_degree_fused(_t(X), sigma)
    dr, _, _ = orc.degree_onthefly(X, sigma)
    np.testing.assert_allclose(degf.cpu().numpy(), dr, rtol=1e-5)


def _with_outlier(X, far):
    """X plus one point `far` away from the first point along every
    coordinate (a single far point among clustered ones)."""
    return np.vstack([X, (X[0] + np.float32(far))[None, :]]).astype(np.float32)


@pytest.mark.parametrize("n,d,far", [(700, 16, 1.0e4), (700, 16, 1.0e5), (300, 64, 1.0e4),
                                     (257, 33, -3.0e4)])
def test_affinity_outlier_points(g, orc, n, d, far):
    """One point far from all others: each point is split in its own scale
    around a median centre, so the far point coarsens only its own row and
    column.  Every entry within the per-pair bound (which carries only the
    pair's own norms), and the entries among the other points within 1e-5
    of the largest entry."""
    X = _with_outlier(_pts(n, d, 3100 + d, scale=1.0), far)
    sigma = np.float32(np.sqrt(d))
    print(f"affinity outlier n={n}+1 d={d} far={far}", flush=True)
    A, deg = g.gpic_affinity(_t(X), sigma)
    torch.cuda.synchronize()
    Ag = A[:, :n + 1].cpu().numpy().astype(np.float64)
    Ar = orc.affinity(X, sigma)
    tol = affinity_tolerance(X, sigma, Ar, True)
    err = np.abs(Ag - Ar)
    assert np.all(err <= tol), f"max err/tol {np.max(err / tol):.3g}"
    assert np.max(err[:n, :n]) <= 1e-5 * np.max(Ar)
    np.testing.assert_allclose(deg.cpu().numpy(), Ag.sum(1), rtol=1e-13)


@pytest.mark.parametrize("far", [1.0e4, 1.0e5])
@pytest.mark.parametrize("sigma_kind", ["one", "median"])
def test_affinity_outlier_end_to_end(g, orc, far, sigma_kind):
    """The 16-D blob shape at n = 4,099 plus one point far from all others
    (at sigma = 1 its row of A underflows to zero: a zero-degree row): v
    after T = 50 within relative L1 1e-4 and the same stop update as the
    oracle, through the matrix-core affinity."""
    import workloads
    w = workloads.make("blobs16d", n=4099)
    X = _with_outlier(w.X, far)
    sigma = np.float32(1.0) if sigma_kind == "one" else w.sigma
    n = X.shape[0]
    eps = 1e-5 / n
    print(f"pic_dense blobs16d n=4099+1 far={far} sigma={float(sigma)}", flush=True)
    out = g.pic_dense(_t(X), sigma, w.k, "fixed", 50)
    conv = g.pic_dense(_t(X), sigma, w.k, "converge", 1000, eps)
    torch.cuda.synchronize()
    Ar = orc.affinity(X, sigma)
    # degrees: within the sum of their entries' bounds (at sigma = 1 every
    # entry is tiny and its relative error is the Gram form's absolute
    # error in dist2 over 2 sigma^2)
    dtol = affinity_tolerance(X, sigma, Ar, True).sum(1)
    Wr, dr, v0r, nzr = orc.degree_normalize(Ar, copy=False)
    del Ar
    ref = orc.power_iterate_dense(Wr, v0r, "fixed", 50)
    refc = orc.power_iterate_dense(Wr, v0r, "converge", 1000, eps)
    del Wr
    assert out.n_zero_rows == nzr
    derr = np.abs(out.degree.cpu().numpy() - dr)
    assert np.all(derr <= dtol), f"degree err/tol {np.max(derr / dtol):.3g}"
    v = out.pi.v.cpu().numpy()
    err = rel_l1(v, ref.v)
    mu = stop_margin(refc.stats, eps, refc.iterations)
    print(f"  rel_l1 = {err:.3e}; iterations gpu={conv.pi.iterations} "
          f"oracle={refc.iterations} margin={mu:.3g}", flush=True)
    assert out.pi.iterations == 50 and err <= 1e-4
    assert conv.pi.converged == refc.converged
    assert conv.pi.iterations == refc.iterations
    assert rel_l1(conv.pi.v.cpu().numpy(), refc.v) <= 1e-4


@pytest.mark.parametrize("n,d", [(2, 2), (3, 1), (64, 2), (1000, 2), (1023, 5),
                                 (300, 16), (257, 17), (99, 40)])
def test_cosine_affinity_parity(g, orc, n, d):
    """Cosine affinity (1 + cos) / 2 against the oracle, with the origin and
    an antipodal pair among the points."""
    X = _pts(n, d, 2000 + n + d, scale=2.0)
    X[0] = 0.0
    if n > 2:
        X[2] = -X[1] * np.float32(3.0)            # cos = -1 with row 1
    print(f"cosine affinity n={n} d={d}", flush=True)
    A, deg = g.gpic_affinity_cosine(_t(X))
    torch.cuda.synchronize()
    Ag = A[:, :n].cpu().numpy().astype(np.float64)
    Ar = orc.affinity_cosine(X)
    assert np.all(np.diag(Ag) == 0.0) and Ag.min() >= 0.0
    err = np.abs(Ag - Ar)
    assert err.max() <= cosine_tolerance(d), f"max err {err.max():.3g}"
    assert np.all(Ag[0, 1:] == 0.5) and np.all(Ag[1:, 0] == 0.5)
    np.testing.assert_allclose(deg.cpu().numpy(), Ag.sum(1), rtol=1e-13)


@pytest.mark.parametrize("n,d", [(777, 2), (1025, 16)])
def test_cosine_normalized_equals_two_calls(g, n, d):
    X = _pts(n, d, 3000 + n, scale=1.5)
    A, deg = g.gpic_affinity_cosine(_t(X))
    W2, deg2, v02, _ = g.gpic_degree_normalize(A, n, deg, True)
    W, degree, v0, nz = g.gpic_affinity_cosine_normalized(_t(X))
    torch.cuda.synchronize()
    assert torch.equal(W[:, :n], W2[:, :n]) and torch.equal(degree, deg2)
    assert torch.equal(v0, v02) and int(nz.item()) == 0


def test_affinity_padding_untouched(g):
    n, d = 37, 2
    X = _pts(n, d, 5)
    A = torch.full((n, 44), -7.0, dtype=torch.float32, device=DEV)
    g.gpic_affinity(_t(X), 1.0, A)
    torch.cuda.synchronize()
    assert torch.all(A[:, n:] == -7.0)


# ------------------------------------------------------- degree / normalise
@pytest.mark.parametrize("given", [False, True])
def test_degree_normalize_parity(g, orc, given):
    n, d = 777, 3
    X = _pts(n, d, 7)
    sigma = np.float32(1.1)
    A, deg = g.gpic_affinity(_t(X), sigma)
    Ag = A[:, :n].cpu().numpy().astype(np.float64)
    W, degree, v0, nz = g.gpic_degree_normalize(A, n, deg if given else None, given)
    torch.cuda.synchronize()
    Wg = W[:, :n].cpu().numpy().astype(np.float64)
    Wr, dr, v0r, nzr = orc.degree_normalize(orc.affinity(X, sigma))
    # against the oracle's float64 chain
    np.testing.assert_allclose(degree.cpu().numpy(), dr, rtol=2e-6)
    np.testing.assert_allclose(v0.cpu().numpy(), v0r, rtol=4e-6)
    np.testing.assert_allclose(Wg, Wr, rtol=4e-6, atol=1e-37)
    # exactly what this stage computes from the stored float32 A
    np.testing.assert_allclose(degree.cpu().numpy(), Ag.sum(1), rtol=1e-13)
    np.testing.assert_allclose(Wg, Ag / Ag.sum(1)[:, None], rtol=2 * EPS32, atol=1e-38)
    np.testing.assert_allclose(Wg.sum(1), 1.0, atol=n * EPS32)       # pin P1
    assert int(nz.item()) == nzr == 0


@pytest.mark.parametrize("n,d", [(777, 3), (1025, 16), (300, 64), (99, 130)])
def test_affinity_normalized_equals_two_calls(g, n, d):
    """W written in one call is bitwise the two-call result (affinity with
    row sums, then in-place scaling with the given degrees)."""
    X = _pts(n, d, 60 + d, scale=1.3)
    sigma = np.float32(np.sqrt(d))
    W1, deg1, v01, nz1 = g.gpic_affinity_normalized(_t(X), sigma)
    A, deg = g.gpic_affinity(_t(X), sigma)
    W2, deg2, v02, nz2 = g.gpic_degree_normalize(A, n, deg, True)
    torch.cuda.synchronize()
    assert torch.equal(deg1, deg2) and torch.equal(v01, v02)
    assert torch.equal(W1[:, :n], W2[:, :n])
    assert int(nz1.item()) == int(nz2.item()) == 0


def test_zero_degree_rows_and_numeric_error(g):
    X = np.array([[0, 0], [0.1, 0], [1000, 1000], [0.2, 0.1]], dtype=np.float32)
    A, deg = g.gpic_affinity(_t(X), 0.05)
    W, degree, v0, nz = g.gpic_degree_normalize(A, 4, deg, True)
    torch.cuda.synchronize()
    assert int(nz.item()) == 1 and float(v0[2]) == 0.0
    assert torch.all(W[2, :4] == 0)
    Z = torch.zeros((4, 4), dtype=torch.float32, device=DEV)
    with pytest.raises(g.GpicError) as ei:
        g.gpic_degree_normalize(Z, 4)
    assert ei.value.status == 4


# -------------------------------------------------------- power iteration
def _oracle_on_fp32_W(orc, X, sigma):
    """The oracle's W rounded once to float32 (stage isolation input)."""
    W, deg, v0, _ = orc.degree_normalize(orc.affinity(X, sigma))
    W32 = W.astype(np.float32)
    return W32, v0


@pytest.mark.parametrize("n", [5, 64, 513, 2050])
def test_power_iteration_stage_isolation(g, orc, n):
    """Same float32 W into both sides: only summation order differs."""
    X = _pts(n, 2, 20 + n)
    W32, v0 = _oracle_on_fp32_W(orc, X, 0.7)
    Wd = torch.zeros((n, g.padded_ld(n)), dtype=torch.float32, device=DEV)
    Wd[:, :n] = _t(W32)
    v = _t(v0.copy())
    out = g.gpic_power_iterate_dense(Wd, v, None, "fixed", 25, n=n)
    ref = orc.power_iterate_dense(W32.astype(np.float64), v0, "fixed", 25)
    assert out.iterations == 25
    np.testing.assert_allclose(v.cpu().numpy(), ref.v, rtol=1e-11, atol=1e-300)
    np.testing.assert_allclose(out.stats, ref.stats, rtol=1e-6, atol=1e-15)
    # a single product
    y = g.gpic_matvec_dense(Wd, _t(v0), n=n)
    np.testing.assert_allclose(y.cpu().numpy(), W32.astype(np.float64) @ v0,
                               rtol=1e-12)


def test_power_iteration_uniform_fixed_point(g, orc):
    """Pin P3 on the GPU: v = 1/n stops after exactly 2 products."""
    n = 300
    X = _pts(n, 2, 31)
    A, deg = g.gpic_affinity(_t(X), 1.0)
    W, _, _, _ = g.gpic_degree_normalize(A, n, deg, True)
    v = torch.full((n,), 1.0 / n, dtype=torch.float64, device=DEV)
    out = g.gpic_power_iterate_dense(W, v, None, "converge", 100, 1e-9, n=n)
    assert out.converged and out.iterations == 2
    np.testing.assert_allclose(v.cpu().numpy(), 1.0 / n, rtol=1e-6)
    assert out.stats[0] == pytest.approx(1.0 / n, rel=1e-6)


def test_power_iteration_resume_and_determinism(g):
    n = 1500
    X = _pts(n, 2, 32)
    A, deg = g.gpic_affinity(_t(X), 0.5)
    W, _, v0, _ = g.gpic_degree_normalize(A, n, deg, True)
    a = v0.clone()
    da = v0.clone()
    r1 = g.gpic_power_iterate_dense(W, a, da, "fixed", 7, n=n)
    r2 = g.gpic_power_iterate_dense(W, a, da, "fixed", 5, n=n)
    b = v0.clone()
    db = v0.clone()
    r3 = g.gpic_power_iterate_dense(W, b, db, "fixed", 12, n=n)
    assert torch.equal(a, b) and torch.equal(da, db)                   # P11
    assert np.array_equal(np.concatenate([r1.stats, r2.stats]), r3.stats)
    c = v0.clone()
    r4 = g.gpic_power_iterate_dense(W, c, None, "fixed", 12, n=n)
    assert torch.equal(b, c) and np.array_equal(r3.stats, r4.stats)   # bitwise repeat


def test_power_iteration_zero_and_one_update(g):
    n = 100
    X = _pts(n, 2, 33)
    A, deg = g.gpic_affinity(_t(X), 1.0)
    W, _, v0, _ = g.gpic_degree_normalize(A, n, deg, True)
    v = v0.clone()
    out = g.gpic_power_iterate_dense(W, v, None, "fixed", 0, n=n)
    assert out.iterations == 0 and torch.equal(v, v0)
    Wn = W[:, :n].double().cpu().numpy()
    out = g.gpic_power_iterate_dense(W, v, None, "fixed", 1, n=n)
    y = Wn @ v0.cpu().numpy()
    np.testing.assert_allclose(v.cpu().numpy(), y / np.abs(y).sum(), rtol=1e-12)


def test_power_iteration_numeric_error(g):
    n = 8
    W = torch.zeros((n, 8), dtype=torch.float32, device=DEV)
    v = torch.full((n,), 1.0 / n, dtype=torch.float64, device=DEV)
    with pytest.raises(g.GpicError) as ei:
        g.gpic_power_iterate_dense(W, v, None, "fixed", 3, n=n)
    assert ei.value.status == 4


# ------------------------------------------------------ end-to-end (dense)
@pytest.mark.parametrize("name", ["blobs2d", "rings2d"])
def test_pic_dense_converge_parity(g, orc, name):
    import workloads
    w = workloads.make(name)
    print(f"pic_dense {name} n={w.n} eps={w.eps}", flush=True)
    out = g.pic_dense(_t(w.X), w.sigma, w.k, "converge", w.max_iter, w.eps)
    torch.cuda.synchronize()
    ref = orc.pic_dense(w.X, w.sigma, w.k, "converge", w.max_iter, w.eps)
    v = out.pi.v.cpu().numpy()
    mu = stop_margin(ref.pi.stats, w.eps, ref.pi.iterations)
    print(f"  iterations gpu={out.pi.iterations} oracle={ref.pi.iterations} "
          f"margin={mu:.3g} rel_l1={rel_l1(v, ref.pi.v):.3e}", flush=True)
    assert out.pi.converged and ref.pi.converged
    assert out.pi.iterations == ref.pi.iterations
    assert rel_l1(v, ref.pi.v) <= 1e-4
    np.testing.assert_allclose(out.pi.stats, ref.pi.stats, rtol=1e-3, atol=1e-3 * w.eps)
    assert out.km.k_eff == ref.km.k_eff == w.k
    check_labels(orc, f"dense {name}", ref.pi.v, ref.km.labels, v, out.km, w.k,
                 expect_separated=True)


@pytest.mark.parametrize("n", [3000, 4099])
def test_pic_dense_fixed_T_parity_16d(g, orc, n):
    """The 16-D blob shape (matrix-core Gram path) at reduced n, T = 50."""
    import workloads
    w = workloads.make("blobs16d", n=n)
    out = g.pic_dense(_t(w.X), w.sigma, w.k, "fixed", 50)
    torch.cuda.synchronize()
    ref = orc.pic_dense(w.X, w.sigma, w.k, "fixed", 50)
    v = out.pi.v.cpu().numpy()
    assert out.pi.iterations == 50
    assert rel_l1(v, ref.pi.v) <= 1e-4
    np.testing.assert_allclose(out.degree.cpu().numpy(), ref.A_degree, rtol=1e-5)
    # the statistic only matters against eps = 1e-5/n: agree to 1e-3 relative
    # or 1e-3 eps absolute (below that it is rounding noise of v)
    np.testing.assert_allclose(out.pi.stats, ref.pi.stats, rtol=1e-3, atol=1e-3 * w.eps)


@pytest.mark.parametrize("name", ["moons", "circles3"])
def test_pic_cosine_parity(g, orc, name):
    """The paper's Experiment I path at n = 3,000: cosine affinity, W, at
    most 3 updates with eps = 1e-5 / n, then k-means, against the oracle."""
    import workloads
    w = workloads.make(name, n=3000)
    out = g.pic_cosine(_t(w.X), w.k, "converge", w.max_iter, w.eps)
    A = orc.affinity_cosine(w.X)
    W, deg, v0, _ = orc.degree_normalize(A, copy=False)
    ref = orc.power_iterate_dense(W, v0, "converge", w.max_iter, w.eps)
    np.testing.assert_allclose(out.degree.cpu().numpy(), deg, rtol=1e-5)
    assert out.pi.iterations == ref.iterations and out.pi.converged == ref.converged
    vg = out.pi.v.cpu().numpy()
    assert rel_l1(vg, ref.v) <= 1e-4
    km = orc.kmeans1d(ref.v, w.k)
    check_labels(orc, f"cosine {name} n={w.n}", ref.v, km.labels, vg, out.km, w.k)


# ------------------------------------------------------------------ k-means
@pytest.mark.parametrize("n,k,dup", [(1, 1, False), (2, 2, False), (5, 3, False),
                                     (9, 9, False), (40, 39, False),
                                     (64, 8, False), (65, 8, False), (66, 8, True),
                                     (1000, 4, False), (4097, 10, False),
                                     (4097, 10, True), (4225, 20, True),
                                     (4291, 7, False), (50000, 10, False),
                                     (20000, 50, True), (274626, 30, False),
                                     (500000, 50, False), (262143, 20, False),
                                     (262144, 20, False), (531440, 30, False),
                                     (531441, 30, True), (300001, 200, True)])
def test_kmeans1d_parity(g, orc, n, k, dup):
    """Sizes straddle the recursion's level counts (F = 64 below 2^18 rows:
    n = 64 / 65, 4225 / 4291; F = 8 from 2^18 = 262,144: 9^6 = 531,441 adds
    a level), the switch between the two (262,143 / 262,144), fewer
    distinct values than k (300,001 values rounded to about 100 integers,
    k = 200), and k = n or n - 1 (the last layer's one row has a single
    split point, or two, with a finite cost)."""
    rng = np.random.default_rng(n + k)
    m = max(1, min(k, n))
    centres = np.sort(rng.uniform(0, 100, size=m))
    v = centres[rng.integers(0, m, size=n)] + rng.standard_normal(n) * 0.5
    if dup:
        v = np.round(v, 0)
    out = g.gpic_kmeans1d(_t(v), k)
    ref = orc.kmeans1d(v, k, "dc" if n > 2000 else "plain")
    check_kmeans(v, out, ref)


@pytest.mark.parametrize("n,k", [(30000, 50), (100000, 17)])
def test_kmeans1d_unclustered(g, orc, n, k):
    """Uniform values (no cluster structure): split points move smoothly."""
    v = np.random.default_rng(n).uniform(-1.0, 1.0, size=n)
    out = g.gpic_kmeans1d(_t(v), k)
    check_kmeans(v, out, orc.kmeans1d(v, k, "dc"))


def test_kmeans1d_special_values(g, orc):
    v = np.array([3.0, -0.0, 0.0, -2.5, 1e-300, -40.0, 7.0, 3.0])
    for k in (1, 3, 6, 8):
        out = g.gpic_kmeans1d(_t(v), k)
        ref = orc.kmeans1d(v, k, "plain")
        check_kmeans(v, out, ref)


# -------------------------------------------------------------- fused path
@pytest.mark.parametrize("n,d", [(300, 2), (1000, 64), (1025, 16), (500, 140)])
def test_fused_parity(g, orc, n, d):
    X = _pts(n, d, 40 + d, scale=1.5)
    sigma = np.float32(np.sqrt(d))
    deg, v0, nz = g.gpic_degree_fused(_t(X), sigma)
    v = v0.clone()
    out = g.gpic_power_iterate_fused(_t(X), sigma, deg, v, None, "fixed", 10)
    torch.cuda.synchronize()
    dr, v0r, _ = orc.degree_onthefly(X, sigma)
    ref = orc.power_iterate_onthefly(X, sigma, dr, v0r, "fixed", 10)
    np.testing.assert_allclose(deg.cpu().numpy(), dr, rtol=1e-5)
    assert rel_l1(v.cpu().numpy(), ref.v) <= 1e-4
    assert out.iterations == 10
    # the fused operator equals the dense one built from the same X
    A, degd = g.gpic_affinity(_t(X), sigma)
    W, _, v0d, _ = g.gpic_degree_normalize(A, n, degd, True)
    vd = v0d.clone()
    g.gpic_power_iterate_dense(W, vd, None, "fixed", 10, n=n)
    assert rel_l1(v.cpu().numpy(), vd.cpu().numpy()) <= 1e-6


@pytest.mark.parametrize("n,d", [(255, 16), (256, 20), (257, 64), (513, 100),
                                 (2050, 33), (4099, 16), (383, 16), (385, 64),
                                 (769, 33), (1025, 128)])
def test_fused_symmetric_edges(g, orc, n, d):
    """The fused operator evaluates each pair once (row groups of 384
    points up to 64 coordinates, 256 above: row sums for the group, column
    sums for later groups; 128- or 32-column tiles): sizes around the group,
    tile and chunk edges, every coordinate-chunk count (d = 16, 20, 33, 64,
    100, 128), one product against the oracle's on-the-fly rows."""
    X = _pts(n, d, 50 + d, scale=1.2)
    sigma = np.float32(np.sqrt(d))
    deg, v0, nz = g.gpic_degree_fused(_t(X), sigma)
    dr, v0r, _ = orc.degree_onthefly(X, sigma)
    np.testing.assert_allclose(deg.cpu().numpy(), dr, rtol=1e-5)
    v = np.random.default_rng(n + d).uniform(0.5, 1.5, size=n)
    y = g.gpic_matvec_fused(_t(X), sigma, deg, _t(v)).cpu().numpy()
    rows = np.arange(n, dtype=np.int64)
    yr = orc.matvec_onthefly_rows(X, sigma, dr, v, rows)
    np.testing.assert_allclose(y, yr, rtol=1e-5)


def test_fused_full_rows_above_symmetric_limit(g, orc):
    """Above 2^19 points the fused operator sums every ordered pair (row
    sweep for the degrees, row products): n = 2^19 + 1, sampled rows
    against the oracle, one by one."""
    n, d = (1 << 19) + 1, 16
    X = _pts(n, d, 77, scale=2.0)
    sigma = np.float32(4.0)
    print(f"gpu: fused full rows n={n} d={d}", flush=True)
    deg, v0, nz = g.gpic_degree_fused(_t(X), sigma)
    rows = np.array([0, 1, 255, 256, 511, 512, n // 3, n - 2, n - 1], dtype=np.int64)
    dr = orc.degree_rows(X, sigma, rows)
    np.testing.assert_allclose(deg.cpu().numpy()[rows], dr, rtol=1e-5)
    v = np.random.default_rng(5).uniform(0.5, 1.5, size=n)
    y = g.gpic_matvec_fused(_t(X), sigma, deg, _t(v)).cpu().numpy()
    dfull = np.zeros(n)
    dfull[rows] = dr
    yr = orc.matvec_onthefly_rows(X, sigma, dfull, v, rows)
    np.testing.assert_allclose(y[rows], yr, rtol=1e-5)


@pytest.mark.parametrize("n,d", [(700, 16), (3000, 64)])
def test_fused_rows_sum_to_one(g, n, d):
    """Pin P3 through the fused operator: its degrees are the row sums of
    the same symmetric A its products use, so W 1 = 1 up to float64
    rounding and v = 1/n stops after two products."""
    X = _pts(n, d, 60 + d)
    sigma = np.float32(np.sqrt(d))
    deg, _, _ = g.gpic_degree_fused(_t(X), sigma)
    ones = torch.ones(n, dtype=torch.float64, device=DEV)
    y = g.gpic_matvec_fused(_t(X), sigma, deg, ones).cpu().numpy()
    np.testing.assert_allclose(y, 1.0, rtol=1e-12)
    v = torch.full((n,), 1.0 / n, dtype=torch.float64, device=DEV)
    out = g.gpic_power_iterate_fused(_t(X), sigma, deg, v, None, "converge", 100, 1e-15)
    assert out.converged and out.iterations == 2
    np.testing.assert_allclose(v.cpu().numpy(), 1.0 / n, rtol=1e-12)


# ---------------------------------------------------------------- CSR path
def test_csr_parity_knn(g, orc):
    import workloads
    w = workloads.make("knn8d", n=4000)
    rp, col, val = w.row_ptr, w.col, w.val
    out = g.pic_csr(_t(rp), _t(col), _t(val.copy()), w.k, "converge", 1000, w.eps)
    torch.cuda.synchronize()
    wr, dr, v0r, _ = orc.degree_normalize_csr(rp, col, val)
    ref = orc.power_iterate_csr(rp, col, wr, v0r, "converge", 1000, w.eps)
    np.testing.assert_allclose(out.degree.cpu().numpy(), dr, rtol=1e-12)
    v = out.pi.v.cpu().numpy()
    assert out.pi.iterations == ref.iterations
    assert rel_l1(v, ref.v) <= 1e-4


def _random_graph(n, per_row, seed, sort_rows=True, band=None):
    """Symmetric random graph, float32 weights in [0.1, 1): neighbours
    anywhere (no locality in the numbering) or within +-band of the row;
    rows sorted by column unless asked otherwise."""
    import scipy.sparse as sp
    rng = np.random.default_rng(seed)
    i = np.repeat(np.arange(n), per_row)
    if band is None:
        j = rng.integers(0, n, size=n * per_row)
    else:
        j = np.clip(i + rng.integers(-band, band + 1, size=n * per_row), 0, n - 1)
    keep = i != j
    w = rng.uniform(0.1, 1.0, size=keep.sum())
    S = sp.coo_matrix((w, (i[keep], j[keep])), shape=(n, n)).tocsr()
    S = S.maximum(S.T).tocsr()
    S.sort_indices()
    rp, col, val = (S.indptr.astype(np.int64), S.indices.astype(np.int32),
                    S.data.astype(np.float32))
    if not sort_rows:
        col, val = col.copy(), val.copy()
        for r in range(0, n, max(1, n // 500)):       # reverse some rows
            a, b = rp[r], rp[r + 1]
            col[a:b], val[a:b] = col[a:b][::-1].copy(), val[a:b][::-1].copy()
    return rp, col, val


@pytest.mark.parametrize("sort_rows,band", [(True, None), (False, None), (True, 5000)])
def test_csr_column_blocked_parity(g, orc, sort_rows, band):
    """n = 600,000 spans three column blocks of 2^18: sorted rows with far
    neighbours take the column-blocked product; unsorted rows, or
    neighbours near the diagonal, the row-wise one.  Stage isolation: the
    oracle iterates on the GPU's float32 W, so v must agree to rounding
    after T = 20, and both must stop at the same update."""
    n = 600_000
    rp, col, val = _random_graph(n, 8, 77, sort_rows, band)
    print(f"gpu: random graph n={n} nnz={col.size} sorted={sort_rows} band={band}",
          flush=True)
    _, dr, v0r, _ = orc.degree_normalize_csr(rp, col, val)
    valg = _t(val.copy())
    _, deg, v0, _ = g.gpic_degree_normalize_csr(_t(rp), _t(col), valg)
    np.testing.assert_allclose(deg.cpu().numpy(), dr, rtol=1e-12)
    wg = valg.cpu().numpy().astype(np.float64)               # the GPU's W
    ref = orc.power_iterate_csr(rp, col, wg, v0r, "fixed", 20)
    v = v0.clone()
    out = g.gpic_power_iterate_csr(_t(rp), _t(col), valg, v, None, "fixed", 20)
    np.testing.assert_allclose(v.cpu().numpy(), ref.v, rtol=1e-9)
    np.testing.assert_allclose(out.stats, ref.stats, rtol=1e-6, atol=1e-18)
    eps = 0.5 * (ref.stats[5] + ref.stats[6])             # a stop between updates 6 and 7
    refc = orc.power_iterate_csr(rp, col, wg, v0r, "converge", 100, eps)
    v = v0.clone()
    outc = g.gpic_power_iterate_csr(_t(rp), _t(col), valg, v, None, "converge", 100, eps)
    assert outc.iterations == refc.iterations == 7
    np.testing.assert_allclose(v.cpu().numpy(), refc.v, rtol=1e-9)


@pytest.mark.parametrize("n,long_rows", [(3001, 0), (4100, 3), (700, 200)])
def test_csr_staged_product_edges(g, n, long_rows):
    """The staged CSR product (tiles of 256 rows, entries staged 2,048 per
    round): tile and round edges, empty rows, rows longer than a round
    (5,000 entries: a thread's sum carried across rounds), and a mean
    above 64 entries per row (the 16-lane row-wise product) when the long
    rows dominate: against the float64 product of the same float32 W."""
    import scipy.sparse as sp
    rng = np.random.default_rng(n + long_rows)
    lens = rng.integers(0, 40, size=n)
    lens[rng.choice(n, 5, replace=False)] = 0                 # empty rows
    lens[:long_rows] = 5000 if n > 5000 else n - 1
    rows = np.repeat(np.arange(n), lens)
    cols = np.concatenate([np.sort(rng.choice(n, size=m, replace=False)) for m in lens])
    W = sp.csr_matrix((rng.uniform(0.0, 1.0, size=rows.size).astype(np.float32),
                       (rows, cols)), shape=(n, n))
    W.sort_indices()
    rp, col, val = W.indptr.astype(np.int64), W.indices.astype(np.int32), W.data
    v = rng.uniform(0.5, 1.5, size=n)
    print(f"staged csr n={n} nnz={col.size} mean={col.size / n:.1f}", flush=True)
    y = g.gpic_matvec_csr(_t(rp), _t(col), _t(val), _t(v)).cpu().numpy()
    np.testing.assert_allclose(y, W.astype(np.float64) @ v, rtol=1e-12, atol=0)


def _relabel(rp, col, val, perm):
    """The graph with node p standing for node perm[p] of the input."""
    import scipy.sparse as sp
    n = rp.size - 1
    S = sp.csr_matrix((val, col, rp), shape=(n, n))
    P = S[perm][:, perm].tocsr()
    P.sort_indices()
    return P.indptr.astype(np.int64), P.indices.astype(np.int32), P.data


def test_knn_graph_local_numbering(g, orc):
    """The kNN graph numbered in the Morton order of the points is the
    oracle's brute-force graph relabelled by the returned permutation: the
    same rows, columns and weights (n = 60,000 of the kNN workload's
    generator, k = 32)."""
    import workloads
    w = workloads.make("knn8d", n=60000)
    print(f"knn graph local n={w.n}", flush=True)
    rp, col, val, perm = g.gpic_knn_graph_local(_t(w.X), 32, 1.0)
    torch.cuda.synchronize()
    perm = perm.cpu().numpy()
    assert np.array_equal(np.sort(perm), np.arange(w.n))
    rpo, colo, valo = _relabel(*orc.knn_graph(w.X, 32, 1.0), perm)
    assert np.array_equal(rp.cpu().numpy(), rpo)
    assert np.array_equal(col.cpu().numpy(), colo)
    vg = val.cpu().numpy()
    assert np.all(np.abs(vg - valo) <= np.spacing(valo))


def test_knn_csr_local_order_matches_original(g):
    """Power iteration over the Morton-numbered graph gives the original
    graph's v permuted (up to summation order), and stops at the same
    update."""
    import workloads
    w = workloads.make("knn8d", n=50000)
    X = _t(w.X)
    rp, col, val = g.gpic_knn_graph(X, 32, 1.0)
    rpl, coll, vall, perm = g.gpic_knn_graph_local(X, 32, 1.0)
    a = g.pic_csr(rp, col, val, w.k, "converge", 1000, w.eps)
    b = g.pic_csr(rpl, coll, vall, w.k, "converge", 1000, w.eps)
    assert a.pi.iterations == b.pi.iterations and a.pi.converged and b.pi.converged
    va = a.pi.v.cpu().numpy()
    vb = b.pi.v.cpu().numpy()
    np.testing.assert_allclose(vb, va[perm.cpu().numpy()], rtol=1e-10)


def _check_knn(g, orc, X, k, sigma):
    rp, col, val = g.gpic_knn_graph(_t(X), k, sigma)
    torch.cuda.synchronize()
    rpo, colo, valo = orc.knn_graph(X, k, sigma)
    assert np.array_equal(rp.cpu().numpy(), rpo)
    assert np.array_equal(col.cpu().numpy(), colo)
    vg = val.cpu().numpy()
    # float64 weights rounded once on both sides; exp differs by < 1 ulp
    # of float64, which can only flip a float32 rounding at a halfway point
    assert np.all(np.abs(vg - valo) <= np.spacing(valo))


@pytest.mark.parametrize("n,d,k,shift", [(3000, 8, 32, 0.0), (40, 3, 39, 0.0),
                                         (2000, 16, 10, 0.0), (2000, 8, 16, 1000.0),
                                         (5001, 2, 7, 0.0), (3000, 1, 5, 0.0),
                                         (1500, 4, 64, 0.0)])
def test_knn_graph_parity(g, orc, n, d, k, shift):
    """The exact kNN graph against the oracle's brute force: same rows,
    columns and weights (k = n - 1, d = 16, points far from the origin)."""
    rng = np.random.default_rng(n + d + k)
    C = 4.0 * rng.standard_normal((10, d))
    X = (C[rng.integers(0, 10, n)] + rng.standard_normal((n, d)) + shift).astype(np.float32)
    print(f"knn graph n={n} d={d} k={k} shift={shift}", flush=True)
    _check_knn(g, orc, X, k, 1.0)


def test_knn_graph_ties(g, orc):
    """Integer lattice (exact distance ties go to the smaller index)."""
    grid = np.arange(12, dtype=np.float32)
    X = np.stack(np.meshgrid(grid, grid), axis=-1).reshape(-1, 2)
    _check_knn(g, orc, X, 4, 1.0)
    X3 = np.random.default_rng(5).integers(0, 4, size=(3000, 3)).astype(np.float32)
    _check_knn(g, orc, X3, 10, 0.7)         # many duplicate points and ties


def test_csr_full_pattern_equals_dense(g):
    n = 300
    X = _pts(n, 2, 50)
    A, deg = g.gpic_affinity(_t(X), 1.0)
    An = A[:, :n].contiguous()
    rp = torch.arange(0, n * n + 1, n, dtype=torch.int64, device=DEV)
    col = torch.arange(n, dtype=torch.int32, device=DEV).repeat(n)
    val = An.reshape(-1).clone()
    _, dcsr, v0c, _ = g.gpic_degree_normalize_csr(rp, col, val)
    W, ddense, v0d, _ = g.gpic_degree_normalize(A, n, deg, True)
    np.testing.assert_allclose(dcsr.cpu().numpy(), ddense.cpu().numpy(), rtol=1e-13)
    vc, vd = v0c.clone(), v0d.clone()
    g.gpic_power_iterate_csr(rp, col, val, vc, None, "fixed", 20)
    g.gpic_power_iterate_dense(W, vd, None, "fixed", 20, n=n)
    np.testing.assert_allclose(vc.cpu().numpy(), vd.cpu().numpy(), rtol=1e-10)


def test_csr_invalid_structure_rejected(g):
    n = 4
    rp = torch.tensor([0, 2, 1, 3, 4], dtype=torch.int64, device=DEV)   # not monotone
    col = torch.tensor([1, 2, 0, 3], dtype=torch.int32, device=DEV)
    val = torch.ones(4, dtype=torch.float32, device=DEV)
    with pytest.raises(g.GpicError) as ei:
        g.gpic_degree_normalize_csr(rp, col, val)
    assert ei.value.status == 1
    rp = torch.tensor([0, 1, 2, 3, 4], dtype=torch.int64, device=DEV)
    col = torch.tensor([1, 2, 0, 9], dtype=torch.int32, device=DEV)      # column >= n
    with pytest.raises(g.GpicError):
        g.gpic_degree_normalize_csr(rp, col, val)


# ------------------------------------- symmetric storage (packed upper tiles)
def _unpack_sym(As, n):
    """Dense float64 n x n matrix from the packed upper tiles (tile (I, J),
    I <= J, of 256 x 256, row-major; lower tiles mirrored)."""
    a = As.cpu().numpy()
    nb = (n + 255) // 256
    full = np.zeros((nb * 256, nb * 256))
    t = 0
    for I in range(nb):
        for J in range(I, nb):
            with np.errstate(invalid="ignore"):      # padding past n is never written
                blk = a[t * 65536:(t + 1) * 65536].reshape(256, 256).astype(np.float64)
            full[256 * I:256 * I + 256, 256 * J:256 * J + 256] = blk
            if I != J:
                full[256 * J:256 * J + 256, 256 * I:256 * I + 256] = blk.T
            t += 1
    return full[:n, :n]


def _upper_mask(n):
    b = np.arange(n) // 256
    return b[:, None] <= b[None, :]


@pytest.mark.parametrize("n,d", [(2, 2), (255, 3), (256, 2), (300, 16), (513, 64),
                                 (777, 17), (1000, 2), (130, 140)])
def test_sym_affinity_equals_dense(g, n, d):
    """Stored entries are bitwise the dense affinity's (same engine and
    operands); degrees are the row sums of the stored symmetric A, which
    differ from the dense row sums only where float32 A_ij and A_ji differ."""
    X = _pts(n, d, 4000 + n + d, scale=1.4)
    sigma = np.float32(np.sqrt(d))
    As, deg, v0, nz = g.gpic_affinity_sym(_t(X), sigma)
    A, degA = g.gpic_affinity(_t(X), sigma)
    W1, deg1, v01, _ = g.gpic_affinity_normalized(_t(X), sigma)
    torch.cuda.synchronize()
    assert As.numel() * 4 == g.sym_bytes(n)
    full = _unpack_sym(As, n)
    Ad = A[:, :n].cpu().numpy().astype(np.float64)
    up = _upper_mask(n)
    assert np.array_equal(full[up], Ad[up])
    assert np.all(np.diag(full) == 0.0)
    assert torch.equal(deg1, degA)
    dg = deg.cpu().numpy()
    np.testing.assert_allclose(dg, full.sum(axis=1), rtol=1e-12)
    np.testing.assert_allclose(dg, deg1.cpu().numpy(), rtol=1e-5)
    np.testing.assert_allclose(v0.cpu().numpy(), dg / dg.sum(), rtol=1e-12)
    np.testing.assert_allclose(v0.cpu().numpy(), v01.cpu().numpy(), rtol=1e-5)
    assert int(nz.item()) == 0


@pytest.mark.parametrize("n", [2, 255, 256, 257, 511, 512, 513, 700, 768, 769, 1025, 1281,
                               2050])
def test_sym_matvec_stage_isolation(g, n):
    """y = D^-1 (A v) from the stored float32 tiles: only summation order
    differs from a float64 product with the unpacked matrix.  Sizes cover
    one block, a ragged last block, and an even and odd number of 256-row
    blocks (the product takes 2 x 2 super-tiles; with an odd count the last
    super-row holds one block).  The storage is filled with NaN before the
    affinity writes it, so padding entries outside [0, n)^2 hold NaN and
    must never reach a sum."""
    X = _pts(n, 3, 60 + n)
    As0 = torch.full((g.sym_bytes(n) // 4,), float("nan"), dtype=torch.float32,
                     device=torch.device("cuda:0"))
    As, deg, v0, _ = g.gpic_affinity_sym(_t(X), 0.9, As=As0)
    rng = np.random.default_rng(n)
    v = rng.random(n)
    y = g.gpic_matvec_sym(As, n, deg, _t(v)).cpu().numpy()
    full = _unpack_sym(As, n)
    ref = (full @ v) / deg.cpu().numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12)
    y2 = g.gpic_matvec_sym(As, n, deg, _t(v)).cpu().numpy()
    assert np.array_equal(y, y2)


@pytest.mark.parametrize("name", ["blobs2d", "rings2d"])
def test_pic_sym_converge_parity(g, orc, name):
    import workloads
    w = workloads.make(name)
    out = g.pic_sym(_t(w.X), w.sigma, w.k, "converge", w.max_iter, w.eps)
    torch.cuda.synchronize()
    ref = orc.pic_dense(w.X, w.sigma, w.k, "converge", w.max_iter, w.eps)
    v = out.pi.v.cpu().numpy()
    mu = stop_margin(ref.pi.stats, w.eps, ref.pi.iterations)
    print(f"  sym {name}: iterations gpu={out.pi.iterations} oracle={ref.pi.iterations} "
          f"margin={mu:.3g} rel_l1={rel_l1(v, ref.pi.v):.3e}", flush=True)
    assert out.pi.converged and ref.pi.converged
    assert out.pi.iterations == ref.pi.iterations
    assert rel_l1(v, ref.pi.v) <= 1e-4
    np.testing.assert_allclose(out.pi.stats, ref.pi.stats, rtol=1e-3, atol=1e-3 * w.eps)
    assert out.km.k_eff == ref.km.k_eff == w.k
    check_labels(orc, f"sym {name}", ref.pi.v, ref.km.labels, v, out.km, w.k,
                 expect_separated=True)


@pytest.mark.parametrize("n", [3000, 4099])
def test_pic_sym_fixed_T_parity_16d(g, orc, n):
    import workloads
    w = workloads.make("blobs16d", n=n)
    out = g.pic_sym(_t(w.X), w.sigma, w.k, "fixed", 50)
    ref = orc.pic_dense(w.X, w.sigma, w.k, "fixed", 50)
    v = out.pi.v.cpu().numpy()
    assert out.pi.iterations == 50
    assert rel_l1(v, ref.pi.v) <= 1e-4
    np.testing.assert_allclose(out.degree.cpu().numpy(), ref.A_degree, rtol=1e-5)
    np.testing.assert_allclose(out.pi.stats, ref.pi.stats, rtol=1e-3, atol=1e-3 * w.eps)
    # resume: 20 + 30 updates equal 50, bitwise
    As, deg, v0, _ = g.gpic_affinity_sym(_t(w.X), w.sigma)
    a, da = v0.clone(), v0.clone()
    g.gpic_power_iterate_sym(As, n, deg, a, da, "fixed", 20)
    g.gpic_power_iterate_sym(As, n, deg, a, da, "fixed", 30)
    assert torch.equal(a, out.pi.v)


@pytest.mark.parametrize("n,d", [(600, 2), (1000, 16)])
def test_sym_uniform_fixed_point(g, n, d):
    """Pin P3 through the symmetric operator: its degrees are the row sums of
    the stored symmetric A, so W 1 = 1 up to float64 rounding and v = 1/n
    stops after 2 products."""
    X = _pts(n, d, 34)
    sigma = np.float32(np.sqrt(d))
    As, deg, _, _ = g.gpic_affinity_sym(_t(X), sigma)
    ones = torch.ones(n, dtype=torch.float64, device=DEV)
    y = g.gpic_matvec_sym(As, n, deg, ones).cpu().numpy()
    np.testing.assert_allclose(y, 1.0, rtol=1e-12)
    v = torch.full((n,), 1.0 / n, dtype=torch.float64, device=DEV)
    out = g.gpic_power_iterate_sym(As, n, deg, v, None, "converge", 100, 1e-15)
    assert out.converged and out.iterations == 2
    np.testing.assert_allclose(v.cpu().numpy(), 1.0 / n, rtol=1e-12)


# --------------------------------------------- out-of-core dense (host W)
def _host_copy(W, n):
    Wh = torch.empty((n, W.shape[1]), dtype=torch.float32, pin_memory=True)
    Wh.copy_(W[:n].cpu())
    return Wh


@pytest.mark.parametrize("n,rows", [(1003, 12), (2048, None), (2049, 16), (3000, 64),
                                    (4099, None)])
def test_dense_host_equals_device(g, n, rows):
    """W streamed from pinned host memory in row panels gives bitwise the
    device-resident path's v, statistics and stop update.  Up to n = 2,048
    the device path runs one launch per update (the previous iteration's tau
    and update fused with the next product), the host path two: the same
    values either way."""
    import workloads
    w = workloads.make("blobs16d", n=n)
    W, deg, v0, _ = g.gpic_affinity_normalized(_t(w.X), w.sigma)
    torch.cuda.synchronize()
    Wh = _host_copy(W, n)
    ws_bytes = None
    if rows is not None:
        pitch = (n + 3) // 4 * 4
        panel = (rows * pitch * 4 + 255) // 256 * 256
        ws_bytes = g.workspace_bytes("pi_dense", n) + 2 * panel
    a = v0.clone()
    ra = g.gpic_power_iterate_dense(W, a, None, "fixed", 20, n=n)
    b = v0.clone()
    rb = g.gpic_power_iterate_dense_host(Wh, b, None, "fixed", 20, ws_bytes=ws_bytes)
    assert rb.iterations == 20 and torch.equal(a, b)
    assert np.array_equal(ra.stats, rb.stats)
    eps = 1e-5 / n
    a = v0.clone()
    ra = g.gpic_power_iterate_dense(W, a, None, "converge", 1000, eps, n=n)
    b = v0.clone()
    rb = g.gpic_power_iterate_dense_host(Wh, b, None, "converge", 1000, eps,
                                         ws_bytes=ws_bytes)
    assert ra.converged and rb.converged and ra.iterations == rb.iterations
    assert torch.equal(a, b)


@pytest.mark.parametrize("mode", ["fixed", "converge"])
def test_dense_host_oracle_parity(g, orc, mode):
    """The out-of-core path against the oracle, n = 3,000 (16-D blobs):
    (1) the whole path, W built on the GPU and streamed from pinned host
    memory in row panels, against the oracle's float64 chain: v within
    relative L1 1e-4 and the identical stop update; (2) stage isolation:
    the oracle's W rounded to float32 streamed the same way, against the
    oracle's iteration over that same float32 W, to 1e-11."""
    import workloads
    n = 3000
    w = workloads.make("blobs16d", n=n)
    eps = 1e-5 / n
    T = 20 if mode == "fixed" else 1000
    pitch = (n + 3) // 4 * 4
    panel = (256 * pitch * 4 + 255) // 256 * 256            # 256-row panels
    ws_bytes = g.workspace_bytes("pi_dense", n) + 2 * panel
    print(f"dense_host oracle parity n={n} mode={mode}", flush=True)
    W, deg, v0, _ = g.gpic_affinity_normalized(_t(w.X), w.sigma)
    torch.cuda.synchronize()
    Wh = _host_copy(W, n)
    del W
    v = v0.clone()
    r = g.gpic_power_iterate_dense_host(Wh, v, None, mode, T, eps, ws_bytes=ws_bytes)
    Wr, dr, v0r, _ = orc.degree_normalize(orc.affinity(w.X, w.sigma), copy=False)
    ref = orc.power_iterate_dense(Wr, v0r, mode, T, eps)
    print(f"  iterations gpu={r.iterations} oracle={ref.iterations} "
          f"rel_l1={rel_l1(v.cpu().numpy(), ref.v):.3e}", flush=True)
    assert r.iterations == ref.iterations and r.converged == ref.converged
    assert rel_l1(v.cpu().numpy(), ref.v) <= 1e-4
    np.testing.assert_allclose(r.stats, ref.stats, rtol=1e-3, atol=1e-3 * eps)
    # stage isolation over the oracle's own W in float32
    W32 = Wr.astype(np.float32)
    ref32 = orc.power_iterate_dense(W32.astype(np.float64), v0r, mode, T, eps)
    Wh32 = torch.empty((n, n), dtype=torch.float32, pin_memory=True)
    Wh32.copy_(torch.from_numpy(W32))
    v = _t(v0r)
    r = g.gpic_power_iterate_dense_host(Wh32, v, None, mode, T, eps, ws_bytes=ws_bytes)
    assert r.iterations == ref32.iterations and r.converged == ref32.converged
    np.testing.assert_allclose(v.cpu().numpy(), ref32.v, rtol=1e-11)


def test_dense_host_pageable_memory(g):
    """W in ordinary (pageable) host memory: slower copies, same bits."""
    import workloads
    n = 1500
    w = workloads.make("rings2d", n=n)
    W, deg, v0, _ = g.gpic_affinity_normalized(_t(w.X), w.sigma)
    torch.cuda.synchronize()
    Wh = W[:n].cpu().contiguous()
    assert not Wh.is_pinned()
    a = v0.clone()
    g.gpic_power_iterate_dense(W, a, None, "fixed", 9, n=n)
    b = v0.clone()
    g.gpic_power_iterate_dense_host(Wh, b, None, "fixed", 9,
                                    ws_bytes=g.workspace_bytes("pi_dense", n) + 2 * 256 * 1024)
    assert torch.equal(a, b)


def test_dense_host_workspace_too_small(g):
    n = 100
    Wh = torch.zeros((n, n), dtype=torch.float32, pin_memory=True)
    v = torch.full((n,), 1.0 / n, dtype=torch.float64, device=DEV)
    with pytest.raises(g.GpicError) as ei:
        g.gpic_power_iterate_dense_host(Wh, v, None, "fixed", 1,
                                        ws_bytes=g.workspace_bytes("pi_dense", n) + 256)
    assert ei.value.status == 2


@pytest.mark.parametrize("n", [4, 4 * 1536 * 256 * 3 + 12])
def test_read_stream_reads_every_float(g, n):
    """The bandwidth reference reads each float once: the sink's sums add up
    to the buffer's sum (ones, so every partial sum is exact)."""
    x = torch.ones(n + 8, dtype=torch.float32, device=DEV)
    x[n:] = 1e6                                   # past n: never read
    sink = g.gpic_read_stream(x, n)
    assert sink.numel() == g.READ_STREAM_SINK
    assert float(sink.sum().item()) == float(n)


@pytest.mark.parametrize("n", [2047, 3001, 4103, 6150])
def test_dense_matvec_prefetch_edges(g, n):
    """Column-group counts around one, two and three passes of the 512
    threads (n/4 = 511, 750, 1025, 1537) with ragged tails: the loads issued
    two groups ahead stay in the row and every entry is used once."""
    rng = np.random.default_rng(n)
    W32 = rng.random((n, n), dtype=np.float32)
    Wd = torch.full((n, g.padded_ld(n)), float("nan"), dtype=torch.float32, device=DEV)
    Wd[:, :n] = _t(W32)                       # padding past n must never be read
    v = rng.random(n)
    y = g.gpic_matvec_dense(Wd, _t(v), n=n).cpu().numpy()
    np.testing.assert_allclose(y, W32.astype(np.float64) @ v, rtol=1e-12)
