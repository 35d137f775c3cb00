"""Pins of the oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formulas: each compares it with a
library routine, a closed form, an invariant of the method, a hand-worked
trace (tests/golden) or exhaustive search.
"""
import itertools
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _pts(n, d, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return (scale * rng.standard_normal((n, d))).astype(np.float32)


# ----------------------------------------------------------------- affinity
def test_affinity_matches_scipy_distance(orc):
    """Gaussian affinity equals exp(-cdist^2 / (2 sigma^2)) off the diagonal."""
    X = _pts(57, 5, 1)
    sigma = np.float32(1.7)
    A = orc.affinity(X, sigma)
    D2 = cdist(X.astype(np.float64), X.astype(np.float64), "sqeuclidean")
    ref = np.exp(-D2 / (2.0 * float(sigma) ** 2))
    np.fill_diagonal(ref, 0.0)
    np.testing.assert_allclose(A, ref, rtol=1e-12, atol=0)
    assert np.all(np.diag(A) == 0.0)


def test_affinity_closed_form_two_points(orc):
    X = np.array([[0, 0], [3, 4]], dtype=np.float32)
    A = orc.affinity(X, 2.0)
    assert A[0, 1] == pytest.approx(np.exp(-25.0 / 8.0), rel=1e-15)
    assert A[0, 0] == 0.0 and A[1, 1] == 0.0


def test_affinity_symmetric_and_invariant(orc):
    """A = A^T exactly; integer translations and a quarter turn (all exact in
    float32) leave A unchanged."""
    rng = np.random.default_rng(7)
    X = rng.integers(-20, 20, size=(40, 2)).astype(np.float32)
    A = orc.affinity(X, 3.0)
    assert np.array_equal(A, A.T)
    At = orc.affinity(X + np.float32(5.0), 3.0)
    Xr = np.stack([-X[:, 1], X[:, 0]], axis=1)
    Ar = orc.affinity(Xr, 3.0)
    np.testing.assert_allclose(At, A, rtol=1e-15)
    np.testing.assert_allclose(Ar, A, rtol=1e-15)


def test_affinity_rows_and_degree_rows_agree(orc):
    X = _pts(33, 3, 2)
    A = orc.affinity(X, 1.1)
    rows = [0, 5, 32]
    np.testing.assert_array_equal(orc.affinity_rows(X, 1.1, rows), A[rows])
    np.testing.assert_allclose(orc.degree_rows(X, 1.1, rows), A[rows].sum(1),
                               rtol=1e-14)


def test_cosine_affinity_matches_scipy_distance(orc):
    """Cosine affinity (1 + cos) / 2 equals 1 - cdist_cosine / 2 off the
    diagonal (scipy's cosine distance is 1 - cos)."""
    X = _pts(61, 5, 11)
    A = orc.affinity_cosine(X)
    ref = 1.0 - 0.5 * cdist(X.astype(np.float64), X.astype(np.float64), "cosine")
    np.fill_diagonal(ref, 0.0)
    np.testing.assert_allclose(A, ref, rtol=1e-12, atol=1e-15)
    assert np.all(np.diag(A) == 0.0) and A.min() >= 0.0


def test_cosine_affinity_closed_form_and_invariance(orc):
    """Points on rays at angles t: a = (1 + cos(t_i - t_j)) / 2; scaling
    points by powers of two and a quarter turn (exact in float32) leave A
    unchanged; the origin gets 1/2 against every point."""
    t = np.array([0.0, 0.5, 1.9, 3.0, 4.4])
    r = np.array([1.0, 2.0, 0.25, 8.0, 3.0])
    X = np.stack([r * np.cos(t), r * np.sin(t)], axis=1).astype(np.float32)
    A = orc.affinity_cosine(X)
    tt = np.arctan2(X[:, 1].astype(np.float64), X[:, 0].astype(np.float64))
    ref = 0.5 * (1.0 + np.cos(tt[:, None] - tt[None, :]))
    np.fill_diagonal(ref, 0.0)
    np.testing.assert_allclose(A, ref, rtol=1e-13, atol=1e-15)
    scale = np.array([1, 4, 0.5, 2, 0.125], dtype=np.float32)[:, None]
    np.testing.assert_array_equal(orc.affinity_cosine(X * scale), A)
    Xr = np.stack([-X[:, 1], X[:, 0]], axis=1)
    np.testing.assert_allclose(orc.affinity_cosine(Xr), A, rtol=1e-15, atol=1e-16)
    Z = np.vstack([X, np.zeros((1, 2), np.float32)])
    Az = orc.affinity_cosine(Z)
    assert np.all(Az[-1, :-1] == 0.5) and np.all(Az[:-1, -1] == 0.5) and Az[-1, -1] == 0.0
    assert np.array_equal(orc.affinity_cosine_rows(X, [1, 3]), A[[1, 3]])


# ------------------------------------------------------ degree / normalise
def test_rows_of_W_sum_to_one_and_v0(orc):
    """P1, P2: W = D^-1 A has unit row sums; v0 = d / sum d has L1 norm 1."""
    X = _pts(200, 3, 3)
    A = orc.affinity(X, 0.8)
    W, deg, v0, nz = orc.degree_normalize(A)
    assert nz == 0
    np.testing.assert_allclose(W.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(deg, A.sum(axis=1), rtol=1e-14)
    np.testing.assert_allclose(v0, deg / deg.sum(), rtol=1e-15)
    assert abs(v0.sum() - 1.0) < 1e-14
    # W is row- (not column-) normalised: W = diag(1/d) A
    np.testing.assert_allclose(W, A / deg[:, None], rtol=1e-15)


def test_zero_degree_row_is_counted(orc):
    X = np.array([[0, 0], [0.1, 0], [1000, 1000]], dtype=np.float32)
    A = orc.affinity(X, 0.05)
    W, deg, v0, nz = orc.degree_normalize(A)
    assert nz == 1 and deg[2] == 0.0 and v0[2] == 0.0
    assert np.all(W[2] == 0.0)
    with pytest.raises(FloatingPointError):
        orc.degree_normalize(np.zeros((3, 3)))


def test_two_points_give_swap_matrix(orc):
    """P8: n = 2 gives W = [[0,1],[1,0]] and v0 = (1/2, 1/2) for any weight."""
    for dist in (0.1, 1.0, 3.0):
        X = np.array([[0, 0], [dist, 0]], dtype=np.float32)
        W, deg, v0, _ = orc.degree_normalize(orc.affinity(X, 1.0))
        assert np.array_equal(W, np.array([[0.0, 1.0], [1.0, 0.0]]))
        assert np.array_equal(v0, np.array([0.5, 0.5]))


# -------------------------------------------------------- power iteration
@pytest.mark.parametrize("name", ["two_node_trace", "three_node_path_trace"])
def test_hand_worked_traces(orc, name):
    g = json.load(open(os.path.join(GOLDEN, name + ".json")))
    if "A" in g:
        W, deg, v0, _ = orc.degree_normalize(np.array(g["A"], dtype=np.float64))
        np.testing.assert_allclose(deg, g["degree"], rtol=1e-15)
        np.testing.assert_allclose(v0, g["v0"], rtol=1e-15)
        np.testing.assert_allclose(W, g["W"], rtol=1e-15)
    else:
        W, _, _, _ = orc.degree_normalize(orc.affinity(np.array(g["X"], np.float32),
                                                       g["sigma"]))
        v0 = np.array(g["v0"])
    r = orc.power_iterate_dense(W, v0, "converge", 100, g["eps"])
    assert r.converged and r.iterations == g["converge"]["iterations"]
    np.testing.assert_allclose(r.v, g["converge"]["v"], rtol=1e-14)
    np.testing.assert_allclose(r.stats, g["converge"]["stats"], rtol=1e-13, atol=1e-15)
    r = orc.power_iterate_dense(W, v0, "fixed", 3)
    assert r.iterations == 3 and not r.converged
    np.testing.assert_allclose(r.v, g["fixed_T3"]["v"], rtol=1e-14)
    np.testing.assert_allclose(r.stats, g["fixed_T3"]["stats"], rtol=1e-13, atol=1e-15)


def test_uniform_vector_is_fixed_point(orc):
    """P3: W 1 = 1, so v = 1/n is fixed; with delta_0 = v_0 the statistic is
    1/n then 0, and the run stops after exactly 2 products."""
    X = _pts(150, 4, 4)
    W, _, _, _ = orc.degree_normalize(orc.affinity(X, 1.3))
    n = 150
    u = np.full(n, 1.0 / n)
    r = orc.power_iterate_dense(W, u, "converge", 50, 1e-9)
    assert r.converged and r.iterations == 2
    np.testing.assert_allclose(r.v, u, rtol=1e-13)
    assert r.stats[0] == pytest.approx(1.0 / n, rel=1e-12)
    assert r.stats[1] < 1e-15

def test_stop_test_is_less_or_equal(orc):
    """The stop test is "<=" (Algorithms 1 and 2).  Two points with
    v0 = (1/2, 1/2) are exact in floating point: the statistic is 1/2, then
    exactly 0, so even eps = 0 stops the run after 2 products."""
    X = np.array([[0, 0], [1, 0]], dtype=np.float32)
    W, _, v0, _ = orc.degree_normalize(orc.affinity(X, 1.0))
    r = orc.power_iterate_dense(W, v0, "converge", 50, 0.0)
    assert r.converged and r.iterations == 2
    assert list(r.stats) == [0.5, 0.0]


def _block_diag_constant(sizes, consts):
    n = sum(sizes)
    A = np.zeros((n, n))
    o = 0
    for m, c in zip(sizes, consts):
        A[o:o + m, o:o + m] = c
        o += m
    np.fill_diagonal(A, 0.0)
    return A


def test_constant_blocks_are_fixed_points(orc):
    """P4: a block-diagonal A with constant blocks gives a piecewise-constant
    v0 that is a fixed point; the run stops after exactly 2 products."""
    sizes, consts = [5, 9, 3], [0.5, 0.25, 2.0]
    A = _block_diag_constant(sizes, consts)
    W, deg, v0, _ = orc.degree_normalize(A)
    o = 0
    for m, c in zip(sizes, consts):
        assert np.allclose(v0[o:o + m], v0[o], rtol=0, atol=0)
        assert v0[o] == pytest.approx(c * (m - 1) / deg.sum(), rel=1e-15)
        o += m
    r = orc.power_iterate_dense(W, v0, "converge", 50, 1e-12)
    assert r.converged and r.iterations == 2
    np.testing.assert_allclose(r.v, v0, rtol=1e-14)


def test_block_diagonal_components_never_mix(orc):
    """P5: components never mix, and v tends to a constant per component,
    proportional to sum_b d_i^2 / sum_b d_i (the left Perron vector of
    W = D^-1 A is d because A is symmetric)."""
    X1 = _pts(30, 2, 5)
    X2 = _pts(20, 2, 6) + np.float32(1000.0)
    X = np.concatenate([X1, X2])
    A = orc.affinity(X, 1.0)
    assert A[:30, 30:].max() == 0.0
    W, deg, v0, _ = orc.degree_normalize(A)
    e = np.zeros(50)
    e[:30] = v0[:30] / v0[:30].sum()
    r = orc.power_iterate_dense(W, e, "fixed", 40)
    assert np.all(r.v[30:] == 0.0)
    r = orc.power_iterate_dense(W, v0, "fixed", 3000)
    lim = np.empty(50)
    for b in (slice(0, 30), slice(30, 50)):
        lim[b] = (deg[b] ** 2).sum() / deg[b].sum()
    lim /= lim.sum()
    np.testing.assert_allclose(r.v, lim, rtol=1e-10)


def test_closed_form_eigendecomposition(orc):
    """P6: W^t = D^-1/2 S^t D^1/2 with S = D^-1/2 A D^-1/2 = U diag(l) U^T;
    every update only rescales, so v_T = W^T v0 / ||W^T v0||_1.  A transposed
    W (column normalisation) or a dropped normalisation fails this."""
    X = _pts(300, 3, 8)
    A = orc.affinity(X, 0.9)
    W, deg, v0, _ = orc.degree_normalize(A)
    s = np.sqrt(deg)
    S = A / s[:, None] / s[None, :]
    lam, U = np.linalg.eigh(S)
    for T in (1, 4, 9):
        z = (U * lam ** T) @ (U.T @ (s * v0)) / s
        z /= np.abs(z).sum()
        r = orc.power_iterate_dense(W, v0, "fixed", T)
        np.testing.assert_allclose(r.v, z, rtol=1e-11)
        assert np.all(r.v >= 0) and abs(r.v.sum() - 1) < 1e-14


def test_single_update_and_zero_updates(orc):
    """P12: T = 0 returns v0; T = 1 returns (W v0) / ||W v0||_1 (numpy matmul)."""
    X = _pts(80, 2, 9)
    W, _, v0, _ = orc.degree_normalize(orc.affinity(X, 0.7))
    r0 = orc.power_iterate_dense(W, v0, "fixed", 0)
    assert r0.iterations == 0 and np.array_equal(r0.v, v0)
    r1 = orc.power_iterate_dense(W, v0, "fixed", 1)
    y = W @ v0
    np.testing.assert_allclose(r1.v, y / np.abs(y).sum(), rtol=1e-14)
    np.testing.assert_allclose(r1.delta, np.abs(y / np.abs(y).sum() - v0),
                               rtol=1e-10, atol=1e-18)


def test_resume_equals_uninterrupted(orc):
    """P11: T1 updates, then T2 more from (v, delta), equals T1 + T2."""
    X = _pts(120, 3, 10)
    W, _, v0, _ = orc.degree_normalize(orc.affinity(X, 1.0))
    a = orc.power_iterate_dense(W, v0, "fixed", 7)
    b = orc.power_iterate_dense(W, a.v, "fixed", 5, delta=a.delta)
    c = orc.power_iterate_dense(W, v0, "fixed", 12)
    assert np.array_equal(b.v, c.v) and np.array_equal(b.delta, c.delta)
    assert np.array_equal(np.concatenate([a.stats, b.stats]), c.stats)


def test_permutation_equivariance(orc):
    """P9: permuting the points permutes v."""
    X = _pts(90, 2, 11)
    p = np.random.default_rng(0).permutation(90)
    r = orc.pic_dense(X, 0.6, 3, "fixed", 10)
    rp = orc.pic_dense(X[p], 0.6, 3, "fixed", 10)
    np.testing.assert_allclose(rp.pi.v, r.pi.v[p], rtol=1e-12)


def test_csr_full_pattern_equals_dense(orc):
    """P13: the CSR path over the full pattern reproduces the dense path."""
    X = _pts(70, 2, 12)
    A = orc.affinity(X, 0.9)
    n = 70
    row_ptr = np.arange(0, n * n + 1, n, dtype=np.int64)
    col = np.tile(np.arange(n, dtype=np.int32), n)
    w, deg, v0, _ = orc.degree_normalize_csr(row_ptr, col, A.ravel())
    W, deg2, v02, _ = orc.degree_normalize(A)
    assert np.array_equal(deg, deg2) and np.array_equal(w, W.ravel())
    rc = orc.power_iterate_csr(row_ptr, col, w, v0, "converge", 500, 1e-5 / n)
    rd = orc.power_iterate_dense(W, v0, "converge", 500, 1e-5 / n)
    assert rc.iterations == rd.iterations and np.array_equal(rc.v, rd.v)


def test_csr_sparse_matches_scipy(orc):
    """One CSR update against scipy.sparse's product."""
    import scipy.sparse as sp
    rng = np.random.default_rng(13)
    M = sp.random(200, 200, density=0.05, random_state=13, format="csr")
    M = M + M.T + sp.eye(200) * 0.0
    M = M.tocsr()
    M.sort_indices()
    w, deg, v0, nz = orc.degree_normalize_csr(M.indptr, M.indices, M.data)
    Wd = sp.diags(np.where(deg > 0, 1.0 / np.where(deg > 0, deg, 1), 0.0)) @ M
    r = orc.power_iterate_csr(M.indptr, M.indices, w, v0, "fixed", 1)
    y = Wd @ v0
    np.testing.assert_allclose(r.v, y / np.abs(y).sum(), rtol=1e-13)
    assert nz == int((np.asarray(M.sum(axis=1)).ravel() == 0).sum())
    del rng


def test_onthefly_equals_dense(orc):
    """P14: recomputing A every sweep gives the dense result."""
    X = _pts(60, 3, 14)
    sigma = 1.2
    A = orc.affinity(X, sigma)
    W, deg, v0, _ = orc.degree_normalize(A)
    deg2, v02, _ = orc.degree_onthefly(X, sigma)
    assert np.array_equal(deg, deg2) and np.array_equal(v0, v02)
    rf = orc.power_iterate_onthefly(X, sigma, deg2, v02, "fixed", 8)
    rd = orc.power_iterate_dense(W, v0, "fixed", 8)
    assert np.array_equal(rf.v, rd.v) and np.array_equal(rf.stats, rd.stats)
    rows = np.array([0, 17, 59])
    y = orc.matvec_onthefly_rows(X, sigma, deg2, rd.v, rows)
    np.testing.assert_allclose(y, (W @ rd.v)[rows], rtol=1e-14)


def test_numeric_error_on_zero_product(orc):
    W = np.zeros((3, 3))
    with pytest.raises(FloatingPointError):
        orc.power_iterate_dense(W, np.full(3, 1 / 3), "fixed", 2)


def test_fixed_mode_never_stops_early(orc):
    X = _pts(50, 2, 15)
    W, _, v0, _ = orc.degree_normalize(orc.affinity(X, 1.0))
    r = orc.power_iterate_dense(W, v0, "fixed", 25, eps=1.0)
    assert r.iterations == 25 and not r.converged and r.stats.shape == (25,)


# ------------------------------------------------------------------ k-means
def _exhaustive(v, k):
    """Minimum within-cluster sum of squares over every labelling."""
    best = np.inf
    for lab in itertools.product(range(k), repeat=len(v)):
        lab = np.array(lab)
        if len(set(lab)) != k:
            continue
        c = sum(((v[lab == j] - v[lab == j].mean()) ** 2).sum() for j in range(k))
        best = min(best, c)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_kmeans_exact_against_all_labellings(orc, seed):
    """P10: the optimum over every labelling (not only contiguous ones)."""
    rng = np.random.default_rng(seed)
    v = rng.standard_normal(7)
    for k in (1, 2, 3):
        for method in ("plain", "dc"):
            r = orc.kmeans1d(v, k, method)
            assert r.cost == pytest.approx(_exhaustive(v, k), rel=1e-12, abs=1e-15)
            cent = np.array([v[r.labels == j].mean() for j in range(r.k_eff)])
            np.testing.assert_allclose(r.centroids, cent, rtol=1e-14)
            assert np.all(np.diff(r.centroids) > 0)


def test_kmeans_special_cases(orc):
    v = np.array([3.0, 1.0, 2.0, 10.0, 11.0])
    r = orc.kmeans1d(v, 1)
    assert np.all(r.labels == 0) and r.centroids[0] == pytest.approx(v.mean())
    r = orc.kmeans1d(v, 5)
    assert r.k_eff == 5 and r.cost == 0.0
    assert list(r.labels) == [2, 0, 1, 3, 4]
    # duplicates never split; fewer distinct values than k gives k_eff < k
    r = orc.kmeans1d(np.array([1.0, 1.0, 2.0, 2.0, 2.0]), 4)
    assert r.k_eff == 2 and list(r.labels) == [0, 0, 1, 1, 1]
    # well-separated groups are recovered
    rng = np.random.default_rng(1)
    g = np.repeat([0.0, 5.0, 9.0, 20.0], 50) + 0.1 * rng.standard_normal(200)
    truth = np.repeat([0, 1, 2, 3], 50)
    r = orc.kmeans1d(g, 4, "dc")
    assert np.array_equal(r.labels, truth)


@pytest.mark.parametrize("seed", range(4))
def test_kmeans_dc_equals_plain(orc, seed):
    """The divide-and-conquer search returns the plain programme's partition."""
    rng = np.random.default_rng(100 + seed)
    n = 1500
    v = np.concatenate([rng.standard_normal(n // 3) * s + m for m, s in
                        ((0, 1), (4, 0.5), (9, 2))])
    if seed % 2:
        v = np.round(v, 1)       # many duplicate values
    for k in (2, 5, 9):
        a = orc.kmeans1d(v, k, "plain")
        b = orc.kmeans1d(v, k, "dc")
        assert a.k_eff == b.k_eff
        assert b.cost == pytest.approx(a.cost, rel=1e-12)
        assert np.array_equal(a.labels, b.labels)


def test_pic_recovers_separated_blobs(orc):
    """End to end on three far-apart blobs: labels match the truth."""
    import workloads
    w = workloads.make("blobs2d")
    r = orc.pic_dense(w.X, w.sigma, w.k, "converge", 1000, w.eps)
    assert r.pi.converged
    from sklearn.metrics import adjusted_rand_score
    assert adjusted_rand_score(w.y_true, r.km.labels) > 0.99


# ------------------------------------------------ P7: 50-digit brute force
def _mp_pic(X, sigma, T, kind="gauss"):
    """Algorithm 1 at 50 significant digits (mpmath), from the float32
    points promoted exactly: A, D, W = D^-1 A, v0 = d / sum d, delta_0 = v0,
    then T updates v <- W v / ||W v||_1 with the velocity statistic."""
    import mpmath as mp
    mp.mp.dps = 50
    n, d = X.shape
    P = [[mp.mpf(float(X[i, c])) for c in range(d)] for i in range(n)]
    s2 = 2 * mp.mpf(float(np.float32(sigma))) ** 2
    A = [[mp.mpf(0)] * n for _ in range(n)]
    for i in range(n):
        for j in range(n):
            if i == j:
                continue
            if kind == "gauss":
                A[i][j] = mp.e ** (-sum((P[i][c] - P[j][c]) ** 2 for c in range(d)) / s2)
            else:
                dot = sum(P[i][c] * P[j][c] for c in range(d))
                ni = mp.sqrt(sum(x * x for x in P[i]))
                nj = mp.sqrt(sum(x * x for x in P[j]))
                A[i][j] = (1 + dot / (ni * nj)) / 2
    deg = [sum(A[i]) for i in range(n)]
    W = [[A[i][j] / deg[i] for j in range(n)] for i in range(n)]
    tot = sum(deg)
    v = [x / tot for x in deg]
    delta = list(v)
    stats = []
    for _ in range(T):
        y = [sum(W[i][j] * v[j] for j in range(n)) for i in range(n)]
        tau = sum(abs(x) for x in y)
        vn = [x / tau for x in y]
        dn = [abs(a - b) for a, b in zip(vn, v)]
        stats.append(max(abs(a - b) for a, b in zip(dn, delta)))
        v, delta = vn, dn
    return ([float(x) for x in deg], np.array([float(x) for x in v]),
            np.array([float(x) for x in stats]), [[float(x) for x in r] for r in W])


@pytest.mark.parametrize("n,seed,kind", [(5, 1, "gauss"), (8, 2, "gauss"), (7, 3, "cosine")])
def test_brute_force_fifty_digits(orc, n, seed, kind):
    """P7: the whole method on n <= 8 points at 50 digits agrees with the
    float64 oracle to rounding: degrees, W, v and every statistic after
    T = 6 updates; a stop threshold placed between two statistics stops
    both at the same update; k-means against all contiguous partitions."""
    X = _pts(n, 2, 900 + seed, scale=1.2)
    sigma = np.float32(0.9)
    T = 6
    deg_m, v_m, st_m, W_m = _mp_pic(X, sigma, T, kind)
    A = orc.affinity(X, sigma) if kind == "gauss" else orc.affinity_cosine(X)
    W, deg, v0, _ = orc.degree_normalize(A)
    np.testing.assert_allclose(deg, deg_m, rtol=1e-14)
    # absolute floor: (1 + cos) / 2 for nearly opposite points cancels in
    # float64 (an error of 1e-16 in cos on an entry near 0)
    np.testing.assert_allclose(W, np.array(W_m), rtol=1e-14, atol=4e-16)
    r = orc.power_iterate_dense(W, v0, "fixed", T)
    np.testing.assert_allclose(r.v, v_m, rtol=1e-13)
    np.testing.assert_allclose(r.stats, st_m, rtol=1e-9, atol=1e-17)
    # stop between updates 3 and 4 (statistics decreasing there)
    if st_m[2] > st_m[3]:
        eps = float(np.sqrt(st_m[2] * st_m[3]))
        rc = orc.power_iterate_dense(W, v0, "converge", 100, eps)
        stop = next(t for t in range(T) if st_m[t] <= eps) + 1
        assert rc.iterations == stop and rc.converged
    # k-means of the 50-digit v by enumerating contiguous partitions
    order = np.argsort(v_m, kind="stable")
    vs = v_m[order]
    for k in (2, 3):
        best = min(sum(((vs[a:b] - vs[a:b].mean()) ** 2).sum()
                       for a, b in zip((0,) + cuts, cuts + (n,)))
                   for cuts in itertools.combinations(range(1, n), k - 1))
        km = orc.kmeans1d(r.v, k)
        assert km.cost == pytest.approx(best, rel=1e-9, abs=1e-20)


# ------------------------------------------------------- kNN input graph
def test_knn_graph_matches_ckdtree(orc):
    """The exact kNN graph equals one built from scipy's k-d tree (a library
    kNN routine) with union symmetrisation and the Gaussian weights."""
    import scipy.sparse as sp
    from scipy.spatial import cKDTree
    n, d, k, sigma = 1500, 8, 10, np.float32(1.3)
    X = _pts(n, d, 71)
    rp, col, val = orc.knn_graph(X, k, sigma)
    P = X.astype(np.float64)
    dist, nb = cKDTree(P).query(P, k=k + 1)
    assert np.all(nb[:, 0] == np.arange(n))            # no duplicate points here
    rows = np.repeat(np.arange(n), k)
    cols = nb[:, 1:].reshape(-1)
    w = np.exp(-(dist[:, 1:].reshape(-1) ** 2) / (2.0 * float(sigma) ** 2))
    K = sp.coo_matrix((w, (rows, cols)), shape=(n, n)).tocsr()
    S = K.maximum(K.T).tocsr()
    S.sort_indices()
    assert np.array_equal(rp, S.indptr) and np.array_equal(col, S.indices)
    np.testing.assert_allclose(val, S.data.astype(np.float32), rtol=2e-7)


def test_knn_rows_matches_ckdtree(orc):
    """The neighbour lists of listed points alone equal scipy's k-d tree
    query (a library kNN routine): same points in the same order, squared
    distances to rounding, Gaussian weights; and on an integer lattice the
    ties go to the smaller index (corner point 0: 1 and 12 at distance 1,
    13 at sqrt 2, then 2 before 24 at distance 2)."""
    from scipy.spatial import cKDTree
    n, d, k, sigma = 2000, 8, 12, np.float32(0.9)
    X = _pts(n, d, 73)
    rows = np.array([0, 1, 777, 1998, 1999], dtype=np.int64)
    nbr, d2, w = orc.knn_rows(X, k, sigma, rows)
    P = X.astype(np.float64)
    dist, nb = cKDTree(P).query(P[rows], k=k + 1)
    assert np.all(nb[:, 0] == rows)
    assert np.array_equal(nbr, nb[:, 1:])
    np.testing.assert_allclose(d2, dist[:, 1:] ** 2, rtol=1e-12)
    np.testing.assert_allclose(w, np.exp(-dist[:, 1:] ** 2 / (2.0 * float(sigma) ** 2)),
                               rtol=2e-7)
    g = np.arange(12, dtype=np.float32)
    L = np.stack(np.meshgrid(g, g), axis=-1).reshape(-1, 2)
    nbr, d2, _ = orc.knn_rows(L, 4, 1.0, [0])
    assert list(nbr[0]) == [1, 12, 13, 2] and list(d2[0]) == [1.0, 1.0, 2.0, 4.0]
    with pytest.raises(ValueError):
        orc.knn_rows(L, 4, 1.0, [144])


def test_knn_graph_ties_and_structure(orc):
    """Integer lattice points (many exact distance ties): ties go to the
    smaller index; the graph is symmetric with equal weights both ways, has
    no self loops, sorted columns and at least k entries per row."""
    g = np.arange(12, dtype=np.float32)
    X = np.stack(np.meshgrid(g, g), axis=-1).reshape(-1, 2)      # 144 points
    n, k = X.shape[0], 4
    rp, col, val = orc.knn_graph(X, k, 1.0)
    A = np.zeros((n, n), dtype=np.float32)
    for i in range(n):
        c = col[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0) and i not in c and c.size >= k
        A[i, c] = val[rp[i]:rp[i + 1]]
    assert np.array_equal(A, A.T)
    # corner point 0 = (0, 0): nearest are (1, 0) idx 1 and (0, 1) idx 12 at
    # distance 1, (1, 1) idx 13 at sqrt 2, then (2, 0) idx 2 and (0, 2) idx
    # 24 tie at 2 and the smaller index wins; no other point has 0 among
    # its own 4 nearest, so row 0 is exactly {1, 2, 12, 13}
    assert list(col[rp[0]:rp[1]]) == [1, 2, 12, 13]
    assert A[0, 1] == np.float32(np.exp(-0.5)) and A[0, 2] == np.float32(np.exp(-2.0))
