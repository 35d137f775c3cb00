"""GPU parity past the 32-bit index limits of each operator's storage.

* Dense W with more than 2^32 entries (n = 70,001, 19.6 GB of float32 W):
  degrees and one product on sampled rows, among them rows whose entries
  lie past entry 2^32, recomputed one by one by the oracle; the update's
  invariants over a few updates.
* Symmetric storage of the same points (entries past 2^31 in the packed
  tiles): sampled rows of one product against the oracle.
* One tile of the staged CSR product with more than 2^31 entries (an
  exact row sum).
* The fused operator at the largest n that evaluates each pair once
  (2^19, d = 64): W 1 = 1 over the whole vector, sampled rows against the
  oracle.
* CSR graphs with more than 2^31 stored entries, one for each product
  form (staged: up to 64 entries per row on average; row-wise: more;
  column-blocked: sorted rows, no locality, n <= 2^23).  Each graph is B
  copies of a random graph G0 on disjoint node ranges (block diagonal).
  The update v <- W v / ||W v||_1 does not depend on the scale of v and
  v_0 = d / sum(d), so every copy iterates as G0 alone with each iterate
  and each stop statistic divided by B.  B is a power of two, so the
  oracle runs on G0 and the GPU's first copy times B must match it to
  rounding, and since every copy's rows sit in the same relative place,
  every copy must hold the same bits.
* The kNN graph builder with room for more than 2^31 entries (n = 17M,
  k = 64): structure and mirror symmetry over the whole graph, sampled rows
  against the oracle's neighbour lists.
* 1-D k-means at its documented maximum, n = 2^30 values, k = 2: the
  split against a brute force over every split point.
"""
import numpy as np
import pytest

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


# --------------------------------------------------------------- dense W
@pytest.fixture(scope="module")
def big_blobs():
    import workloads
    return workloads.make("blobs16d", n=70_001)


def _sample_rows(n, ld, seed):
    """Row edges, rows around the one whose entries first pass 2^32, the
    last rows, and random rows."""
    cross = (1 << 32) // ld
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 255, 256, cross - 1, cross, cross + 1, n - 2, n - 1]
    return np.unique(np.concatenate([fixed, rng.choice(n, 12, replace=False)])
                     ).astype(np.int64)


def test_dense_past_2_32_entries(g, orc, big_blobs):
    w = big_blobs
    n = w.n
    assert n * g.padded_ld(n) > 1 << 32
    print(f"gpu: dense blobs16d n={n} ({n * g.padded_ld(n) * 4 / 1e9:.1f} GB of W)",
          flush=True)
    W, deg, v0, nz = g.gpic_affinity_normalized(_t(w.X), w.sigma)
    rows = _sample_rows(n, W.stride(0), 3)
    dr = orc.degree_rows(w.X, w.sigma, rows)
    np.testing.assert_allclose(deg.cpu().numpy()[rows], dr, rtol=1e-5)
    # one product on a positive v, the sampled rows recomputed one by one
    vr = np.random.default_rng(8).uniform(0.5, 1.5, size=n)
    y = g.gpic_matvec_dense(W, _t(vr), n=n).cpu().numpy()
    dfull = np.zeros(n)
    dfull[rows] = dr
    yr = orc.matvec_onthefly_rows(w.X, w.sigma, dfull, vr, rows)
    np.testing.assert_allclose(y[rows], yr, rtol=1e-5)
    # three updates: v stays a probability vector, and the last update is
    # y / ||y||_1 of the product of the second iterate
    v = v0.clone()
    g.gpic_power_iterate_dense(W, v, None, "fixed", 2, n=n)
    v2 = v.clone()
    out = g.gpic_power_iterate_dense(W, v, None, "fixed", 1, n=n)
    assert out.iterations == 1
    y2 = g.gpic_matvec_dense(W, v2, n=n).cpu().numpy()
    vg = v.cpu().numpy()
    np.testing.assert_allclose(vg, y2 / np.abs(y2).sum(), rtol=1e-12)
    assert np.all(vg >= 0) and abs(vg.sum() - 1.0) < 1e-12
    del W
    torch.cuda.empty_cache()


def test_sym_past_2_31_entries(g, orc, big_blobs):
    w = big_blobs
    n = w.n
    assert g.sym_bytes(n) // 4 > 1 << 31
    print(f"gpu: symmetric blobs16d n={n} ({g.sym_bytes(n) / 1e9:.1f} GB of tiles)",
          flush=True)
    As, deg, v0, nz = g.gpic_affinity_sym(_t(w.X), w.sigma)
    rows = _sample_rows(n, n, 5)
    dr = orc.degree_rows(w.X, w.sigma, rows)
    np.testing.assert_allclose(deg.cpu().numpy()[rows], dr, rtol=1e-5)
    vr = np.random.default_rng(9).uniform(0.5, 1.5, size=n)
    y = g.gpic_matvec_sym(As, n, deg, _t(vr)).cpu().numpy()
    dfull = np.zeros(n)
    dfull[rows] = dr
    yr = orc.matvec_onthefly_rows(w.X, w.sigma, dfull, vr, rows)
    np.testing.assert_allclose(y[rows], yr, rtol=1e-5)
    del As
    torch.cuda.empty_cache()


def test_csr_staged_tile_past_2_31_entries(g):
    """One 256-row tile of the staged product holding more than 2^31
    entries: row 256 holds 2^31 + 100 entries of weight 1 (columns cycling
    over all nodes), the other rows of its tile and of the graph none, and
    v = 1, so y at that row is exactly its entry count and 0 elsewhere.
    The rows after it in the tile lie more than 2^31 entries past the
    early rounds, the case whose round bounds must be clamped in 64 bits
    before they are narrowed.  (A mean of 64 entries per row at most keeps
    the staged product: n = 2^25 + 2^20.)"""
    n = (1 << 25) + (1 << 20)
    big = (1 << 31) + 100
    assert big <= 64 * n
    print(f"gpu: staged tile with {big} entries in one row, n={n}", flush=True)
    rp = torch.zeros(n + 1, dtype=torch.int64, device=DEV)
    rp[257:] = big
    col = (torch.arange(big, dtype=torch.int64, device=DEV) % n).to(torch.int32)
    val = torch.ones(big, dtype=torch.float32, device=DEV)
    v = torch.ones(n, dtype=torch.float64, device=DEV)
    y = g.gpic_matvec_csr(rp, col, val, v)
    assert float(y[256].item()) == float(big)
    y[256] = 0.0
    assert float(y.abs().max().item()) == 0.0
    del rp, col, val, v, y
    torch.cuda.empty_cache()


# ---------------------------------------------------- fused operator
def test_fused_pair_once_at_2_19(g, orc):
    """The fused operator's largest size that evaluates each pair once,
    n = 2^19 points of 64 dimensions (4.3 GB of column partial sums):
    sampled degrees and one product against the oracle's rows, and over
    the whole vector W 1 = 1 to 1e-12 (the degrees are the row sums of the
    same symmetric A the product uses, each pair's term shared by its row
    and its column)."""
    import workloads
    n = 1 << 19
    X, _ = workloads.blobs_equal(n=n, d=64, k=20, seed=17)
    sigma = np.float32(4.0)
    print(f"gpu: fused pair-once n={n} d=64", flush=True)
    Xg = _t(X)
    deg, v0, nz = g.gpic_degree_fused(Xg, sigma)
    ones = torch.ones(n, dtype=torch.float64, device=DEV)
    y1 = g.gpic_matvec_fused(Xg, sigma, deg, ones).cpu().numpy()
    np.testing.assert_allclose(y1, 1.0, rtol=1e-12)
    rng = np.random.default_rng(6)
    rows = np.unique(np.concatenate([[0, 1, 383, 384, n // 2, n - 385, n - 384, n - 2, n - 1],
                                     rng.choice(n, 12, replace=False)])).astype(np.int64)
    dr = orc.degree_rows(X, sigma, rows)
    np.testing.assert_allclose(deg.cpu().numpy()[rows], dr, rtol=1e-4)
    vr = rng.uniform(0.5, 1.5, size=n)
    y = g.gpic_matvec_fused(Xg, sigma, deg, _t(vr)).cpu().numpy()
    dfull = np.zeros(n)
    dfull[rows] = dr
    yr = orc.matvec_onthefly_rows(X, sigma, dfull, vr, rows)
    np.testing.assert_allclose(y[rows], yr, rtol=1e-4)
    del Xg, deg, v0, ones
    torch.cuda.empty_cache()


# ------------------------------------------------------------------- CSR
def _replicate(rp0, col0, val0, B):
    """B copies of G0 on the GPU, copy b on nodes [b m, (b + 1) m)."""
    m, nnz0 = rp0.size - 1, col0.size
    assert B * m < 1 << 31
    offs = torch.arange(B, dtype=torch.int32, device=DEV) * m
    col = (_t(col0).unsqueeze(0) + offs.unsqueeze(1)).reshape(-1)
    val = _t(val0).repeat(B)
    starts = (_t(rp0[:-1]).unsqueeze(0)
              + torch.arange(B, dtype=torch.int64, device=DEV).unsqueeze(1) * nnz0)
    end = torch.tensor([B * nnz0], dtype=torch.int64, device=DEV)
    rp = torch.cat([starts.reshape(-1), end])
    return rp, col, val


def _copies_equal(x, B):
    """Every one of the B equal-length slices of x holds the bits of the first."""
    xs = x.view(B, -1)
    same = True
    for b in range(1, B):
        same = same and torch.equal(xs[b], xs[0])
    return same


@pytest.mark.parametrize("form,m,k,B", [
    ("staged", 104_729, 41, 512),       # 41 entries per row: staged tiles
    ("row-wise", 104_729, 81, 256),     # 81 per row: 16 lanes per row
    ("column-blocked", 1 << 19, 257, 16),   # n = 2^23, sorted rows, far columns
])
def test_csr_past_2_31_entries(g, orc, form, m, k, B):
    import workloads
    rp0, col0, val0 = workloads.random_kout_graph(m, k, 11 + k)
    n, nnz = B * m, B * col0.size
    assert nnz > 1 << 31 and (B & (B - 1)) == 0
    print(f"gpu: csr {form} n={n} nnz={nnz} ({B} copies of m={m}, k={k})", flush=True)
    rp, col, val = _replicate(rp0, col0, val0, B)
    _, deg, v0, nz = g.gpic_degree_normalize_csr(rp, col, val)
    assert int(nz.item()) == 0
    _, dr, v0r, _ = orc.degree_normalize_csr(rp0, col0, val0)
    assert _copies_equal(deg, B) and _copies_equal(val, B)
    np.testing.assert_allclose(deg[:m].cpu().numpy(), dr, rtol=1e-12)
    np.testing.assert_allclose(v0[:m].cpu().numpy() * B, v0r, rtol=1e-12)
    # stage isolation: the oracle iterates on the GPU's float32 W of a copy
    wg = val[:col0.size].cpu().numpy().astype(np.float64)
    T = 6
    ref = orc.power_iterate_csr(rp0, col0, wg, v0r, "fixed", T)
    v = v0.clone()
    out = g.gpic_power_iterate_csr(rp, col, val, v, None, "fixed", T)
    assert out.iterations == T
    assert _copies_equal(v, B)
    np.testing.assert_allclose(v[:m].cpu().numpy() * B, ref.v, rtol=1e-9)
    np.testing.assert_allclose(out.stats * B, ref.stats, rtol=1e-6, atol=1e-18)
    del rp, col, val, deg, v0, v
    torch.cuda.empty_cache()


# ------------------------------------------------------------- kNN graph
def _mix64(x):
    """A 64-bit mixing step on int64 tensors (wrapping arithmetic)."""
    x = x ^ (x >> 31)
    x = x * 0x7FB5D329728EA185
    x = x ^ (x >> 27)
    x = x * 0x2545F4914F6CDD1D
    return x ^ (x >> 33)


def _mirror_fingerprints(rp, col, val, chunk=1 << 27):
    """Wrapping sums of a hash of (min(i, j), max(i, j), weight bits) over
    the stored entries with i < j and over those with i > j: equal when
    every edge is stored both ways with the same weight."""
    nnz = col.numel()
    lo_sum = torch.zeros((), dtype=torch.int64, device=DEV)
    hi_sum = torch.zeros((), dtype=torch.int64, device=DEV)
    bounds = rp[1:].contiguous()
    for s in range(0, nnz, chunk):
        p = torch.arange(s, min(nnz, s + chunk), dtype=torch.int64, device=DEV)
        r = torch.searchsorted(bounds, p, right=True)
        c = col[s:s + p.numel()].to(torch.int64)
        wb = val[s:s + p.numel()].view(torch.int32).to(torch.int64)
        h = _mix64(torch.minimum(r, c) * 0x100000001B3 + torch.maximum(r, c)
                   + (wb << 40))
        lo_sum += torch.where(r < c, h, torch.zeros_like(h)).sum()
        hi_sum += torch.where(r > c, h, torch.zeros_like(h)).sum()
        assert not bool((r == c).any())                      # no self loops
    return int(lo_sum.item()), int(hi_sum.item())


def test_knn_graph_past_2_31_entries(g, orc):
    """n = 17,000,000 8-D points, k = 64: room for 2 n k > 2^31 entries.
    Whole graph: rows sorted, at least k entries each, no self loops, every
    edge stored both ways with one weight (hash fingerprints).  Sampled
    rows against the oracle's neighbour lists: each of a row's k nearest
    is in the row with its weight, and a sampled entry that is not among
    them has the row's point among its own k nearest."""
    import workloads
    n, k, sigma = 17_000_000, 64, 1.0
    assert 2 * n * k > 1 << 31 and 2 * n * k < 1 << 32
    X, _ = workloads.blobs_equal(n=n, d=8, k=50, seed=31)
    print(f"gpu: knn graph n={n} d=8 k={k}", flush=True)
    rp, col, val = g.gpic_knn_graph(_t(X), k, sigma)
    torch.cuda.empty_cache()
    nnz = col.numel()
    print(f"  nnz={nnz}", flush=True)
    assert int(rp[0].item()) == 0 and int(rp[-1].item()) == nnz
    assert n * k <= nnz <= 2 * n * k
    assert int((rp[1:] - rp[:-1]).min().item()) >= k
    starts = torch.zeros(nnz, dtype=torch.bool, device=DEV)
    starts[rp[:-1]] = True
    up = col[1:] > col[:-1]
    assert bool((up | starts[1:]).all())                     # rows strictly sorted
    del starts, up
    lo, hi = _mirror_fingerprints(rp, col, val)
    assert lo == hi
    rows = np.concatenate([[0, 1, n // 2, n - 1],
                           np.random.default_rng(4).choice(n, 4, replace=False)])
    nbr, d2, w = orc.knn_rows(X, k, sigma, rows)
    rph = rp.cpu().numpy()
    extra = []
    for t, i in enumerate(rows):
        c = col[rph[i]:rph[i + 1]].cpu().numpy()
        v = val[rph[i]:rph[i + 1]].cpu().numpy()
        pos = np.searchsorted(c, nbr[t])
        assert np.all(pos < c.size) and np.array_equal(c[pos], nbr[t])
        assert np.all(np.abs(v[pos] - w[t]) <= np.spacing(w[t]))
        rest = np.setdiff1d(c, nbr[t])
        for j in rest[[0, rest.size // 2, -1]] if rest.size else []:
            extra.append((int(i), int(j), float(v[np.searchsorted(c, j)])))
    if extra:
        nb2, _, w2 = orc.knn_rows(X, k, sigma, [j for _, j, _ in extra])
        for (i, j, wij), nj, wj in zip(extra, nb2, w2):
            hit = np.nonzero(nj == i)[0]
            assert hit.size == 1, f"entry ({i}, {j}) without i among j's nearest"
            assert abs(wij - wj[hit[0]]) <= np.spacing(wj[hit[0]])
    print(f"  sampled rows {len(rows)}, reverse entries checked {len(extra)}", flush=True)
    del rp, col, val
    torch.cuda.empty_cache()


# --------------------------------------------------------------- k-means
def _mixture_quantiles(n, seed):
    """n sorted values: evenly spaced quantiles of a mixture of two
    overlapping uniform distributions (60 % on [-3, 1], 40 % on [0, 3]),
    each shifted by a seeded fraction of its spacing, then merged; a k = 2
    optimum sits inside the overlap.  No sort of random values at n = 2^30."""
    rng = np.random.default_rng(seed)
    na = int(0.6 * n)
    parts = []
    for m, lo, hi in ((na, -3.0, 1.0), (n - na, 0.0, 3.0)):
        u = np.arange(m, dtype=np.float64)
        u += rng.uniform(0.25, 0.75)
        u *= (hi - lo) / m
        u += lo
        parts.append(u)
    v = np.concatenate(parts)
    del parts, u
    v.sort(kind="stable")                   # two sorted runs: a merge
    return v


def _split_cost(vs, s):
    """Within-cluster sum of squares of vs[:s] and vs[s:] (sorted vs),
    each side centred on its own mean; numpy's pairwise sums."""
    tot = 0.0
    for part in (vs[:s], vs[s:]):
        tot += float(np.sum(np.square(part - part.mean())))
    return tot


def _best_split(vs, chunk=1 << 25):
    """Brute force over all n - 1 split points with centred float64 prefix
    sums (left size j: S2_j - S1_j^2 / j, the right side alike)."""
    n = vs.size
    u = vs - vs.mean()
    S1 = np.cumsum(u)
    np.square(u, out=u)
    S2 = np.cumsum(u, out=u)
    t1, t2 = S1[-1], S2[-1]
    best, arg = np.inf, -1
    for a in range(1, n, chunk):
        e = min(n, a + chunk)
        j = np.arange(a, e, dtype=np.float64)
        s1, s2 = S1[a - 1:e - 1], S2[a - 1:e - 1]
        c = s2 - s1 * s1 / j
        c += (t2 - s2) - np.square(t1 - s1) / (n - j)
        i = int(np.argmin(c))
        if c[i] < best:
            best, arg = float(c[i]), a + i
    return arg


def test_kmeans1d_at_2_30_values(g):
    """The documented maximum n = 2^30, k = 2: the values in an affine
    permutation of their sorted order, so the GPU sorts them.  Its clusters
    must be contiguous in value, its split as good as the best of all
    2^30 - 1 split points (both costs recomputed with pairwise sums, to
    1e-9), its reported cost and centroids those of its own split."""
    n = 1 << 30
    print(f"gpu: kmeans1d n={n} k=2", flush=True)
    vs = _mixture_quantiles(n, 21)
    assert np.all(np.diff(vs[:: 1 << 20]) >= 0)
    perm_a, perm_b = 0x9E3779B1, 12345             # odd: a bijection modulo 2^30
    vsg = _t(vs)
    idx = (torch.arange(n, dtype=torch.int64, device=DEV) * perm_a + perm_b) % n
    v = vsg[idx]
    del vsg, idx
    torch.cuda.empty_cache()
    km = g.gpic_kmeans1d(v, 2)
    assert km.k_eff == 2
    lab = km.labels
    a = int((lab == 0).sum().item())
    lo_max = float(torch.where(lab == 0, v, torch.full_like(v, -np.inf)).max().item())
    hi_min = float(torch.where(lab == 1, v, torch.full_like(v, np.inf)).min().item())
    assert 0 < a < n and lo_max < hi_min and lo_max == vs[a - 1] and hi_min == vs[a]
    cent = km.centroids.cpu().numpy()
    del v, lab, km.labels
    torch.cuda.empty_cache()
    b = _best_split(vs)
    ca, cb = _split_cost(vs, a), _split_cost(vs, b)
    print(f"  split gpu={a} brute force={b} cost {ca:.12e} vs {cb:.12e}", flush=True)
    assert abs(ca - cb) <= 1e-9 * cb
    assert km.cost == pytest.approx(ca, rel=1e-9)
    np.testing.assert_allclose(cent, [vs[:a].mean(), vs[a:].mean()], rtol=1e-9)
