"""GPU parity past the 32-bit index limits of each operator's storage.

* Dense W with more than 2^32 entries (n = 70,001, 19.6 GB of float32 W):
  degrees and one product on sampled rows, among them rows whose entries
  lie past entry 2^32, recomputed one by one by the oracle; the update's
  invariants over a few updates.
* Symmetric storage of the same points (entries past 2^31 in the packed
  tiles): sampled rows of one product against the oracle.
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
