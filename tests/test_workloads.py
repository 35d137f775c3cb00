"""The seeded generators are deterministic and shaped as described."""
import numpy as np

import workloads


def test_deterministic_and_shapes():
    a = workloads.make("blobs2d")
    b = workloads.make("blobs2d")
    assert a.meta()["sha256_X"] == b.meta()["sha256_X"]
    assert a.X.shape == (1000, 2) and a.X.dtype == np.float32
    assert np.bincount(a.y_true).tolist() == [334, 333, 333]
    assert a.eps == 1e-5 / 1000 and a.sigma == np.float32(1.0)
    c = workloads.make("blobs2d", seed=101)
    assert c.meta()["sha256_X"] != a.meta()["sha256_X"]


def test_rings_and_blobs16d():
    r = workloads.make("rings2d")
    assert r.X.shape == (10000, 2)
    rad = np.hypot(r.X[:, 0], r.X[:, 1])
    for c, rr in enumerate((1.0, 3.0, 5.0)):
        assert abs(np.median(rad[r.y_true == c]) - rr) < 0.05
    w = workloads.make("blobs16d", n=3000)
    assert w.X.shape == (3000, 16) and w.k == 10 and w.max_iter == 50
    assert np.bincount(w.y_true).sum() == 3000
    assert w.sigma.dtype == np.float32 and w.sigma > 0


def test_split_rules():
    assert workloads.split_equal(10, 3).tolist() == [4, 3, 3]
    rng = np.random.default_rng(0)
    s = workloads.split_dirichlet(rng, 1001, 7, 5.0)
    assert s.sum() == 1001 and s.min() >= 0


def test_knn_graph_small():
    w = workloads.make("knn8d", n=2000)
    rp, col, val = w.row_ptr, w.col, w.val
    n = 2000
    assert rp.shape == (n + 1,) and rp[0] == 0 and rp[-1] == col.shape[0]
    deg = np.diff(rp)
    assert deg.min() >= 32                      # union symmetrisation
    assert np.all(col >= 0) and np.all(col < n)
    for i in range(0, n, 97):                   # sorted, no self loops
        c = col[rp[i]:rp[i + 1]]
        assert np.all(np.diff(c) > 0) and i not in c
    import scipy.sparse as sp
    M = sp.csr_matrix((val, col, rp), shape=(n, n))
    assert abs(M - M.T).max() == 0
    assert val.dtype == np.float32 and np.all(val > 0) and np.all(val <= 1)


def test_random_kout_graph():
    rp, col, val = workloads.random_kout_graph(300, 7, 3)
    assert rp.dtype == np.int64 and col.dtype == np.int32 and val.dtype == np.float32
    assert np.array_equal(rp, np.arange(301) * 7) and col.shape == val.shape == (2100,)
    assert np.all(col >= 0) and np.all(col < 300)
    assert np.all(np.diff(col.reshape(300, 7), axis=1) >= 0)      # rows sorted
    assert np.all(val >= 0.1) and np.all(val < 1.0)
    again = workloads.random_kout_graph(300, 7, 3)
    assert all(np.array_equal(a, b) for a, b in zip((rp, col, val), again))
