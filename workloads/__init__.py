"""Seeded synthetic inputs shaped like the paper's clustering workloads.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no arithmetic of the clustering method itself: it draws points, picks
the Gaussian width and (for the sparse workload) builds the kNN input graph,
then hands plain numpy arrays to whichever side is being exercised.

The paper's own data sets (two moons, three circles; Experiment I, Table 2)
are not available, so these stand in for them, with the paper's m = 2 shape
at small n and n = 50,000 just above its largest case (45,000).

Every generator draws from ``numpy.random.default_rng(seed)`` in a fixed
order: centres, then cluster sizes, then the points cluster by cluster,
then one permutation applied to points and true labels, then (where the
width is data dependent) the sample used to pick it.  Points are drawn in
float64 and rounded to float32 exactly once.
"""
from __future__ import annotations

import dataclasses
import hashlib
import os
from typing import Optional

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "make", "blobs_uniform_centres", "rings", "two_moons",
    "blobs_dirichlet", "blobs_equal", "knn_graph", "random_kout_graph", "sha256_of",
    "split_equal", "split_dirichlet", "median_pair_distance_sigma",
]


@dataclasses.dataclass
class Workload:
    name: str
    X: np.ndarray                 # float32 [n, d], row-major
    y_true: np.ndarray            # int32 [n]
    sigma: np.float32             # Gaussian width handed to both sides
    eps: float                    # stopping precision (1e-5 / n)
    k: int                        # clusters for the final 1-D k-means
    mode: str                     # "converge" or "fixed"
    max_iter: int                 # T in fixed mode, the cap otherwise
    path: str                     # "dense", "fused", "csr" or "cosine" (dense W)
    seed: int
    # sparse workload only: fp32 CSR affinity graph, rows sorted by column
    row_ptr: Optional[np.ndarray] = None   # int64 [n + 1]
    col: Optional[np.ndarray] = None       # int32 [nnz]
    val: Optional[np.ndarray] = None       # float32 [nnz]

    @property
    def n(self) -> int:
        return int(self.X.shape[0])

    @property
    def d(self) -> int:
        return int(self.X.shape[1])

    def meta(self) -> dict:
        m = {"name": self.name, "n": self.n, "d": self.d,
             "sigma": float(self.sigma), "eps": self.eps, "k": self.k,
             "mode": self.mode, "max_iter": self.max_iter,
             "path": self.path, "seed": self.seed,
             "sha256_X": sha256_of(self.X)}
        if self.val is not None:
            m["nnz"] = int(self.val.shape[0])
            m["sha256_csr"] = sha256_of(self.row_ptr, self.col, self.val)
        return m


def sha256_of(*arrays: np.ndarray) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()


def split_equal(n: int, k: int) -> np.ndarray:
    """Equal cluster sizes; the first n % k clusters get one extra point."""
    sizes = np.full(k, n // k, dtype=np.int64)
    sizes[: n % k] += 1
    return sizes


def split_dirichlet(rng: np.random.Generator, n: int, k: int,
                    alpha: float) -> np.ndarray:
    """floor(n p) with p ~ Dirichlet(alpha 1_k); the remainder goes to the
    largest fractional parts, ties to the lower index."""
    p = rng.dirichlet(np.full(k, alpha))
    raw = n * p
    sizes = np.floor(raw).astype(np.int64)
    frac = raw - sizes
    rem = n - int(sizes.sum())
    order = sorted(range(k), key=lambda c: (-frac[c], c))
    for c in order[:rem]:
        sizes[c] += 1
    return sizes


def _finish(rng, pts64, labels):
    perm = rng.permutation(pts64.shape[0])
    X = np.ascontiguousarray(pts64[perm].astype(np.float32))
    y = np.ascontiguousarray(labels[perm].astype(np.int32))
    return X, y


def _gaussian_clusters(rng, centres, sizes, std):
    d = centres.shape[1]
    pts, lab = [], []
    for c, (mu, m) in enumerate(zip(centres, sizes)):
        pts.append(mu + std * rng.standard_normal((int(m), d)))
        lab.append(np.full(int(m), c, dtype=np.int32))
    return np.concatenate(pts), np.concatenate(lab)


def blobs_uniform_centres(n=1000, d=2, k=3, box=10.0, std=1.0, seed=1):
    """Isotropic blobs, centres uniform in [-box, box]^d, equal sizes."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(-box, box, size=(k, d))
    sizes = split_equal(n, k)
    pts, lab = _gaussian_clusters(rng, centres, sizes, std)
    return _finish(rng, pts, lab)


def rings(n=10000, radii=(1.0, 3.0, 5.0), noise=0.1, seed=2):
    """Concentric rings in 2-D: angle uniform, radius r + N(0, noise^2)."""
    rng = np.random.default_rng(seed)
    k = len(radii)
    sizes = split_equal(n, k)
    pts, lab = [], []
    for c, (r, m) in enumerate(zip(radii, sizes)):
        th = rng.uniform(0.0, 2.0 * np.pi, size=int(m))
        rr = r + noise * rng.standard_normal(int(m))
        pts.append(np.stack([rr * np.cos(th), rr * np.sin(th)], axis=1))
        lab.append(np.full(int(m), c, dtype=np.int32))
    return _finish(rng, np.concatenate(pts), np.concatenate(lab))


def two_moons(n=45000, noise=0.05, seed=6):
    """Two interleaved half circles in 2-D (the classic two-moons shape):
    upper (cos t, sin t), lower (1 - cos t, 1/2 - sin t), t ~ U[0, pi],
    plus N(0, noise^2) on each coordinate."""
    rng = np.random.default_rng(seed)
    sizes = split_equal(n, 2)
    pts, lab = [], []
    for c, m in enumerate(sizes):
        t = rng.uniform(0.0, np.pi, size=int(m))
        if c == 0:
            p = np.stack([np.cos(t), np.sin(t)], axis=1)
        else:
            p = np.stack([1.0 - np.cos(t), 0.5 - np.sin(t)], axis=1)
        pts.append(p + noise * rng.standard_normal(p.shape))
        lab.append(np.full(int(m), c, dtype=np.int32))
    return _finish(rng, np.concatenate(pts), np.concatenate(lab))


def blobs_dirichlet(n=50000, d=16, k=10, centre_var=25.0, std=1.0,
                    alpha=5.0, seed=3):
    """Blobs with centres N(0, centre_var I) and Dirichlet(alpha) sizes."""
    rng = np.random.default_rng(seed)
    centres = np.sqrt(centre_var) * rng.standard_normal((k, d))
    sizes = split_dirichlet(rng, n, k, alpha)
    pts, lab = _gaussian_clusters(rng, centres, sizes, std)
    X, y = _finish(rng, pts, lab)
    return X, y, rng


def blobs_equal(n=200000, d=64, k=20, centre_var=16.0, std=1.0, seed=4):
    """Blobs with centres N(0, centre_var I) and equal sizes."""
    rng = np.random.default_rng(seed)
    centres = np.sqrt(centre_var) * rng.standard_normal((k, d))
    sizes = split_equal(n, k)
    pts, lab = _gaussian_clusters(rng, centres, sizes, std)
    return _finish(rng, pts, lab)


def median_pair_distance_sigma(rng, X, sample=1000) -> np.float32:
    """Median Euclidean distance over all pairs of a sample of `sample`
    points drawn without replacement, computed in float64 from the float32
    points and rounded once to float32."""
    n = X.shape[0]
    idx = rng.choice(n, size=min(sample, n), replace=False)
    P = X[idx].astype(np.float64)
    iu, ju = np.triu_indices(P.shape[0], k=1)
    diff = P[iu] - P[ju]
    dist = np.sqrt(np.einsum("ij,ij->i", diff, diff))
    return np.float32(np.median(dist))


def knn_graph(X: np.ndarray, knn: int = 32, sigma: float = 1.0,
              workers: int = -1):
    """Symmetric kNN input graph in fp32 CSR.

    Exact kNN of every point (self excluded), symmetrised by union; the
    edge weight is exp(-|x_i - x_j|^2 / (2 sigma^2)) evaluated in float64 on
    the float32 points and rounded once to float32.  Rows are sorted by
    column.  Returns (row_ptr int64 [n+1], col int32 [nnz], val fp32 [nnz]).
    """
    from scipy.spatial import cKDTree
    import scipy.sparse as sp
    n = X.shape[0]
    P = X.astype(np.float64)
    tree = cKDTree(P)
    dist, nb = tree.query(P, k=knn + 1, workers=workers)
    rows, cols = [], []
    # drop the point itself; keep the knn nearest others
    own = nb == np.arange(n)[:, None]
    keep = ~own
    # rows where self was not returned (exact duplicates) keep the first knn
    cnt = keep.sum(axis=1)
    over = np.where(cnt > knn)[0]
    for i in over:
        kk = np.where(keep[i])[0]
        keep[i, kk[knn:]] = False
    rows = np.repeat(np.arange(n, dtype=np.int64), knn)
    cols = nb[keep].astype(np.int64)
    assert cols.shape[0] == n * knn
    diff = P[rows] - P[cols]
    w = np.exp(-np.einsum("ij,ij->i", diff, diff) / (2.0 * sigma * sigma))
    K = sp.coo_matrix((w, (rows, cols)), shape=(n, n)).tocsr()
    S = K.maximum(K.T).tocsr()
    S.sort_indices()
    row_ptr = S.indptr.astype(np.int64)
    col = S.indices.astype(np.int32)
    val = S.data.astype(np.float32)
    return row_ptr, col, val


def random_kout_graph(m: int, k: int, seed: int):
    """A CSR graph of m nodes with exactly k stored entries per row.

    Row i holds k columns drawn uniformly from [0, m) with replacement
    (repeats kept, so a row's columns are non-decreasing rather than
    strictly increasing) and sorted, with float32 weights drawn uniformly
    from [0.1, 1).  No locality: a row's neighbours lie anywhere.  Draw
    order: the columns row by row, then the weights.  Returns
    (row_ptr int64 [m+1], col int32 [m k], val float32 [m k]).
    """
    rng = np.random.default_rng(seed)
    col = np.sort(rng.integers(0, m, size=(m, k), dtype=np.int64), axis=1)
    val = rng.uniform(0.1, 1.0, size=m * k).astype(np.float32)
    row_ptr = np.arange(m + 1, dtype=np.int64) * k
    return row_ptr, col.reshape(-1).astype(np.int32), val


# name -> (builder, description); builders take (seed, n_override)
def _c1(seed, n):
    n = n or 1000
    X, y = blobs_uniform_centres(n=n, d=2, k=3, box=10.0, std=1.0, seed=seed)
    return Workload("blobs2d", X, y, np.float32(1.0), 1e-5 / n, 3,
                    "converge", 1000, "dense", seed)


def _c2(seed, n):
    n = n or 10000
    X, y = rings(n=n, seed=seed)
    return Workload("rings2d", X, y, np.float32(0.3), 1e-5 / n, 3,
                    "converge", 1000, "dense", seed)


def _c3(seed, n):
    n = n or 50000
    X, y, rng = blobs_dirichlet(n=n, d=16, k=10, seed=seed)
    sigma = median_pair_distance_sigma(rng, X, 1000)
    return Workload("blobs16d", X, y, sigma, 1e-5 / n, 10,
                    "fixed", 50, "dense", seed)


def _c4(seed, n):
    n = n or 200000
    X, y = blobs_equal(n=n, d=64, k=20, seed=seed)
    return Workload("blobs64d", X, y, np.float32(4.0), 1e-5 / n, 20,
                    "fixed", 30, "fused", seed)


def _moons(seed, n):
    n = n or 45000
    X, y = two_moons(n=n, seed=seed)
    return Workload("moons", X, y, np.float32(1.0), 1e-5 / n, 2,
                    "converge", 3, "cosine", seed)


def _circles3(seed, n):
    n = n or 45000
    X, y = rings(n=n, radii=(1.0, 2.0, 3.0), noise=0.05, seed=seed)
    return Workload("circles3", X, y, np.float32(1.0), 1e-5 / n, 3,
                    "converge", 3, "cosine", seed)


def _c5(seed, n, cache_dir=None):
    n = n or 2000000
    k = 50
    X, y = blobs_equal(n=n, d=8, k=k, seed=seed)
    rp = col = val = None
    path = None
    if cache_dir:
        path = os.path.join(cache_dir, f"knn8d_n{n}_s{seed}.npz")
        if os.path.exists(path):
            z = np.load(path)
            if z["sha_X"].item() == sha256_of(X):
                rp, col, val = z["row_ptr"], z["col"], z["val"]
    if rp is None:
        rp, col, val = knn_graph(X, knn=32, sigma=1.0)
        if path:
            os.makedirs(cache_dir, exist_ok=True)
            np.savez(path, row_ptr=rp, col=col, val=val,
                     sha_X=np.array(sha256_of(X)))
    return Workload("knn8d", X, y, np.float32(1.0), 1e-5 / n, k,
                    "converge", 1000, "csr", seed, rp, col, val)


def relabel_rcm(w: Workload) -> Workload:
    """The same graph and points with nodes renumbered by reverse
    Cuthill-McKee (scipy), so that neighbours get nearby numbers.  Point i of
    the result is point perm[i] of the input; rows stay sorted by column."""
    import scipy.sparse as sp
    from scipy.sparse.csgraph import reverse_cuthill_mckee
    S = sp.csr_matrix((w.val, w.col, w.row_ptr), shape=(w.n, w.n))
    perm = reverse_cuthill_mckee(S, symmetric_mode=True)
    P = S[perm][:, perm].tocsr()
    P.sort_indices()
    return Workload(w.name + "_rcm", np.ascontiguousarray(w.X[perm]),
                    np.ascontiguousarray(w.y_true[perm]), w.sigma, w.eps, w.k,
                    w.mode, w.max_iter, w.path, w.seed, P.indptr.astype(np.int64),
                    P.indices.astype(np.int32), P.data.astype(np.float32))


def _c5_rcm(seed, n, cache_dir=None):
    return relabel_rcm(_c5(seed, n, cache_dir))


WORKLOADS = {
    # n=1,000, d=2, 3 blobs (centres U[-10,10]^2), sigma 1, to convergence
    "blobs2d": (_c1, 1),
    # n=10,000, d=2, rings r=1,3,5 (noise 0.1), sigma 0.3, to convergence
    "rings2d": (_c2, 2),
    # n=50,000, d=16, 10 Dirichlet(5) blobs, sigma = median pair distance;
    # dense W of 2.5e9 entries, T = 50 (and to convergence)
    "blobs16d": (_c3, 3),
    # n=200,000, d=64, 20 equal blobs, sigma 4, fused operator, T = 30
    "blobs64d": (_c4, 4),
    # n=2,000,000, d=8, 50 blobs, 32-NN union graph, CSR, to convergence
    "knn8d": (_c5, 5),
    # the same graph with nodes renumbered by reverse Cuthill-McKee
    "knn8d_rcm": (_c5_rcm, 5),
    # the paper's Experiment I shapes: n=45,000 (15k, 30k via n=), d=2,
    # cosine affinity, at most 3 updates, eps = 1e-5/n, dense W
    "moons": (_moons, 6),
    "circles3": (_circles3, 7),
}


def make(name: str, seed: Optional[int] = None, n: Optional[int] = None,
         cache_dir: Optional[str] = None) -> Workload:
    """Build a named workload; `n` shrinks it for quick parity cases."""
    fn, default_seed = WORKLOADS[name]
    s = default_seed if seed is None else seed
    if name in ("knn8d", "knn8d_rcm"):
        return fn(s, n, cache_dir)
    return fn(s, n)
