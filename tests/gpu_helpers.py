"""Shared helpers for the GPU parity tests (comparison metrics only)."""
import numpy as np
import pytest
from scipy.optimize import linear_sum_assignment

EPS32 = float(np.finfo(np.float32).eps)


def rel_l1(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.abs(a - b).sum() / np.abs(b).sum())


def matched_agreement(a, b) -> float:
    """Label agreement after the best one-to-one matching of label ids."""
    a = np.asarray(a)
    b = np.asarray(b)
    ka, kb = a.max() + 1, b.max() + 1
    M = np.zeros((ka, kb))
    np.add.at(M, (a, b), 1)
    r, c = linear_sum_assignment(-M)
    return float(M[r, c].sum() / a.shape[0])


def separation_ok(v_oracle, v_gpu, labels_oracle, factor=100.0) -> bool:
    """Every gap between consecutive clusters of the oracle's sorted v is at
    least `factor` times the largest |v_gpu - v_oracle| (the guard under
    which label agreement is a parity criterion)."""
    v = np.asarray(v_oracle)
    err = float(np.abs(np.asarray(v_gpu) - v).max())
    k = labels_oracle.max() + 1
    lo = np.array([v[labels_oracle == c].min() for c in range(k)])
    hi = np.array([v[labels_oracle == c].max() for c in range(k)])
    gaps = lo[1:] - hi[:-1]
    return bool(np.all(gaps >= factor * err))


# One line per label comparison after the whole path: whether the
# separation guard held.  conftest prints them at the end of the session.
LABEL_GUARD = []


def partition_cost(v, labels, k_eff):
    """Within-cluster sum of squares of a labelling, from its members."""
    return float(sum(((v[labels == c] - v[labels == c].mean()) ** 2).sum()
                     for c in range(k_eff)))


def check_kmeans(v, out, ref):
    """Unique: k_eff and the optimal cost.  The labels must equal the
    oracle's, or (exact cost ties) form an equally optimal partition into
    contiguous runs of the sorted values, numbered by ascending centroid,
    that never splits equal values."""
    assert out.k_eff == ref.k_eff
    assert out.cost == pytest.approx(ref.cost, rel=1e-9, abs=1e-12)
    lab = out.labels.cpu().numpy()
    if np.array_equal(lab, ref.labels):
        np.testing.assert_allclose(out.centroids.cpu().numpy(), ref.centroids,
                                   rtol=1e-10, atol=1e-300)
        return
    order = np.argsort(v, kind="stable")
    ls = lab[order]
    assert np.all(np.diff(ls) >= 0) and set(ls) == set(range(out.k_eff))
    vs = v[order]
    same = vs[1:] == vs[:-1]
    assert np.all(ls[1:][same] == ls[:-1][same])
    assert partition_cost(v, lab, out.k_eff) == pytest.approx(ref.cost, rel=1e-9,
                                                               abs=1e-12)


def check_labels(orc, tag, v_ref, labels_ref, v_gpu, km_gpu, k, expect_separated=False):
    """Label parity after the whole path.

    Under the guard (every gap between the oracle's clusters in sorted v at
    least 100x the largest |v_gpu - v_oracle|) the GPU's labels must agree
    with the oracle's to >= 0.999 after matching.  Where the guard fails
    the labels cannot be compared (rounding may move a point across a gap
    narrower than the vectors' difference): that is recorded as "not
    separated", and the GPU's labels must instead be the exact k-means
    optimum of the GPU's own v (the oracle's k-means on v_gpu), which keeps
    the k-means step pinned either way.  expect_separated makes a failed
    guard an error (for workloads whose clusters are known to separate)."""
    held = separation_ok(v_ref, v_gpu, labels_ref)
    agree = matched_agreement(km_gpu.labels.cpu().numpy(), labels_ref)
    line = (f"{tag}: {'separated' if held else 'not separated'}, "
            f"matched agreement {agree:.6f}")
    LABEL_GUARD.append(line)
    print(f"  labels {line}", flush=True)
    if expect_separated:
        assert held, f"{tag}: clusters expected to separate"
    if held:
        assert agree >= 0.999
    else:
        check_kmeans(np.asarray(v_gpu), km_gpu, orc.kmeans1d(np.asarray(v_gpu), k))


def stop_margin(stats, eps, t_star) -> float:
    """min over t in {t*-1, t*} (0-based update indices) of |s_t - eps| / eps."""
    ts = [t for t in (t_star - 2, t_star - 1) if 0 <= t < len(stats)]
    return float(min(abs(stats[t] - eps) / eps for t in ts))


def gram_centre(X):
    """The centre the matrix-core engine's Gram form works on: per
    coordinate, the lower median (position (m - 1) // 2 in sorted order) of
    the m = min(n, 1024) points at the evenly spaced indices t n // m."""
    X = np.asarray(X, dtype=np.float32)
    n = X.shape[0]
    m = min(n, 1024)
    idx = (np.arange(m, dtype=np.int64) * n) // m
    return np.sort(X[idx].astype(np.float64), axis=0)[(m - 1) // 2]


def affinity_tolerance(X, sigma, A_ref, gram: bool):
    """Per-entry bound on |A_gpu - A_ref| from the arithmetic of each engine.

    Direct differences (VALU engine): each squared distance carries a
    relative error of a few float32 ulps, (d + 4) eps32 dist2.

    Gram form (matrix-core engine), u = 2^-24, over the centred points
    x = float32(x_raw - z), z the centre of `gram_centre` (each centred
    coordinate rounded once: the difference x_i - x_j is off by at most
    u (|x_ik| + |x_jk|) per coordinate, which adds at most
    4 u (|x_i|^2 + |x_j|^2) to dist2), M_p = max_k |x_pk| per point:
      * point p is scaled into [-1, 1] by its own 2^-S_p (2^S_p <= 2 M_p)
        and every coordinate split into half-precision parts hi + lo,
        which carry it to within max(2^-22 |x_pk|, 2^-25 2^S_p)
        <= 2^-22 |x_pk| + u M_p;
      * three of the four part products are summed (lo.lo, at most
        2^-22 |x_ik||x_jk|, is dropped); part products are exact in
        float32, so the dot product is off by at most
        12 u sum_k |x_ik||x_jk| + u (M_j |x_i|_1 + M_i |x_j|_1);
      * the float32 accumulation of 3d products adds at most
        3d u |x_i||x_j|;
      * the two multiply-adds sc_j (mr_i D + gam_j) + cn_i round
        mr_i D + gam_j (at most c (2 |x_i||x_j| + |x_j|^2) 2^-S_j before the
        exact scaling by sc_j) and the result; gam_j and cn_i are rounded
        once each: together u c (3 (|x_i|^2 + |x_j|^2) + dist2).
    With 2 |x_i||x_j| <= |x_i|^2 + |x_j|^2 this stays below, in dist2,
      u [(6d + 24)(|x_i|^2 + |x_j|^2) + 2 (M_j |x_i|_1 + M_i |x_j|_1)]
    plus u dist2 (carried by the exponent term below).  Only the pair's own
    points enter: a point far from the rest widens its own rows and
    columns, no others.
    Either engine: an error e in dist2 moves A = exp(-dist2 / (2 sigma^2))
    by A e / (2 sigma^2); the float32 coefficient c, exp2 and the final
    rounding add 4 eps32 dist2 and a few ulps of A.
    """
    X64 = np.asarray(X, dtype=np.float64)
    d = X64.shape[1]
    s2 = 2.0 * float(sigma) ** 2
    with np.errstate(divide="ignore"):
        dist2 = -np.log(np.where(A_ref > 0, A_ref, 1.0)) * s2
    if gram:
        u = EPS32 / 2
        Xc = (X64 - gram_centre(X)).astype(np.float32).astype(np.float64)
        nrmc = (Xc * Xc).sum(1)
        l1 = np.abs(Xc).sum(1)
        Mp = np.abs(Xc).max(1)
        e = u * ((6 * d + 24) * (nrmc[:, None] + nrmc[None, :])
                 + 2 * (Mp[None, :] * l1[:, None] + Mp[:, None] * l1[None, :]))
    else:
        e = (d + 4) * EPS32 * dist2
    # the exponent itself is formed in float32: c * dist2 rounds once more
    e = e + 4 * EPS32 * dist2
    # float32 underflow: values below the smallest normal may flush to 0
    return A_ref * e / s2 + 8 * EPS32 * A_ref + 2.4e-38


def cosine_tolerance(d):
    """Absolute bound on |A_gpu - A_ref| for the cosine affinity
    max(0, (1 + x_i.x_j rinv_i rinv_j) / 2): the float32 dot product of d
    terms is off by at most d eps32 |x_i| |x_j| (Cauchy-Schwarz), the
    reciprocal norms and the two products add 4 eps32 relative, halving
    keeps that, and the final fused multiply-add rounds once at magnitude
    <= 1; (d + 8) eps32 covers the sum with margin."""
    return (d + 8) * EPS32
