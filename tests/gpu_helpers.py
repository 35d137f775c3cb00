"""Shared helpers for the GPU parity tests (comparison metrics only)."""
import numpy as np
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


def stop_margin(stats, eps, t_star) -> float:
    """min over t in {t*-1, t*} (0-based update indices) of |s_t - eps| / eps."""
    ts = [t for t in (t_star - 2, t_star - 1) if 0 <= t < len(stats)]
    return float(min(abs(stats[t] - eps) / eps for t in ts))


def affinity_tolerance(X, sigma, A_ref, gram: bool):
    """Per-entry bound on |A_gpu - A_ref| from the arithmetic of each engine.

    Direct differences (VALU engine): each squared distance carries a
    relative error of a few float32 ulps, (d + 4) eps32 dist2.

    Gram form (matrix-core engine), u = 2^-24, over the centred points
    x = float32(x_raw - mean) (each centred coordinate rounded once: the
    difference x_i - x_j is off by at most u (|x_ik| + |x_jk|) per
    coordinate, which adds at most 4 u (|x_i|^2 + |x_j|^2) to dist2 for
    the distances that matter here), M = max |x|:
      * every coordinate is scaled into [-1, 1] by 2^-S (2^S <= 2M) and
        split into half-precision parts hi + lo, which carry it to within
        max(2^-22 |x|, 2^-25 2^S) <= 2^-22 |x| + u M;
      * three of the four part products are summed (lo.lo, at most
        2^-22 |x_ik||x_jk|, is dropped); part products are exact in
        float32, so per pair of points the dot product is off by at most
        12 u sum_k |x_ik||x_jk| + u M (|x_i|_1 + |x_j|_1) from the parts;
      * the float32 accumulation of 3d products and the start value
        -|x_j|^2 / 2 adds at most 3d u (|x_i||x_j| + |x_j|^2 / 2);
      * rounding |x_j|^2 / 2, c |x_i|^2 and the final multiply-add adds
        u (|x_i|^2 + |x_j|^2 + dist2).
    With 2 |x_i||x_j| <= |x_i|^2 + |x_j|^2 this gives, in dist2,
      u [(6d + 20)(|x_i|^2 + |x_j|^2) + 2 M (|x_i|_1 + |x_j|_1)].
    Either engine: an error e in dist2 moves A = exp(-dist2 / (2 sigma^2))
    by A e / (2 sigma^2); the float32 coefficient c, exp2 and the final
    rounding add 4 eps32 dist2 and a few ulps of A.
    """
    X64 = np.asarray(X, dtype=np.float64)
    d = X64.shape[1]
    s2 = 2.0 * float(sigma) ** 2
    nrm = (X64 * X64).sum(1)
    with np.errstate(divide="ignore"):
        dist2 = -np.log(np.where(A_ref > 0, A_ref, 1.0)) * s2
    if gram:
        u = EPS32 / 2
        Xc = (X64 - X64.mean(0)).astype(np.float32).astype(np.float64)
        nrmc = (Xc * Xc).sum(1)
        l1 = np.abs(Xc).sum(1)
        M = float(np.abs(Xc).max())
        e = u * ((6 * d + 20) * (nrmc[:, None] + nrmc[None, :])
                 + 2 * M * (l1[:, None] + l1[None, :]))
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
