"""Float64 brute-force checker -- TEST INFRASTRUCTURE ONLY.

An implementation of the same definitions as ``cd_oracle.c`` written
independently in NumPy float64 (inputs are promoted exactly).  It pins the
float32 oracle (near-tie classification, finite differences, F-score band)
and is never used by the product path.

Squared distance: sum over axes of (p - q)^2 in float64.
"""
from __future__ import annotations

import numpy as np


def _as64(a) -> np.ndarray:
    a = np.asarray(a)
    if a.ndim != 3 or a.shape[2] != 3:
        raise ValueError(f"expected a [B, N, 3] cloud, got shape {a.shape}")
    return a.astype(np.float64)


def sq_dist_matrix(p, q) -> np.ndarray:
    """[n, m] float64 squared distances between rows of p [n,3] and q [m,3]."""
    p = np.asarray(p, np.float64)
    q = np.asarray(q, np.float64)
    diff = p[:, None, :] - q[None, :, :]
    return np.einsum("nmc,nmc->nm", diff, diff)


def best_two(P, Q, chunk: int = 512):
    """Per query: (d1, i1, d2) in float64.

    d1 is the smallest distance to any target, i1 the lowest index attaining
    it, d2 the smallest distance over the remaining targets (equal to d1 when
    the minimum is attained twice; +inf when there is a single target).
    """
    P, Q = _as64(P), _as64(Q)
    B, NP, NQ = P.shape[0], P.shape[1], Q.shape[1]
    d1 = np.empty((B, NP))
    d2 = np.empty((B, NP))
    i1 = np.empty((B, NP), np.int64)
    for b in range(B):
        for s in range(0, NP, chunk):
            D = sq_dist_matrix(P[b, s:s + chunk], Q[b])
            a = np.argmin(D, axis=1)  # first occurrence = lowest index
            rows = np.arange(D.shape[0])
            d1[b, s:s + chunk] = D[rows, a]
            i1[b, s:s + chunk] = a
            if NQ > 1:
                D[rows, a] = np.inf
                d2[b, s:s + chunk] = D.min(axis=1)
            else:
                d2[b, s:s + chunk] = np.inf
    return d1, i1, d2


def nn_min64(P, Q, chunk: int = 512) -> np.ndarray:
    """Float64 nearest-neighbour squared distance of every query [B, NP]."""
    P, Q = _as64(P), _as64(Q)
    out = np.empty(P.shape[:2])
    for b in range(P.shape[0]):
        for s in range(0, P.shape[1], chunk):
            out[b, s:s + chunk] = sq_dist_matrix(P[b, s:s + chunk], Q[b]).min(axis=1)
    return out


def chamfer64(X, Y, w1: float = 1.0, w2: float = 1.0) -> np.ndarray:
    """Per-item Chamfer distance, every step in float64."""
    return w1 * nn_min64(X, Y).mean(axis=1) + w2 * nn_min64(Y, X).mean(axis=1)


def near_tie_mask(d1, d2, rel: float = 1e-6) -> np.ndarray:
    """Queries whose best two distinct-index distances differ by at most rel*d2
    but are not exactly equal: there the argmin is decided by rounding."""
    d1 = np.asarray(d1)
    d2 = np.asarray(d2)
    return (d2 - d1 <= rel * d2) & (d1 != d2)


def index_ok(P, Q, idx, d1, i1, d2, rel: float = 1e-6) -> np.ndarray:
    """Per query: is `idx` an acceptable nearest neighbour?

    Must equal the float64 lowest-index argmin, except at near-ties (see
    near_tie_mask), where any target within rel of the minimum is accepted.
    """
    P, Q = _as64(P), _as64(Q)
    idx = np.asarray(idx, np.int64)
    ok = idx == i1
    loose = near_tie_mask(d1, d2, rel) & ~ok
    if loose.any():
        b, i = np.nonzero(loose)
        j = idx[b, i]
        valid = (j >= 0) & (j < Q.shape[1])
        jj = np.where(valid, j, 0)
        d = ((P[b, i] - Q[b, jj]) ** 2).sum(axis=1)
        ok[b, i] = valid & (d <= d1[b, i] * (1.0 + rel))
    return ok


def fscore_bracket(d1_xy, d1_yx, tau: float, rel: float = 1e-6):
    """F-score@tau bounds from float64 distances.

    Points whose float64 distance lies within rel*tau of tau are "band" points:
    rounding of the float32 squared distance may put them on either side.
    Returns (F_lo, F_hi) per item, counting band points as misses / hits.
    """
    t = float(tau)
    r_xy = np.sqrt(np.asarray(d1_xy, np.float64))
    r_yx = np.sqrt(np.asarray(d1_yx, np.float64))

    def counts(r):
        band = np.abs(r - t) <= rel * t
        sure = (r < t) & ~band
        return sure.sum(axis=1), (sure | band).sum(axis=1)

    lo_p, hi_p = counts(r_xy)
    lo_r, hi_r = counts(r_yx)
    N, M = r_xy.shape[1], r_yx.shape[1]

    def f(cp, cr):
        P = cp / N
        R = cr / M
        with np.errstate(invalid="ignore", divide="ignore"):
            return np.where(P + R > 0, 2 * P * R / np.where(P + R > 0, P + R, 1), 0.0)

    return f(lo_p, lo_r), f(hi_p, hi_r)


def backward64(grad_out, X, Y, idx_xy, idx_yx, w1: float = 1.0, w2: float = 1.0):
    """Float64 gradient of sum_b grad_out[b] * chamfer[b] for fixed neighbours,
    written with np.add.at scatters (independent of the C oracle's loops)."""
    X, Y = _as64(X), _as64(Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    go = np.asarray(grad_out, np.float64).reshape(B, 1, 1)
    gX = np.zeros_like(X)
    gY = np.zeros_like(Y)
    for b in range(B):
        jx = np.asarray(idx_xy[b], np.int64)
        iy = np.asarray(idx_yx[b], np.int64)
        txy = 2.0 * go[b] * (w1 / N) * (X[b] - Y[b, jx])
        tyx = 2.0 * go[b] * (w2 / M) * (Y[b] - X[b, iy])
        gX[b] += txy
        np.add.at(gY[b], jx, -txy)
        gY[b] += tyx
        np.add.at(gX[b], iy, -tyx)
    return gX, gY
