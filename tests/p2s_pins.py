"""Pins for the point-to-surface oracle (Kaolin Sec. 2.5: point-to-surface loss
for meshes).  Each pin takes an oracle module and raises AssertionError on a
disagreement with hand-worked values, the optimality certificate of the
closest point (the projection onto a convex set), brute force, exact ties,
invariances or exact finite differences."""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _fr(p):
    return float(Fraction(p[0], p[1]))


def _golden():
    with open(os.path.join(GOLDEN, "p2s_example.json")) as f:
        return json.load(f)


def pin_hand_worked(orc):
    g = _golden()
    a, b, c = (np.array(v, np.float32) for v in g["triangle"])
    for case in g["cases"]:
        d2, w = orc.point_triangle([case["p"]], [a], [b], [c])
        assert abs(d2[0] - _fr(case["d2"])) <= 1e-15, (case["region"], d2[0])
        assert np.allclose(w[0], [_fr(x) for x in case["w"]], rtol=0, atol=1e-15), (case["region"], w[0])


def _random_pairs(rng, n, scale=1.0):
    p = rng.normal(0, scale, (n, 3)).astype(np.float32)
    tri = rng.normal(0, scale, (n, 3, 3)).astype(np.float32)
    return p, tri[:, 0], tri[:, 1], tri[:, 2]


def pin_projection_certificate(orc, n=4000):
    # q = sum w_i v_i is the closest point of the triangle T to p iff q lies in
    # T and (p - q) . (x - q) <= 0 for every x in T; the second condition is
    # linear in x, so checking the three vertices suffices.  With d2 = |p - q|^2
    # this certifies both the distance and the barycentric coordinates.
    rng = np.random.default_rng(11)
    for scale, flat in ((1.0, False), (1.0, True), (1e-3, False), (50.0, False)):
        p, a, b, c = _random_pairs(rng, n, scale)
        if flat:  # points near the plane of the triangle, inside and out
            p = (a + rng.uniform(-0.5, 1.5, (n, 1)) * (b - a) + rng.uniform(-0.5, 1.5, (n, 1)) * (c - a)
                 + rng.normal(0, 1e-3 * scale, (n, 3))).astype(np.float32)
        d2, w = orc.point_triangle(p, a, b, c)
        V = np.stack([a, b, c], 1).astype(np.float64)
        q = np.einsum("ni,nij->nj", w, V)
        P = p.astype(np.float64)
        tol = 1e-12 * scale * scale
        assert np.all(w >= -1e-12) and np.allclose(w.sum(1), 1.0, rtol=0, atol=1e-12)
        for i in range(3):
            assert np.all(np.einsum("nj,nj->n", P - q, V[:, i] - q) <= 1e-9 * scale * scale)
        assert np.allclose(d2, ((P - q) ** 2).sum(1), rtol=1e-9, atol=tol)


def pin_brute_force_grid(orc, n=40, k=300):
    # Minimum over a dense barycentric grid: never below the oracle, and at
    # most the grid's spacing away.
    rng = np.random.default_rng(12)
    p, a, b, c = _random_pairs(rng, n)
    d2, _ = orc.point_triangle(p, a, b, c)
    s, t = np.meshgrid(np.arange(k + 1) / k, np.arange(k + 1) / k, indexing="ij")
    keep = (s + t) <= 1.0
    s, t = s[keep], t[keep]
    for m in range(n):
        A, Bv, C = (x[m].astype(np.float64) for x in (a, b, c))
        pts = A + s[:, None] * (Bv - A) + t[:, None] * (C - A)
        g = ((pts - p[m].astype(np.float64)) ** 2).sum(1).min()
        h = (np.linalg.norm(Bv - A) + np.linalg.norm(C - A)) / k
        assert d2[m] <= g + 1e-12, (m, d2[m], g)
        assert g <= (np.sqrt(d2[m]) + h) ** 2 + 1e-12, (m, d2[m], g)


def pin_degenerate_triangles(orc):
    # Collinear vertices: the distance to the segment; coincident: to the point.
    d2, w = orc.point_triangle([[0.5, 1, 0], [3, 0, 0]], [[0, 0, 0]] * 2, [[1, 0, 0]] * 2,
                               [[2, 0, 0]] * 2)
    assert np.allclose(d2, [1.0, 1.0], rtol=0, atol=1e-15), d2
    d2, w = orc.point_triangle([[1, 2, 2]], [[0, 0, 0]], [[0, 0, 0]], [[0, 0, 0]])
    assert abs(d2[0] - 9.0) <= 1e-15 and abs(w[0].sum() - 1.0) <= 1e-15


def pin_mesh_argmin_and_ties(orc):
    g = _golden()["tie"]
    V = np.array([g["V"]], np.float32)
    F = np.array([g["F"]], np.int32)
    P = np.array([[g["p"]]], np.float32)
    for order in ([0, 1], [1, 0]):
        dist, fidx, _ = orc.p2s_forward(P, V, F[:, order])
        assert dist[0, 0] == _fr(g["d2"]) and fidx[0, 0] == 0, (order, dist, fidx)
    # A small random mesh: the face choice equals the lowest-index minimum of
    # the per-face distances, and the reported w are that face's.
    P, V, F = synth.p2s_workload(2, 300, level=1, seed=13)
    dist, fidx, w = orc.p2s_forward(P, V, F)
    for b in range(2):
        tri = V[b][F[b]]
        for s in range(0, 300, 7):
            n = len(F[b])
            d2, ww = orc.point_triangle(np.repeat(P[b, s:s + 1], n, 0), tri[:, 0], tri[:, 1], tri[:, 2])
            j = int(np.argmin(d2))
            assert fidx[b, s] == j and dist[b, s] == d2[j] and np.array_equal(w[b, s], ww[j])


def pin_invariances(orc):
    rng = np.random.default_rng(14)
    p, a, b, c = _random_pairs(rng, 500)
    d2, w = orc.point_triangle(p, a, b, c)
    # Cyclic order of the vertices: same distance, rotated coordinates.
    d2r, wr = orc.point_triangle(p, b, c, a)
    assert np.allclose(d2r, d2, rtol=1e-12, atol=1e-15) and np.allclose(wr, w[:, [1, 2, 0]], atol=1e-9)
    # Scaling by 4: distances by 16 (exact in binary floating point).
    d2s, ws = orc.point_triangle(4 * p, 4 * a, 4 * b, 4 * c)
    assert np.array_equal(d2s, 16 * d2) and np.array_equal(ws, w)
    # Translation by a dyadic offset on a coarse grid (exact in float32).
    q = lambda x: np.round(x * 64) / 64  # noqa: E731
    p, a, b, c = (q(x).astype(np.float32) for x in (p, a, b, c))
    d2, _ = orc.point_triangle(p, a, b, c)
    off = np.array([3.5, -1.25, 0.75], np.float32)
    d2t, _ = orc.point_triangle(p + off, a + off, b + off, c + off)
    assert np.allclose(d2t, d2, rtol=1e-12, atol=1e-14)


def pin_gradient_exact_differences(orc):
    # Within one region the squared distance is a quadratic polynomial of the
    # coordinates, so a central difference is exact.  Points and vertices on a
    # 1/64 grid, step 2^-12: every input stays exact in float32.
    P, V, F = synth.p2s_workload(1, 60, level=1, seed=15)
    V = (np.round(V * 64) / 64).astype(np.float32)
    P = (np.round(P * 64) / 64).astype(np.float32)
    g = np.linspace(0.5, 1.5, P.shape[1])[None]
    dist, fidx, _ = orc.p2s_forward(P, V, F)
    gP, gV, _, _ = orc.p2s_backward(P, V, F, fidx, g)
    h = 2.0 ** -12

    def loss(Pm, Vm):
        # Distances to the same faces (the face choice is not differentiated).
        tri = Vm[0][F[0][fidx[0]]]
        d2, _ = orc.point_triangle(Pm[0], tri[:, 0], tri[:, 1], tri[:, 2])
        return float((g[0] * d2).sum())

    checked = 0
    for s in range(P.shape[1]):
        for i in range(3):
            Pp, Pm = P.copy(), P.copy()
            Pp[0, s, i] += h
            Pm[0, s, i] -= h
            fd = (loss(Pp, V) - loss(Pm, V)) / (2 * h)
            if abs(fd - gP[0, s, i]) <= 1e-9 * (1 + abs(fd)):
                checked += 1
    assert checked >= 0.9 * 3 * P.shape[1], checked      # region changes are rare
    # In the vertices the distance is rational, not quadratic: a step of 2^-20
    # (still exact in float32 on this grid) leaves an O(h^2) error far below
    # the tolerance, and the double cancellation error is about 1e-10.
    hv = 2.0 ** -20
    used = np.unique(F[0][fidx[0]])
    ok = 0
    for v in used[:40]:
        for i in range(3):
            Vp, Vm = V.copy(), V.copy()
            Vp[0, v, i] += hv
            Vm[0, v, i] -= hv
            fd = (loss(P, Vp) - loss(P, Vm)) / (2 * hv)
            ok += abs(fd - gV[0, v, i]) <= 1e-6 * (1 + abs(fd))
    assert ok >= 0.9 * 3 * min(40, len(used)), ok


def pin_on_surface_points(orc):
    # Points sampled on the mesh itself (dyadic barycentrics on a dyadic mesh)
    # are at distance 0 up to rounding, and gradients vanish with them.
    P, V, F = synth.p2s_workload(1, 10, level=2, seed=16)
    V = (np.round(V * 256) / 256).astype(np.float32)
    rng = np.random.default_rng(17)
    f = rng.integers(0, F.shape[1], 500)
    wts = np.array([[0.25, 0.25, 0.5], [0.5, 0.25, 0.25], [0.125, 0.375, 0.5]])[rng.integers(0, 3, 500)]
    Pq = np.einsum("nk,nkj->nj", wts, V[0][F[0][f]].astype(np.float64))[None].astype(np.float32)
    dist, fidx, _ = orc.p2s_forward(Pq, V, F)
    assert np.all(dist <= 1e-12), dist.max()


ALL_PINS = [pin_hand_worked, pin_projection_certificate, pin_brute_force_grid,
            pin_degenerate_triangles, pin_mesh_argmin_and_ties, pin_invariances,
            pin_gradient_exact_differences, pin_on_surface_points]
