"""Pins for the mesh-sampling oracle (Kaolin Sec. 2.1: differentiable surface
sampling with the reparameterization trick).  Each pin takes an oracle module
and raises AssertionError on a disagreement with a hand-worked value, a closed
form, a statistical property of the uniform surface measure, or an identity."""
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
    with open(os.path.join(GOLDEN, "mesh_sampling_example.json")) as f:
        return json.load(f)


def pin_hand_worked(orc):
    g = _golden()
    V = np.array([g["V"]], np.float32)
    F = np.array([g["F"]], np.int32)
    ar = orc.face_areas(V, F)[0]
    assert np.allclose(ar, [_fr(a) for a in g["areas"]], rtol=0, atol=1e-15), ar
    fidx = np.array([[s["face"] for s in g["samples"]]], np.int32)
    r1 = np.array([[s["r1"] for s in g["samples"]]], np.float32)
    r2 = np.array([[s["r2"] for s in g["samples"]]], np.float32)
    P = orc.sample_points(V, F, fidx, r1, r2)[0]
    want = np.array([[_fr(c) for c in s["p"]] for s in g["samples"]])
    assert np.allclose(P, want, rtol=0, atol=1e-15), (P, want)
    fc = g["face_choice"]
    got = orc.sample_faces(V, F, np.array([fc["u"]], np.float32))[0]
    assert list(got) == fc["face"], got
    bw = g["backward"]
    gP = np.zeros((1, 3, 3))
    gP[0, 0] = bw["gP"]
    gV, _, nV = orc.sample_backward(V, F, fidx, r1, r2, gP)
    want = np.array([[_fr(c) for c in v] for v in bw["gV"]])
    assert np.allclose(gV[0, :3], want, rtol=0, atol=1e-15), gV[0]
    assert np.all(gV[0, 3:] == 0) and list(nV[0]) == [2, 2, 2, 1, 1, 1]


def pin_vertices_at_corner_uniforms(orc):
    # r1 = 0 gives vertex a; r1 = 1 gives b when r2 = 0 and c when r2 = 1 (closed form).
    V, F = synth.triangle_soup(2, 5, 3)
    fidx = np.array([[0, 1, 2], [4, 3, 2]], np.int32)
    r1 = np.array([[0, 1, 1], [0, 1, 1]], np.float32)
    r2 = np.array([[0.3, 0, 1], [0.9, 0, 1]], np.float32)
    P = orc.sample_points(V, F, fidx, r1, r2)
    for b in range(2):
        for s, corner in enumerate((0, 1, 2)):
            v = V[b, F[b, fidx[b, s], corner]]
            assert np.array_equal(P[b, s], v.astype(np.float64)), (b, s, P[b, s], v)


def pin_area_closed_forms(orc):
    # Right triangle with legs a, b has area ab/2; collinear points have area 0;
    # scaling by 2^k multiplies areas by 4^k.
    V = np.array([[[0, 0, 0], [3, 0, 0], [0, 4, 0], [1, 1, 1], [2, 2, 2], [5, 5, 5]]], np.float32)
    F = np.array([[[0, 1, 2], [3, 4, 5], [0, 2, 1]]], np.int32)
    ar = orc.face_areas(V, F)[0]
    assert ar[0] == 6.0 and ar[1] == 0.0 and ar[2] == 6.0, ar
    V2, F2 = synth.grid_mesh(1, 6, 4)
    a1 = orc.face_areas(V2, F2)
    a2 = orc.face_areas(V2 * np.float32(4), F2)
    assert np.allclose(a2, 16 * a1, rtol=1e-14, atol=0)


def pin_face_choice_rules(orc):
    # The zero-area face is never chosen; the choice is the first face whose
    # cumulative area exceeds u * total (strict).
    V = np.array([[[0, 0, 0], [1, 0, 0], [0, 1, 0], [2, 2, 2], [3, 3, 3], [4, 4, 4],
                   [0, 0, 0], [4, 0, 0], [0, 1, 0]]], np.float32)
    F = np.array([[[0, 1, 2], [3, 4, 5], [6, 7, 8]]], np.int32)  # areas 1/2, 0, 2
    u = np.array([[0.0, 0.19, 0.2, 0.5, 0.999]], np.float32)
    got = orc.sample_faces(V, F, u)[0]
    # total 5/2: u*5/2 < 1/2 iff u < 0.2 (0.2 in float32 is just above 0.2).
    assert list(got) == [0, 0, 2, 2, 2], got
    # Exactly on a boundary: areas 1/2, 0, 3/2 and u = 1/4 give u*total = 1/2 =
    # cdf_0 = cdf_1, so the strict rule skips faces 0 and 1 and picks face 2.
    V = np.array([[[0, 0, 0], [1, 0, 0], [0, 1, 0], [1, 1, 1], [2, 2, 2], [3, 3, 3],
                   [0, 0, 0], [3, 0, 0], [0, 1, 0]]], np.float32)
    got = orc.sample_faces(V, F, np.array([[0.25, 0.2499999, 0.0]], np.float32))[0]
    assert list(got) == [2, 0, 0], got


def pin_statistics(orc, S=200000):
    # Empirical face frequencies match area fractions and the mean of the
    # samples on a face is its centroid (uniform measure), both within 5 sigma.
    V, F = synth.triangle_soup(1, 20, 7)
    u, r1, r2 = synth.uniforms(1, S, 8)
    fidx = orc.sample_faces(V, F, u)[0]
    ar = orc.face_areas(V, F)[0]
    p = ar / ar.sum()
    cnt = np.bincount(fidx, minlength=20)
    sig = np.sqrt(S * p * (1 - p))
    assert np.all(np.abs(cnt - S * p) <= 5 * sig + 1), (cnt, S * p)
    P = orc.sample_points(V, F, fidx[None], r1, r2)[0]
    for f in range(20):
        sel = fidx == f
        if sel.sum() < 1000:
            continue
        tri = V[0, F[0, f]].astype(np.float64)
        cen = tri.mean(0)
        spread = np.sqrt(((tri - cen) ** 2).sum(1).max())
        err = np.abs(P[sel].mean(0) - cen)
        assert np.all(err <= 5 * spread / np.sqrt(sel.sum())), (f, err, spread)
        # Every sample lies in the triangle's plane, inside its bounding box.
        assert np.all(P[sel] >= tri.min(0) - 1e-12) and np.all(P[sel] <= tri.max(0) + 1e-12)


def pin_adjoint_identity(orc):
    # P is linear in V, so <gP, P(V + D) - P(V)> = <gV, D> for any D (D dyadic
    # and small so V + D is exact in float32).
    V, F = synth.grid_mesh(2, 7, 9)
    u, r1, r2 = synth.uniforms(2, 3000, 10)
    fidx = orc.sample_faces(V, F, u)
    rng = np.random.default_rng(11)
    gP = rng.standard_normal((2, 3000, 3))
    gV, sV, nV = orc.sample_backward(V, F, fidx, r1, r2, gP)
    D = (rng.integers(-8, 9, V.shape) / 1024.0).astype(np.float32)
    lhs = (gP * (orc.sample_points(V + D, F, fidx, r1, r2) - orc.sample_points(V, F, fidx, r1, r2))).sum()
    rhs = (gV * D.astype(np.float64)).sum()
    assert abs(lhs - rhs) <= 1e-10 * (np.abs(gP).sum() + 1.0), (lhs, rhs)
    assert nV.sum() == 2 * 3000 * 3


def pin_translation_equivariance(orc):
    # Vertices on a 2^-10 grid and a dyadic shift keep V + t exact in float32,
    # so the areas (hence the face choice) are unchanged and P moves by t.
    V, F = synth.triangle_soup(2, 30, 12)
    V = (np.round(V * 1024.0) / 1024.0).astype(np.float32)
    u, r1, r2 = synth.uniforms(2, 500, 13)
    fidx = orc.sample_faces(V, F, u)
    t = np.array([0.25, -0.5, 1.0], np.float32)
    assert np.array_equal(orc.sample_faces(V + t, F, u), fidx)
    P0 = orc.sample_points(V, F, fidx, r1, r2)
    P1 = orc.sample_points(V + t, F, fidx, r1, r2)
    assert np.allclose(P1 - P0, t.astype(np.float64), rtol=0, atol=1e-12)


ALL_PINS = [
    pin_hand_worked,
    pin_vertices_at_corner_uniforms,
    pin_area_closed_forms,
    pin_face_choice_rules,
    pin_statistics,
    pin_adjoint_identity,
    pin_translation_equivariance,
]
