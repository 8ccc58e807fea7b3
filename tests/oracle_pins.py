"""Pins that tie the CPU oracle to facts fixed outside itself.

Each ``pin_*`` function takes an oracle module (the real one, or a mutant
built by the mutation test) and raises AssertionError when the oracle
disagrees with a hand-worked value, a closed form, an invariant, float64
brute force or float64 finite differences.  The definitions they hold the
oracle to are those of Kaolin Sec. 2.5 (Chamfer distance for point clouds)
under the readings recorded in the design notes.
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import synth
from oracle import check64

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U32 = 2.0 ** -24


def _frac(pair):
    return float(Fraction(pair[0], pair[1]))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- hand-worked
def pin_worked_example(orc):
    g = _load("worked_example.json")
    X = np.array([g["X"]], np.float32)
    Y = np.array([g["Y"]], np.float32)
    for fused in (False, True):
        dxy, ixy, dyx, iyx = orc.nn(X, Y, fused)
        assert np.array_equal(dxy[0], np.array(g["dist_xy"], np.float32)), (fused, dxy)
        assert np.array_equal(ixy[0], g["idx_xy"]), (fused, ixy)
        assert np.array_equal(dyx[0], np.array(g["dist_yx"], np.float32)), (fused, dyx)
        assert np.array_equal(iyx[0], g["idx_yx"]), (fused, iyx)
    cd = orc.chamfer(dxy, dyx)
    assert abs(cd[0] - _frac(g["chamfer"])) < 1e-15, cd
    gX, gY, *_ = orc.backward([1.0], X, Y, ixy, iyx)
    refX = np.array([[_frac(c) for c in p] for p in g["gX"]])
    refY = np.array([[_frac(c) for c in p] for p in g["gY"]])
    assert np.allclose(gX[0], refX, rtol=0, atol=1e-15), gX
    assert np.allclose(gY[0], refY, rtol=0, atol=1e-15), gY
    fs = g["fscore"]
    f, p, r, _, _ = orc.fscore(dxy, dyx, fs["tau"])
    assert abs(p[0] - _frac(fs["precision"])) < 1e-15, p
    assert abs(r[0] - _frac(fs["recall"])) < 1e-15, r
    assert abs(f[0] - _frac(fs["f"])) < 1e-15, f


def pin_tie_lowest_index(orc):
    g = _load("tie_example.json")
    X = np.array([g["X"]], np.float32)
    for case in g["cases"]:
        Y = np.array([case["Y"]], np.float32)
        for fused in (False, True):
            d, i = orc.nn_one_way(X, Y, fused)
            assert i[0, 0] == case["idx_xy"], (case, fused, i)
            assert d[0, 0] == case["dist_xy"], (case, fused, d)


def pin_fscore_strict_threshold(orc):
    # A point exactly at distance tau is not a match (strict d < tau^2): here
    # d = 0.25 = 0.5^2 exactly, so P = R = 0 and F = 0; just above, F = 1.
    X = np.zeros((1, 1, 3), np.float32)
    Y = np.array([[[0.5, 0.0, 0.0]]], np.float32)
    dxy, _, dyx, _ = orc.nn(X, Y)
    f, p, r, cp, cr = orc.fscore(dxy, dyx, 0.5)
    assert cp[0] == 0 and cr[0] == 0 and f[0] == 0.0, (f, cp, cr)
    f, *_ = orc.fscore(dxy, dyx, np.nextafter(np.float32(0.5), np.float32(1)))
    assert f[0] == 1.0, f
    # Unequal counts: P = 2/4, R = 1/2 -> F = 1/2;  P = 1/4, R = 1/2 -> F = 1/3.
    X = np.array([[[0, 0, 0], [0.25, 0, 0], [4, 0, 0], [8, 0, 0]]], np.float32)
    Y = np.array([[[0, 0, 0], [6, 0, 0]]], np.float32)
    dxy, _, dyx, _ = orc.nn(X, Y)
    f, p, r, *_ = orc.fscore(dxy, dyx, 1.0)
    assert p[0] == 0.5 and r[0] == 0.5 and f[0] == 0.5, (f, p, r)
    f, p, r, *_ = orc.fscore(dxy, dyx, 0.25)
    assert p[0] == 0.25 and r[0] == 0.5 and abs(f[0] - 1.0 / 3.0) < 1e-15, (f, p, r)


# ---------------------------------------------------------------- closed forms
def pin_single_pair_closed_form(orc):
    # N = M = 1: both directions see the same pair, so
    # chamfer = (w1 + w2) |x - y|^2 and gX = 2 g (w1 + w2)(x - y) = -gY.
    rng = np.random.default_rng(11)
    for _ in range(8):
        x = rng.integers(-64, 65, (1, 1, 3)) / 32.0
        y = rng.integers(-64, 65, (1, 1, 3)) / 32.0
        X, Y = x.astype(np.float32), y.astype(np.float32)
        w1, w2 = float(rng.integers(1, 5)), float(rng.integers(1, 5)) / 2
        go = float(rng.integers(-3, 4))
        dxy, ixy, dyx, iyx = orc.nn(X, Y)
        d = float(((x - y) ** 2).sum())
        assert dxy[0, 0] == d and dyx[0, 0] == d and ixy[0, 0] == 0 and iyx[0, 0] == 0
        assert orc.chamfer(dxy, dyx, w1, w2)[0] == (w1 + w2) * d
        gX, gY, *_ = orc.backward([go], X, Y, ixy, iyx, w1, w2)
        assert np.array_equal(gX[0, 0], 2 * go * (w1 + w2) * (x - y)[0, 0]), gX
        assert np.array_equal(gY[0, 0], -2 * go * (w1 + w2) * (x - y)[0, 0]), gY


def pin_lattice_closed_form(orc, B=2, dims=(8, 8, 4), h=1.0 / 16, shift=(1 / 64, -3 / 256, 1 / 128)):
    # Y = permuted (X + s) with |s_k| < h/2: every nearest distance is |s|^2
    # exactly, the neighbour of x_i is y_perm(i), chamfer = 2|s|^2 and
    # gX_i = -2 s (1/N + 1/M), gY_j = +2 s (1/N + 1/M) (all dyadic, exact).
    X, Y, perm = synth.lattice_pair(B, dims, h, shift, seed=5)
    s = np.array(shift)
    s2 = float((s ** 2).sum())
    N = X.shape[1]
    for fused in (False, True):
        dxy, ixy, dyx, iyx = orc.nn(X, Y, fused)
        assert np.all(dxy == s2) and np.all(dyx == s2)
        assert np.array_equal(ixy, perm)
        inv = np.empty_like(perm)
        for b in range(B):
            inv[b, perm[b]] = np.arange(N)
        assert np.array_equal(iyx, inv)
    assert np.all(orc.chamfer(dxy, dyx) == 2 * s2)
    gX, gY, *_ = orc.backward(np.ones(B), X, Y, ixy, iyx)
    k = 2.0 * (1.0 / N + 1.0 / N)
    assert np.array_equal(gX, np.broadcast_to(-k * s, gX.shape))
    assert np.array_equal(gY, np.broadcast_to(k * s, gY.shape))
    tau_in, tau_out = np.sqrt(s2) * 1.01, np.sqrt(s2) * 0.99
    assert np.all(orc.fscore(dxy, dyx, tau_in)[0] == 1.0)
    assert np.all(orc.fscore(dxy, dyx, tau_out)[0] == 0.0)


# ---------------------------------------------------------------- brute force
def _small_clouds(seed):
    out = []
    shapes = [(2, 37, 53), (3, 64, 17), (1, 1, 29), (2, 23, 1), (1, 130, 129)]
    kinds = ["uniform", "sphere", "mesh", "gmm", "grid_dup"]
    for t, (B, N, M) in enumerate(shapes):
        out.append(synth.generate(kinds[t % len(kinds)], B, N, M, seed + t))
    return out


def pin_bruteforce_float64(orc, seed=100):
    # The float32 oracle against float64 brute force: distances within the
    # float32 rounding of five operations, indices exact except at near-ties.
    for X, Y in _small_clouds(seed):
        for fused in (False, True):
            for P, Q in ((X, Y), (Y, X)):
                d, i = orc.nn_one_way(P, Q, fused)
                d1, i1, d2 = check64.best_two(P, Q)
                assert np.all(np.abs(d - d1) <= 8 * U32 * d1), np.max(np.abs(d - d1) / np.maximum(d1, 1e-30))
                ok = check64.index_ok(P, Q, i, d1, i1, d2)
                assert ok.all(), np.argwhere(~ok)[:5]
        dxy, ixy, dyx, iyx = orc.nn(X, Y)
        w1, w2 = 0.75, 1.5
        cd = orc.chamfer(dxy, dyx, w1, w2)
        ref = check64.chamfer64(X, Y, w1, w2)
        assert np.all(np.abs(cd - ref) <= 1e-6 * ref), (cd, ref)


def pin_fscore_bracket(orc, seed=200):
    for X, Y in _small_clouds(seed):
        dxy, _, dyx, _ = orc.nn(X, Y)
        d1xy = check64.nn_min64(X, Y)
        d1yx = check64.nn_min64(Y, X)
        for tau in (0.05, 0.1, 0.3):
            t32 = float(np.float32(tau))
            f, p, r, cp, cr = orc.fscore(dxy, dyx, tau)
            lo, hi = check64.fscore_bracket(d1xy, d1yx, t32)
            assert np.all(f >= lo - 1e-15) and np.all(f <= hi + 1e-15), (f, lo, hi)
            exact = lo == hi  # no point within rounding of the threshold
            assert np.array_equal(cp[exact], (d1xy < t32 * t32).sum(1)[exact])
            assert np.array_equal(cr[exact], (d1yx < t32 * t32).sum(1)[exact])


def pin_finite_differences(orc, seed=300, h=1e-6):
    # Chamfer is locally quadratic while no nearest neighbour changes, so the
    # float64 central difference equals the derivative up to rounding (~1e-9).
    rng = np.random.default_rng(seed)
    checked = total = 0
    for B, N, M in ((1, 5, 7), (2, 9, 4), (1, 16, 16)):
        X = rng.uniform(-1, 1, (B, N, 3)).astype(np.float32)
        Y = rng.uniform(-1, 1, (B, M, 3)).astype(np.float32)
        go = rng.uniform(0.5, 2.0, B)
        w1, w2 = 0.7, 1.3
        dxy, ixy, dyx, iyx = orc.nn(X, Y)
        gX, gY, *_ = orc.backward(go, X, Y, ixy, iyx, w1, w2)
        X64, Y64 = X.astype(np.float64), Y.astype(np.float64)

        def loss(Xp, Yp):
            return float((go * check64.chamfer64(Xp, Yp, w1, w2)).sum())

        def stable(Xp, Yp):
            a = check64.best_two(Xp, Yp)
            c = check64.best_two(Yp, Xp)
            return (np.array_equal(a[1], ixy) and np.array_equal(c[1], iyx)
                    and np.all(a[2] - a[0] > 1e-3) and np.all(c[2] - c[0] > 1e-3))

        for cloud, grad in ((0, gX), (1, gY)):
            base = (X64, Y64)[cloud]
            for idx in np.ndindex(base.shape):
                total += 1
                e = np.zeros_like(base)
                e[idx] = h
                args_p = (X64 + e, Y64) if cloud == 0 else (X64, Y64 + e)
                args_m = (X64 - e, Y64) if cloud == 0 else (X64, Y64 - e)
                if not (stable(*args_p) and stable(*args_m)):
                    continue
                checked += 1
                fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
                assert abs(fd - grad[idx]) <= 1e-7 * max(1.0, abs(grad[idx])), (cloud, idx, fd, grad[idx])
    assert checked >= 0.9 * total, (checked, total)


# ---------------------------------------------------------------- invariants
def pin_invariants(orc, seed=400):
    rng = np.random.default_rng(seed)
    X, Y = synth.generate("mesh", 2, 96, 80, seed)
    # Identity: CD(X, X) = 0, every point its own (first) neighbour.
    d, i = orc.nn_one_way(X, X)
    assert np.all(d == 0) and np.array_equal(i, np.broadcast_to(np.arange(96), i.shape))
    assert np.all(orc.chamfer(d, d) == 0)
    # Symmetry: (x-y)^2 == (y-x)^2 exactly, so the two directions swap bitwise.
    for fused in (False, True):
        a = orc.nn(X, Y, fused)
        b = orc.nn(Y, X, fused)
        assert np.array_equal(a[0], b[2]) and np.array_equal(a[1], b[3])
        assert np.array_equal(a[2], b[0]) and np.array_equal(a[3], b[1])
    dxy, ixy, dyx, iyx = orc.nn(X, Y)
    assert np.array_equal(orc.chamfer(dxy, dyx), orc.chamfer(dyx, dxy))
    # Scaling by 2^k: distances scale by exactly 4^k, indices unchanged,
    # gradients scale by 2^k.
    for k in (-3, 2):
        s = np.float32(2.0 ** k)
        d2 = orc.nn(X * s, Y * s)
        assert np.array_equal(d2[0], dxy * s * s) and np.array_equal(d2[1], ixy)
        assert np.array_equal(d2[2], dyx * s * s) and np.array_equal(d2[3], iyx)
    go = np.array([1.0, -0.5])
    gX, gY, *_ = orc.backward(go, X, Y, ixy, iyx)
    gXs, gYs, *_ = orc.backward(go, X * np.float32(4), Y * np.float32(4), ixy, iyx)
    assert np.allclose(gXs, 4 * gX, rtol=1e-12, atol=0) and np.allclose(gYs, 4 * gY, rtol=1e-12, atol=0)
    # Gradient identities for any consistent argmin: translation invariance
    # (sum of all gradients is 0) and Euler's theorem for the degree-2
    # homogeneous loss (sum x.gX + sum y.gY = 2 sum_b go_b CD_b).
    cd = orc.chamfer(dxy, dyx)
    for b in range(2):
        tot = gX[b].sum(0) + gY[b].sum(0)
        assert np.all(np.abs(tot) <= 1e-12), tot
        eul = (X[b].astype(np.float64) * gX[b]).sum() + (Y[b].astype(np.float64) * gY[b]).sum()
        ref = 2 * go[b] * check64.chamfer64(X[b:b + 1], Y[b:b + 1])[0]
        assert abs(eul - ref) <= 1e-6 * abs(ref), (eul, ref)
        assert abs(cd[b] - ref / (2 * go[b])) <= 1e-6 * abs(cd[b])
    # Permutation: permuting X permutes dist_xy/idx_xy and relabels idx_yx.
    Xg, Yg = synth.generate("uniform", 1, 70, 50, seed + 1)
    dxy, ixy, dyx, iyx = orc.nn(Xg, Yg)
    p = rng.permutation(70)
    q = rng.permutation(50)
    d2 = orc.nn(Xg[:, p], Yg[:, q])
    qinv = np.argsort(q)
    pinv = np.argsort(p)
    assert np.array_equal(d2[0], dxy[:, p]) and np.array_equal(d2[1], qinv[ixy[:, p]])
    assert np.array_equal(d2[2], dyx[:, q]) and np.array_equal(d2[3], pinv[iyx[:, q]])
    # Translation by a dyadic vector on the 1/256 grid: bitwise identical.
    Xq, Yq = synth.generate("grid_dup", 1, 300, 300, seed + 2)
    t = np.array([1 / 256, -5 / 256, 3 / 128], np.float32)
    a = orc.nn(Xq, Yq)
    b = orc.nn(Xq + t, Yq + t)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def pin_duplicates_lowest_index(orc, seed=500):
    # Exact duplicates among the targets: the neighbour must be the first copy.
    X, Y = synth.generate("grid_dup", 2, 200, 150, seed)
    Y = np.concatenate([Y, Y[:, ::-1]], axis=1)  # every target appears twice
    for fused in (False, True):
        d, i = orc.nn_one_way(X, Y, fused)
        d1, i1, d2 = check64.best_two(X, Y)
        assert np.array_equal(i, i1)  # grid distances are exact in float32
        assert np.all(d == d1)


ALL_PINS = [
    pin_worked_example,
    pin_tie_lowest_index,
    pin_fscore_strict_threshold,
    pin_single_pair_closed_form,
    pin_lattice_closed_form,
    pin_bruteforce_float64,
    pin_fscore_bracket,
    pin_finite_differences,
    pin_invariants,
    pin_duplicates_lowest_index,
]
