"""Pins for the approximate-EMD oracle (Kaolin Sec. 2.5: a quadratic
approximation of the Earth-mover's distance for point clouds).  Each pin
takes an oracle module (emd_oracle or a mutated copy) and raises
AssertionError on a disagreement with the exact transport cost (assignment
solver; 1-D sorted matching), a hand-worked case, the marginal constraints,
invariances, or finite differences of the fixed-plan cost."""
from __future__ import annotations

import json
import os

import numpy as np
from scipy.optimize import linear_sum_assignment

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _marginal_gap(orc, X, Y, F, G, eps):
    """Total violation of the row and column sums of the plan, item 0."""
    C = orc.cost_matrix(X[0], Y[0])
    P = orc.plan(F[0], G[0], C, eps)
    N, M = C.shape
    return np.abs(P.sum(1) - 1.0 / N).sum() + np.abs(P.sum(0) - 1.0 / M).sum(), C.max()


def pin_hand_worked(orc):
    with open(os.path.join(GOLDEN, "emd_example.json")) as f:
        g = json.load(f)
    X = np.array([g["X"]], np.float32)
    Y = np.array([g["Y"]], np.float32)
    for eps in (0.05, 0.02):
        cost, F, G = orc.sinkhorn(X, Y, 1.0, eps, 60)
        d = np.sqrt(2.0) - 1.0
        excess = d / (1.0 + np.exp(d / eps))
        assert abs(cost[0] - (1.0 + excess)) <= 1e-9 + 1e-6 * excess, (eps, cost, 1 + excess)


def pin_exact_assignment(orc):
    # N = M: the optimal coupling is a permutation (Birkhoff), so EMD = mean
    # matched distance of the optimal assignment.  The entropic plan's cost
    # lies above it by at most eps (log N + log M), minus whatever the
    # residual marginal gap allows.
    rng = np.random.default_rng(5)
    for N, scale in ((40, 1.0), (25, 10.0)):
        X = rng.normal(0, scale, (1, N, 3)).astype(np.float32)
        Y = rng.normal(0, scale, (1, N, 3)).astype(np.float32)
        C = orc.cost_matrix(X[0], Y[0])
        r, c = linear_sum_assignment(C)
        exact = C[r, c].mean()
        eps = 1e-3 * scale
        cost, F, G = orc.sinkhorn(X, Y, scale, eps, 600)
        gap, cmax = _marginal_gap(orc, X, Y, F, G, eps)
        assert gap < 1e-3, gap
        assert exact - gap * cmax - 1e-9 <= cost[0] <= exact + eps * 2 * np.log(N) + gap * cmax, \
            (cost[0], exact, gap)


def pin_one_dimensional_sorted_matching(orc):
    # On a line the optimal coupling of equal-size uniform sets matches the
    # sorted orders: EMD = mean |x_(k) - y_(k)| (no solver involved).
    rng = np.random.default_rng(6)
    N = 60
    xs = np.sort(rng.uniform(-1, 1, N))
    ys = np.sort(rng.uniform(-1, 1, N) + 0.3)
    X = np.zeros((1, N, 3), np.float32)
    Y = np.zeros((1, N, 3), np.float32)
    X[0, :, 0] = rng.permutation(xs)
    Y[0, :, 0] = rng.permutation(ys)
    exact = np.abs(np.sort(X[0, :, 0].astype(np.float64)) - np.sort(Y[0, :, 0].astype(np.float64))).mean()
    eps = 1e-3
    cost, F, G = orc.sinkhorn(X, Y, 1.0, eps, 800)
    gap, cmax = _marginal_gap(orc, X, Y, F, G, eps)
    assert gap < 0.02, gap          # Sinkhorn converges slowly at small eps
    assert exact - gap * cmax - 1e-9 <= cost[0] <= exact + eps * 2 * np.log(N) + gap * cmax, (cost, exact)


def pin_marginals_unequal_sizes(orc):
    # N != M: column sums exact after the last g-update, row sums converged.
    rng = np.random.default_rng(7)
    X = rng.normal(0, 1, (1, 30, 3)).astype(np.float32)
    Y = rng.normal(0, 1, (1, 45, 3)).astype(np.float32)
    cost, F, G = orc.sinkhorn(X, Y, 1.0, 0.02, 300)
    C = orc.cost_matrix(X[0], Y[0])
    P = orc.plan(F[0], G[0], C, 0.02)
    assert np.allclose(P.sum(0), 1.0 / 45, rtol=0, atol=1e-12)
    assert np.allclose(P.sum(1), 1.0 / 30, rtol=0, atol=1e-3)
    # More iterations at the final eps only shrink the row-marginal error.
    _, F2, G2 = orc.sinkhorn(X, Y, 1.0, 0.02, 1200)
    P2 = orc.plan(F2[0], G2[0], C, 0.02)
    assert np.abs(P2.sum(1) - 1.0 / 30).max() < np.abs(P.sum(1) - 1.0 / 30).max()
    assert abs(P.sum() - 1.0) < 1e-9 and abs((P * C).sum() - cost[0]) < 1e-12


def pin_invariances(orc):
    rng = np.random.default_rng(8)
    X = (np.round(rng.normal(0, 1, (1, 20, 3)) * 64) / 64).astype(np.float32)
    Y = (np.round(rng.normal(0, 1, (1, 30, 3)) * 64) / 64).astype(np.float32)
    base, _, _ = orc.sinkhorn(X, Y, 1.0, 0.05, 80)
    off = np.array([2.5, -0.75, 1.25], np.float32)
    t, _, _ = orc.sinkhorn(X + off, Y + off, 1.0, 0.05, 80)
    assert abs(t[0] - base[0]) <= 1e-9 * base[0], (t, base)
    px = rng.permutation(20)
    py = rng.permutation(30)
    p, _, _ = orc.sinkhorn(X[:, px], Y[:, py], 1.0, 0.05, 80)
    assert abs(p[0] - base[0]) <= 1e-9 * base[0], (p, base)
    # Scaling the clouds and the schedule by 2 scales the cost by 2.
    s, _, _ = orc.sinkhorn(2 * X, 2 * Y, 2.0, 0.1, 80)
    assert abs(s[0] - 2 * base[0]) <= 1e-9 * base[0], (s, base)


def pin_identical_clouds(orc):
    rng = np.random.default_rng(9)
    X = rng.uniform(-1, 1, (1, 50, 3)).astype(np.float32)
    eps = 1e-3
    cost, F, G = orc.sinkhorn(X, X.copy(), 1.0, eps, 500)
    assert 0.0 <= cost[0] <= eps * 2 * np.log(50), cost


def pin_fixed_plan_gradient(orc):
    # d/dX of sum_ij P_ij |x_i - y_j| with P held fixed, by central differences.
    rng = np.random.default_rng(10)
    X = rng.normal(0, 1, (1, 12, 3)).astype(np.float32)
    Y = rng.normal(0, 1, (1, 15, 3)).astype(np.float32)
    eps = 0.05
    _, F, G = orc.sinkhorn(X, Y, 1.0, eps, 100)
    gX, gY = orc.backward(X, Y, F, G, eps, np.array([1.5]))
    x0 = X[0].astype(np.float64)
    y0 = Y[0].astype(np.float64)
    P = orc.plan(F[0], G[0], orc.cost_matrix(x0, y0), eps)
    h = 1e-6
    for arr, grad in ((x0, gX[0]), (y0, gY[0])):
        for i in range(arr.shape[0]):
            for c in range(3):
                keep = arr[i, c]
                arr[i, c] = keep + h
                up = (P * orc.cost_matrix(x0, y0)).sum()
                arr[i, c] = keep - h
                dn = (P * orc.cost_matrix(x0, y0)).sum()
                arr[i, c] = keep
                fd = 1.5 * (up - dn) / (2 * h)
                assert abs(fd - grad[i, c]) <= 1e-6 * (1 + abs(fd)), (i, c, fd, grad[i, c])


def pin_step_composes_to_the_schedule(orc):
    # The one-iteration function, applied along the schedule from g = 0,
    # reproduces the scheduled run.
    rng = np.random.default_rng(11)
    X = rng.normal(0, 1, (2, 9, 3)).astype(np.float32)
    Y = rng.normal(0, 1, (2, 13, 3)).astype(np.float32)
    cost, F, G = orc.sinkhorn(X, Y, 0.7, 0.05, 7)
    g = np.zeros((2, 13))
    for e in orc.schedule(0.7, 0.05, 7):
        f, g = orc.sinkhorn_step(X, Y, g, e)
    assert np.allclose(f, F, rtol=0, atol=1e-12) and np.allclose(g, G, rtol=0, atol=1e-12)


def pin_schedule(orc):
    s = orc.schedule(1.0, 0.01, 3)
    assert np.allclose(s, [1.0, 0.1, 0.01], rtol=1e-15, atol=0)
    assert np.array_equal(orc.schedule(0.5, 0.25, 1), [0.25])


ALL_PINS = [pin_hand_worked, pin_exact_assignment, pin_one_dimensional_sorted_matching,
            pin_marginals_unequal_sizes, pin_invariances, pin_identical_clouds,
            pin_fixed_plan_gradient, pin_step_composes_to_the_schedule, pin_schedule]
