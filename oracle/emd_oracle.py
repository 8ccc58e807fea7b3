"""CPU oracle for the approximate Earth-mover's distance -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU baseline may
use it; it shares no code with the HIP library.

Kaolin Sec. 2.5 names, beside the Chamfer distance, an approximate form of the
Earth-mover's distance among its point-cloud metrics, citing Fan et al. (2017),
whose EMD is the optimal transport cost between the two sets with Euclidean
ground distance.  Reading taken here: the transport problem with uniform masses
a_i = 1/N, b_j = 1/M,

    EMD(X, Y) = min over couplings P with row sums a and column sums b
                of  sum_ij P_ij C_ij,      C_ij = |x_i - y_j|  (Euclidean),

approximated by entropic regularisation (Cuturi 2013) solved with log-domain
Sinkhorn iterations, each of which touches all N*M pairs (quadratic work, as
opposed to the cubic cost of an exact assignment).  The iteration uses an
explicit geometric schedule of the regularisation eps, warm-starting the
potentials from one value to the next:

    eps_t = eps_start * (eps_end / eps_start) ** (t / (n_iters - 1)),  t = 0..n_iters-1
    f_i  <- -eps_t * log sum_j b_j exp((g_j - C_ij) / eps_t)
    g_j  <- -eps_t * log sum_i a_i exp((f_i - C_ij) / eps_t)

starting from g = 0.  With eps = eps_end, the plan is
P_ij = a_i b_j exp((f_i + g_j - C_ij) / eps) (its column sums are exactly b after
the last g-update) and the reported value is the transport cost sum_ij P_ij C_ij.

Backward: the plan is held fixed (the envelope gradient of the regularised
problem), so d cost / d x_i = sum_j P_ij (x_i - y_j) / C_ij and
d cost / d y_j = -sum_i P_ij (x_i - y_j) / C_ij (0 where C_ij = 0).

Everything in float64 from the float32 inputs; dense N x M matrices, so meant
for the sizes the tests use.
"""
from __future__ import annotations

import numpy as np

__all__ = ["schedule", "sinkhorn", "sinkhorn_step", "plan", "cost_matrix", "backward"]


def schedule(eps_start: float, eps_end: float, n_iters: int) -> np.ndarray:
    """The regularisation of every iteration (geometric from eps_start to eps_end)."""
    if n_iters < 1 or not (eps_start > 0 and eps_end > 0):
        raise ValueError("need n_iters >= 1 and positive eps")
    if n_iters == 1:
        return np.array([float(eps_end)])
    t = np.arange(n_iters) / (n_iters - 1)
    return float(eps_start) * (float(eps_end) / float(eps_start)) ** t


def cost_matrix(x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """C_ij = |x_i - y_j| in float64 for one item."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    return np.sqrt(((x[:, None, :] - y[None, :, :]) ** 2).sum(-1))


def _lse(z: np.ndarray, axis: int) -> np.ndarray:
    m = z.max(axis=axis, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=axis, keepdims=True))).squeeze(axis)


def sinkhorn(X, Y, eps_start: float, eps_end: float, n_iters: int):
    """(cost [B], f [B, N], g [B, M]) after the scheduled iterations."""
    X = np.asarray(X, np.float32)
    Y = np.asarray(Y, np.float32)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    eps = schedule(eps_start, eps_end, n_iters)
    la, lb = -np.log(N), -np.log(M)
    cost = np.empty(B)
    F = np.empty((B, N))
    G = np.empty((B, M))
    for b in range(B):
        C = cost_matrix(X[b], Y[b])
        f = np.zeros(N)
        g = np.zeros(M)
        for e in eps:
            f = -e * _lse((g[None, :] - C) / e + lb, axis=1)
            g = -e * _lse((f[:, None] - C) / e + la, axis=0)
        P = plan(f, g, C, eps[-1])
        cost[b] = (P * C).sum()
        F[b], G[b] = f, g
    return cost, F, G


def sinkhorn_step(X, Y, G, eps: float):
    """One iteration (the f-update, then the g-update) from given potentials
    G [B, M] at regularisation eps: (F_new [B, N], G_new [B, M])."""
    X = np.asarray(X, np.float32)
    Y = np.asarray(Y, np.float32)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    F = np.empty((B, N))
    Gn = np.empty((B, M))
    for b in range(B):
        C = cost_matrix(X[b], Y[b])
        F[b] = -eps * _lse((np.asarray(G[b], np.float64)[None, :] - C) / eps - np.log(M), axis=1)
        Gn[b] = -eps * _lse((F[b][:, None] - C) / eps - np.log(N), axis=0)
    return F, Gn


def plan(f, g, C, eps):
    """P_ij = a_i b_j exp((f_i + g_j - C_ij) / eps), uniform masses."""
    N, M = C.shape
    return np.exp((np.asarray(f)[:, None] + np.asarray(g)[None, :] - C) / eps) / (N * M)


def backward(X, Y, F, G, eps, grad_out):
    """(gX [B, N, 3], gY [B, M, 3]) of sum_b grad_out[b] * cost[b] with the
    plan of (F, G, eps) held fixed."""
    X = np.asarray(X, np.float32)
    Y = np.asarray(Y, np.float32)
    B = X.shape[0]
    gX = np.empty(X.shape)
    gY = np.empty(Y.shape)
    for b in range(B):
        x = X[b].astype(np.float64)
        y = Y[b].astype(np.float64)
        C = cost_matrix(x, y)
        P = plan(F[b], G[b], C, eps)
        W = np.divide(P, C, out=np.zeros_like(P), where=C > 0)
        diff = x[:, None, :] - y[None, :, :]
        gX[b] = grad_out[b] * (W[..., None] * diff).sum(1)
        gY[b] = -grad_out[b] * (W[..., None] * diff).sum(0)
    return gX, gY
