"""Comparison helpers for the GPU parity tests: HIP path vs the CPU oracle.

Bars (per the readings in the design notes):
  * same-precision parity: against the oracle's fused mode (float32,
    fma(dz,dz, fma(dy,dy, dx*dx)), the order the kernel uses) distances and
    indices must be bitwise equal;
  * against the oracle's separately rounded order: distances within 1e-5
    relative; an index may differ only at a near-tie, i.e. where the float64
    best two distinct-index distances differ by at most 1e-6 relative and the
    GPU's choice lies within 1e-6 of the float64 minimum;
  * Chamfer within 1e-5 relative of the float64-accumulated oracle value;
  * F-score counts exact (same float32 distances, exact threshold test);
  * gradients within 1e-4 relative plus the float-atomic reordering bound
    4 n 2^-24 S (n contributions with absolute sum S per component); since
    the scatter sums are exact (fixed point), also within 4 2^-24 S + 2 2^-24
    |g| (each term's float32 rounding plus one final rounding), and bitwise
    equal from run to run.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_1911_05063_amd as cd

U32 = 2.0 ** -24


def to_gpu(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.array(a, copy=True, order="C")).to("cuda:0")


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def gpu_forward(X: np.ndarray, Y: np.ndarray):
    out = cd.nn_distance(to_gpu(X), to_gpu(Y))
    torch.cuda.synchronize()
    return tuple(to_np(t) for t in out)


def assert_nn_bitwise(gpu, ref, what=""):
    names = ("dist_xy", "idx_xy", "dist_yx", "idx_yx")
    # No index is -1 (no neighbour found) for finite inputs within range.
    for n, g in zip(names[1::2], gpu[1::2]):
        assert g.size == 0 or g.min() >= 0, f"{what} {n}: an index is negative"
    for n, g, r in zip(names, gpu, ref):
        if not np.array_equal(g, r):
            bad = np.argwhere(g != r)
            b, i = bad[0]
            raise AssertionError(f"{what} {n}: {len(bad)} mismatches, first at {tuple(bad[0])}: "
                                 f"gpu={g[b, i]!r} oracle={r[b, i]!r}")


def _row_best_two64(p: np.ndarray, Q: np.ndarray):
    d = ((Q.astype(np.float64) - p.astype(np.float64)) ** 2).sum(axis=1)
    i1 = int(np.argmin(d))
    d1 = d[i1]
    d[i1] = np.inf
    d2 = d.min() if len(d) > 1 else np.inf
    return d1, i1, d2


def assert_nn_unfused(P, Q, dist_gpu, idx_gpu, dist_ref, idx_ref, rel_d=1e-5, rel_tie=1e-6):
    """GPU one-way result vs the separately rounded float32 oracle."""
    err = np.abs(dist_gpu.astype(np.float64) - dist_ref)
    assert np.all(err <= rel_d * dist_ref), f"max rel dist err {np.max(err / np.maximum(dist_ref, 1e-38))}"
    zero = dist_ref == 0
    assert np.all(dist_gpu[zero] == 0)
    for b, i in np.argwhere(idx_gpu != idx_ref):
        d1, i1, d2 = _row_best_two64(P[b, i], Q[b])
        j = int(idx_gpu[b, i])
        assert 0 <= j < Q.shape[1]
        dj = float(((Q[b, j].astype(np.float64) - P[b, i].astype(np.float64)) ** 2).sum())
        near = (d2 - d1 <= rel_tie * d2) and d1 != d2
        assert near and dj <= d1 * (1 + rel_tie), (b, i, j, int(idx_ref[b, i]), d1, d2, dj)


def sample_nn(P, Q, rows, fused=True):
    """Oracle nearest neighbours for the sampled query rows (b, i) only."""
    out_d = np.empty(len(rows), np.float32)
    out_i = np.empty(len(rows), np.int32)
    for b in np.unique(rows[:, 0]):
        sel = np.nonzero(rows[:, 0] == b)[0]
        d, i = oracle.nn_one_way(P[b:b + 1, rows[sel, 1]], Q[b:b + 1], fused)
        out_d[sel] = d[0]
        out_i[sel] = i[0]
    return out_d, out_i


def assert_chamfer(cd_gpu, dist_xy, dist_yx, w1=1.0, w2=1.0, rel=1e-5):
    ref = oracle.chamfer(dist_xy, dist_yx, w1, w2)
    err = np.abs(cd_gpu.astype(np.float64) - ref)
    assert np.all(err <= rel * np.abs(ref) + 1e-38), (cd_gpu, ref)
    # A float64 sum rounded once: expect agreement to within one float32 ulp.
    assert np.all(err <= np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)), (cd_gpu, ref)


def assert_fscore(f_gpu, p_gpu, r_gpu, dist_xy, dist_yx, tau):
    f, p, r, _, _ = oracle.fscore(dist_xy, dist_yx, tau)
    assert np.array_equal(p_gpu, p.astype(np.float32)), (p_gpu, p)
    assert np.array_equal(r_gpu, r.astype(np.float32)), (r_gpu, r)
    assert np.array_equal(f_gpu, f.astype(np.float32)), (f_gpu, f)


def assert_grad(gX, gY, X, Y, idx_xy, idx_yx, grad_out, w1=1.0, w2=1.0, rel=1e-4):
    rX, rY, sX, sY, nX, nY = oracle.backward(grad_out, X, Y, idx_xy, idx_yx, w1, w2)
    for name, g, r, s, n in (("gX", gX, rX, sX, nX), ("gY", gY, rY, sY, nY)):
        tol = rel * np.abs(r) + 4.0 * (n[..., None] + 2) * U32 * s
        err = np.abs(g.astype(np.float64) - r)
        if not np.all(err <= tol):
            k = np.unravel_index(np.argmax(err - tol), err.shape)
            raise AssertionError(f"{name} at {k}: gpu={g[k]} ref={r[k]} tol={tol[k]} n={n[k[:2]]}")
    return max(float(np.max(np.abs(gX - rX) / np.maximum(np.abs(rX), 1e-30))),
               float(np.max(np.abs(gY - rY) / np.maximum(np.abs(rY), 1e-30))))


def assert_grad_exact_sums(gX, gY, X, Y, idx_xy, idx_yx, grad_out=None, w1=1.0, w2=1.0,
                           g_xy=None, g_yx=None):
    """The exact-sum bound: every term carries at most a few float32
    roundings (difference, products, the per-item scale), the sum none, the
    result one."""
    if g_xy is None:
        rX, rY, sX, sY, _, _ = oracle.backward(grad_out, X, Y, idx_xy, idx_yx, w1, w2)
    else:
        rX, rY, sX, sY, _, _ = oracle.backward_pointwise(g_xy, g_yx, X, Y, idx_xy, idx_yx)
    for name, g, r, s in (("gX", gX, rX, sX), ("gY", gY, rY, sY)):
        tol = 4 * U32 * s + 2 * U32 * np.abs(r) + 1e-38
        err = np.abs(g.astype(np.float64) - r)
        if not np.all(err <= tol):
            k = np.unravel_index(np.argmax(err - tol), err.shape)
            raise AssertionError(f"{name} at {k}: gpu={g[k]} ref={r[k]} tol={tol[k]}")


def gradient_identities(gX, gY, X, Y, grad_out, chamfer_vals, rel=1e-4):
    """Translation invariance (sum of gradients = 0) and Euler's identity
    (sum x.gX + sum y.gY = 2 sum_b grad_out_b chamfer_b), in float64."""
    X64, Y64 = X.astype(np.float64), Y.astype(np.float64)
    gX64, gY64 = gX.astype(np.float64), gY.astype(np.float64)
    for b in range(X.shape[0]):
        tot = gX64[b].sum(0) + gY64[b].sum(0)
        scale = np.abs(gX64[b]).sum(0) + np.abs(gY64[b]).sum(0)
        assert np.all(np.abs(tot) <= 1e-5 * scale + 1e-30), (b, tot, scale)
        eul = (X64[b] * gX64[b]).sum() + (Y64[b] * gY64[b]).sum()
        ref = 2.0 * float(grad_out[b]) * float(chamfer_vals[b])
        assert abs(eul - ref) <= rel * abs(ref) + 1e-30, (b, eul, ref)
