"""Seeded sweep of random shapes through the whole Chamfer path on the GPU.

Each case draws (kind, B, N, M) from a fixed seed, so the list is the same on
every run: ragged tails in both clouds, one to several query groups, target
splits of one and two block sizes, local and bounded fixed-point shifts and
chunked senders in the backward.  Per case: forward bitwise against the
oracle's fused evaluation, the Chamfer value and F-score against the oracle
formulas, cd_metrics against cd_reduce / cd_fscore bitwise, the backward
within the exact-sum bound, and a repeat of the backward bitwise.
"""
import numpy as np
import pytest
import torch

import gpu_checks as gc
import oracle
import paper_1911_05063_amd as cd
import synth

pytestmark = pytest.mark.gpu

KINDS = ("uniform", "sphere", "mesh", "gmm", "grid_dup")


def _cases(seed=2024):
    """24 shapes log-uniform in [1, 40000] (mostly small and ragged), 16 with
    both clouds in [2000, 40000] (several query groups and target blocks,
    senders beyond one pass), at most 3e8 pairs each, two launches long
    enough for the small final target blocks, and four with B a multiple of 8."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < 40:
        kind = KINDS[rng.integers(len(KINDS))]
        B = int(rng.integers(1, 5))
        if len(out) < 24:
            N = int(np.exp(rng.uniform(0, np.log(40000))))
            M = int(np.exp(rng.uniform(0, np.log(40000))))
        else:
            N, M = (int(v) for v in rng.integers(2000, 40001, 2))
        if B * N * M <= 3.0e8:
            out.append((kind, B, N, M, int(rng.integers(1 << 30))))
    # Launches of one to a few rounds: large target blocks, then small ones.
    out += [("mesh", 4, 8192, 16384, 77), ("gmm", 2, 16385, 30000, 78)]
    # B a multiple of 8 (the merge gives XCD x the items b = x mod 8), ragged
    # clouds of several merge blocks, direct and bucketed backward.
    out += [("uniform", 8, 2500, 777, 79), ("grid_dup", 16, 1300, 3001, 80),
            ("sphere", 24, 600, 259, 81), ("gmm", 8, 20000, 20001, 82)]
    return out


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-B{c[1]}-N{c[2]}-M{c[3]}")
def test_random_shape_whole_path(case):
    kind, B, N, M, seed = case
    print(f"[sweep] {kind} B={B} N={N} M={M} seed={seed}", flush=True)
    X, Y = synth.generate(kind, B, N, M, seed)
    Xg, Yg = gc.to_gpu(X), gc.to_gpu(Y)
    dxy, ixy, dyx, iyx = cd.nn_distance(Xg, Yg)
    g = tuple(gc.to_np(t) for t in (dxy, ixy, dyx, iyx))
    ref = oracle.nn(X, Y, fused=True)
    gc.assert_nn_bitwise(g, ref, f"{kind} B={B} N={N} M={M}")

    taus = (0.005, 0.05)
    ch, f, p, r = cd.metrics(dxy, dyx, taus=taus)
    gc.assert_chamfer(gc.to_np(ch), g[0], g[2])
    ch2 = cd.chamfer_reduce(dxy, dyx)
    assert torch.equal(ch, ch2)
    for k, tau in enumerate(taus):
        f1, p1, r1 = cd.f_score(dxy, dyx, tau)
        assert torch.equal(f[k], f1) and torch.equal(p[k], p1) and torch.equal(r[k], r1)
        gc.assert_fscore(gc.to_np(f1), gc.to_np(p1), gc.to_np(r1), g[0], g[2], tau)

    go = np.random.default_rng(seed + 1).uniform(0.5, 1.5, B).astype(np.float32)
    gX, gY = cd.chamfer_backward(gc.to_gpu(go), Xg, Yg, ixy, iyx)
    gX2, gY2 = cd.chamfer_backward(gc.to_gpu(go), Xg, Yg, ixy, iyx)
    assert torch.equal(gX, gX2) and torch.equal(gY, gY2)
    gc.assert_grad_exact_sums(gc.to_np(gX), gc.to_np(gY), X, Y, g[1], g[3], go)
