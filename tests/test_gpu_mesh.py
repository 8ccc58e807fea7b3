"""GPU parity of differentiable mesh surface sampling (Kaolin Sec. 2.1) against
the mesh oracle, and of the mesh -> samples -> Chamfer -> vertex-gradient chain."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
import gpu_checks as gc

pytestmark = pytest.mark.gpu
U32 = 2.0 ** -24


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no ROCm GPU visible")
    import paper_1911_05063_amd as cd
    assert os.path.exists(cd.LIB_PATH), "libcd_hip.so missing: build before running GPU tests"
    yield


import paper_1911_05063_amd as cd  # noqa: E402


def _faces_valid(V, F, u, fidx_gpu, band=1e-5):
    """Every GPU face choice equals the oracle's, or the target lies within
    band * total of the GPU face's interval of the float64 cumulative areas."""
    ref = oracle.sample_faces(V, F, u)
    bad = np.argwhere(fidx_gpu != ref)
    if len(bad) == 0:
        return 0
    ar = oracle.face_areas(V, F)
    cdf = np.cumsum(ar, axis=1)
    for b, s in bad:
        f = int(fidx_gpu[b, s])
        tot = cdf[b, -1]
        t = float(u[b, s]) * tot
        lo = cdf[b, f - 1] if f > 0 else 0.0
        assert 0 <= f < F.shape[1] and lo - band * tot <= t <= cdf[b, f] + band * tot, (b, s, f, ref[b, s])
    return len(bad)


def _points_close(P_gpu, V, F, fidx, r1, r2):
    ref = oracle.sample_points(V, F, fidx, r1, r2)
    # Bound: a few float32 roundings of each weighted term plus the sqrt.
    Vb = V.astype(np.float64)
    scale = np.zeros_like(ref)
    for b in range(V.shape[0]):
        tri = Vb[b][F[b][fidx[b]]]          # [S, 3 vertices, 3]
        scale[b] = np.abs(tri).sum(axis=1)
    assert np.all(np.abs(P_gpu - ref) <= 8 * U32 * scale + 1e-30), np.max(np.abs(P_gpu - ref) / (scale + 1e-30))


def _abs_grad_sums(nv, F, fidx, gP):
    """G [B, nv, 3]: per vertex and component, the sum of |gP| over the samples
    whose face holds the vertex (a vertex repeated in a face counts each time)."""
    G = np.zeros((F.shape[0], nv, 3))
    for b in range(F.shape[0]):
        ok = (fidx[b] >= 0) & (fidx[b] < F.shape[1])
        for i in range(3):
            np.add.at(G[b], F[b, fidx[b][ok], i], np.abs(gP[b][ok].astype(np.float64)))
    return G


def _backward_close(gV, V, F, fidx, r1, r2, gP):
    """The backward's bound: the sums are exact; what remains is the float32
    weights (1 - sqrt(r1) can cancel: absolute error a few 2^-24, times |gP|),
    the float32 product and one rounding at the end."""
    rV, _, _ = oracle.sample_backward(V, F, fidx, r1, r2, gP)
    G = _abs_grad_sums(V.shape[1], F, fidx, gP)
    tol = 6 * U32 * G + 2 * U32 * np.abs(rV)
    assert np.all(np.abs(gV - rV) <= tol + 1e-30), np.max(np.abs(gV - rV) - tol)


# Cases span one and several sample chunks per item, one and several vertex
# slices (grid 70: 4900 vertices), ragged last chunks, S = 1 and S = 0, and the
# backward's chunk sizes: 512 samples (most cases), 1024 (grid 10), 2048 (soup
# 40 x 20) held in registers, and 2560 (520 items: one chunk each) in the loop.
@pytest.mark.parametrize("maker,B,n,S", [("soup", 3, 200, 5000), ("grid", 2, 40, 7000),
                                         ("soup", 1, 1, 100), ("grid", 4, 3, 1),
                                         ("grid", 1, 70, 40001), ("soup", 2, 1500, 3333),
                                         ("soup", 2, 5, 0), ("grid", 1, 10, 200000),
                                         ("soup", 40, 20, 12000), ("soup", 520, 10, 2100)])
def test_sampling_matches_oracle(maker, B, n, S):
    V, F = synth.triangle_soup(B, n, 61) if maker == "soup" else synth.grid_mesh(B, n, 62)
    u, r1, r2 = synth.uniforms(B, S, 63)
    print(f"[case] sampling {maker} B={B} n={n} S={S}", flush=True)
    Vg, Fg = gc.to_gpu(V), gc.to_gpu(F)
    fidx = gc.to_np(cd.mesh_sample_faces(Vg, Fg, gc.to_gpu(u)))
    _faces_valid(V, F, u, fidx)
    P = gc.to_np(cd.mesh_sample_points(Vg, Fg, gc.to_gpu(fidx), gc.to_gpu(r1), gc.to_gpu(r2)))
    _points_close(P, V, F, fidx, r1, r2)
    rng = np.random.default_rng(64)
    gP = rng.standard_normal((B, S, 3)).astype(np.float32)
    gV = gc.to_np(cd.mesh_sample_backward(V.shape[1], Fg, gc.to_gpu(fidx), gc.to_gpu(r1),
                                          gc.to_gpu(r2), gc.to_gpu(gP)))
    _backward_close(gV, V, F, fidx, r1, r2, gP)


def test_sampling_hand_worked_example(golden_dir):
    with open(os.path.join(golden_dir, "mesh_sampling_example.json")) as f:
        g = json.load(f)
    V = np.array([g["V"]], np.float32)
    F = np.array([g["F"]], np.int32)
    fidx = np.array([[s["face"] for s in g["samples"]]], np.int32)
    r1 = np.array([[s["r1"] for s in g["samples"]]], np.float32)
    r2 = np.array([[s["r2"] for s in g["samples"]]], np.float32)
    P = gc.to_np(cd.mesh_sample_points(gc.to_gpu(V), gc.to_gpu(F), gc.to_gpu(fidx), gc.to_gpu(r1),
                                       gc.to_gpu(r2)))
    want = np.array([[float(c[0]) / c[1] for c in s["p"]] for s in g["samples"]], np.float32)
    assert np.array_equal(P[0], want)  # all values dyadic: exact in float32
    fc = g["face_choice"]
    got = gc.to_np(cd.mesh_sample_faces(gc.to_gpu(V), gc.to_gpu(F), gc.to_gpu(np.array([fc["u"]], np.float32))))
    assert list(got[0]) == fc["face"]


def test_degenerate_meshes():
    # All-zero-area mesh: no face can be chosen (-1) and its samples are NaN;
    # a face with an out-of-range vertex has area 0 and is never chosen.
    V = np.array([[[0, 0, 0], [1, 1, 1], [2, 2, 2]], [[0, 0, 0], [1, 0, 0], [0, 1, 0]]], np.float32)
    F = np.array([[[0, 1, 2], [0, 2, 1]], [[0, 1, 7], [0, 1, 2]]], np.int32)
    u = np.array([[0.1, 0.9], [0.0, 0.99]], np.float32)
    fidx = gc.to_np(cd.mesh_sample_faces(gc.to_gpu(V), gc.to_gpu(F), gc.to_gpu(u)))
    assert fidx.tolist() == [[-1, -1], [1, 1]]
    r = np.full((2, 2), 0.5, np.float32)
    P = gc.to_np(cd.mesh_sample_points(gc.to_gpu(V), gc.to_gpu(F), gc.to_gpu(fidx), gc.to_gpu(r), gc.to_gpu(r)))
    assert np.all(np.isnan(P[0])) and np.all(np.isfinite(P[1]))
    gV = gc.to_np(cd.mesh_sample_backward(3, gc.to_gpu(F), gc.to_gpu(fidx), gc.to_gpu(r), gc.to_gpu(r),
                                          gc.to_gpu(np.ones((2, 2, 3), np.float32))))
    assert np.all(gV[0] == 0) and np.all(np.isfinite(gV[1]))
    assert np.allclose(gV[1].sum(axis=0), 2.0, rtol=1e-6)  # weights sum to 1 per sample


def test_mesh_to_chamfer_chain_gradient():
    # Mesh reconstruction loss: sample the predicted mesh, Chamfer against a
    # target cloud, backward to the vertices -- against the oracles chained on
    # the GPU's own samples and neighbours.
    B, S = 3, 3000
    V, F = synth.triangle_soup(B, 50, 71)
    _, Y = synth.generate("mesh", B, 10, 2500, 72)
    u, r1, r2 = synth.uniforms(B, S, 73)
    Vg = gc.to_gpu(V).requires_grad_(True)
    Fg = gc.to_gpu(F)
    fidx = cd.mesh_sample_faces(Vg.detach(), Fg, gc.to_gpu(u))
    P = cd.MeshSample.apply(Vg, Fg, fidx, gc.to_gpu(r1), gc.to_gpu(r2))
    loss = cd.chamfer_distance(P, gc.to_gpu(Y)).sum()
    loss.backward()
    Pn = gc.to_np(P.detach())
    dxy, ixy, dyx, iyx = oracle.nn(Pn, Y, fused=True)
    gP, _, _, _, _, _ = oracle.backward(np.ones(B), Pn, Y, ixy, iyx)
    rV, sV, nV = oracle.sample_backward(V, F, gc.to_np(fidx), r1, r2, gP)
    gV = gc.to_np(Vg.grad)
    # gP itself carries float32 rounding from the GPU backward (1e-4 relative
    # plus reordering), which the linear map to the vertices propagates; the
    # float32 weights add a few 2^-24 times |gP| (as in _backward_close).
    tol = 2e-4 * np.abs(rV) + 1e-4 * sV + 6 * U32 * _abs_grad_sums(V.shape[1], F, gc.to_np(fidx), gP) + 1e-12
    assert np.all(np.abs(gV - rV) <= tol), np.max(np.abs(gV - rV) - tol)


def test_full_size_mesh_sampling():
    # The mesh workload's shape: 16 soups of 200 triangles, 16384 samples each.
    B, S = 16, 16384
    V, F = synth.triangle_soup(B, 200, 3)
    u, r1, r2 = synth.uniforms(B, S, 4)
    Vg, Fg = gc.to_gpu(V), gc.to_gpu(F)
    fidx = gc.to_np(cd.mesh_sample_faces(Vg, Fg, gc.to_gpu(u)))
    nbad = _faces_valid(V, F, u, fidx)
    assert nbad <= 10
    P = gc.to_np(cd.mesh_sample_points(Vg, Fg, gc.to_gpu(fidx), gc.to_gpu(r1), gc.to_gpu(r2)))
    _points_close(P, V, F, fidx, r1, r2)
    rng = np.random.default_rng(5)
    gP = rng.standard_normal((B, S, 3)).astype(np.float32)
    gV = gc.to_np(cd.mesh_sample_backward(V.shape[1], Fg, gc.to_gpu(fidx), gc.to_gpu(r1),
                                          gc.to_gpu(r2), gc.to_gpu(gP)))
    _backward_close(gV, V, F, fidx, r1, r2, gP)


@pytest.mark.parametrize("n", [900, 3000, 6000])
def test_zero_area_faces_never_chosen_and_reproducible(n):
    # 900, 3000 and 6000 faces (one face per scan thread, up to four kept in
    # registers, several stashed between the scan's passes), every third one
    # invalid (a vertex index out of range) and every third one degenerate (a
    # repeated vertex): no sample may land on either, and the face choice and
    # the backward are bitwise reproducible.
    B, S = 2, 50000
    V, F = synth.triangle_soup(B, n, 81)
    F = F.copy()
    F[:, 0::3, 2] = 3 * n + 5
    F[:, 1::3, 2] = F[:, 1::3, 0]
    u, r1, r2 = synth.uniforms(B, S, 82)
    u[:, :64] = np.linspace(0.0, 1.0, 64, endpoint=False, dtype=np.float32)
    Vg, Fg = gc.to_gpu(V), gc.to_gpu(F)
    fidx = gc.to_np(cd.mesh_sample_faces(Vg, Fg, gc.to_gpu(u)))
    assert np.all(fidx % 3 == 2), np.unique(fidx % 3)
    assert np.array_equal(fidx, gc.to_np(cd.mesh_sample_faces(Vg, Fg, gc.to_gpu(u))))
    # The oracle takes only in-range indices: give it the invalid faces as
    # zero-area ones, which the library treats the same way.
    F_or = F.copy()
    F_or[:, 0::3] = 0
    _faces_valid(V, F_or, u, fidx)
    gP = np.random.default_rng(83).standard_normal((B, S, 3)).astype(np.float32)
    args = (V.shape[1], Fg, gc.to_gpu(fidx), gc.to_gpu(r1), gc.to_gpu(r2), gc.to_gpu(gP))
    g1 = gc.to_np(cd.mesh_sample_backward(*args))
    g2 = gc.to_np(cd.mesh_sample_backward(*args))
    assert np.array_equal(g1, g2)
    _backward_close(g1, V, F_or, fidx, r1, r2, gP)
