"""CPU oracle for the batched Chamfer distance -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package.  The product path (``paper_1911_05063_amd``) never
imports it, and it never imports the product path: the two share no code.

Two independent implementations live here:

* ``cd_oracle.c`` (loaded through ctypes): the float32 nearest-neighbour
  definition, lowest-index tie-break, float64 sums / F-score / gradients.
  It is the parity reference for the HIP path.
* ``check64`` (NumPy, float64): brute force used to pin the C oracle -- it
  classifies near-ties, supplies the finite-difference gradient reference and
  brackets the F-score against threshold rounding.
* ``mesh_oracle.c``: differentiable surface sampling of triangle meshes
  (Kaolin Sec. 2.1, reparameterization trick): area-weighted face choice,
  reparameterised points and their backward to the vertices, in double.
* ``p2s_oracle.c``: the point-to-surface distance of Kaolin Sec. 2.5 (points
  to the closest face of a triangle mesh), its face choice and its backward
  to the points and vertices, in double.
* ``emd_oracle`` (NumPy, float64): the approximate Earth-mover's distance of
  Kaolin Sec. 2.5 as scheduled log-domain Sinkhorn iterations on the
  Euclidean transport problem, and its fixed-plan backward.

Every function follows Kaolin Sec. 2.5 (Chamfer distance for point clouds,
defined through its citation of Fan et al.) under the readings listed in the
repository's design notes: squared distances, sum of the two directional
means, lowest index on exact ties, F-score with the strict test d < tau^2.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cd_oracle.c")
_MESH_SRC = os.path.join(_HERE, "mesh_oracle.c")
_P2S_SRC = os.path.join(_HERE, "p2s_oracle.c")
# Every C source of the oracle library, in link order.
SOURCES = (_SRC, _MESH_SRC, _P2S_SRC)
LIB_PATH = os.path.join(_HERE, "libcd_oracle.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the C oracle (gcc, no FP contraction, OpenMP) into oracle/libcd_oracle.so."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", *SOURCES, "-o", LIB_PATH + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build()
    lib = ctypes.CDLL(LIB_PATH)
    i64, f32p, f64p = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_nn.argtypes = [i64, i64, i64, f32p, f32p, ctypes.c_int, f32p, f32p]
    lib.oracle_chamfer.argtypes = [i64, i64, i64, f32p, f32p, ctypes.c_double, ctypes.c_double, f64p]
    lib.oracle_fscore.argtypes = [i64, i64, i64, f32p, f32p, ctypes.c_float, f64p, f64p, f64p,
                                  f64p, f64p]
    lib.oracle_backward_pointwise.argtypes = [i64, i64, i64, f64p, f64p, f32p, f32p, f32p, f32p,
                                              f64p, f64p, f64p, f64p, f32p, f32p]
    vp = ctypes.c_void_p
    lib.oracle_face_areas.argtypes = [i64, i64, i64, vp, vp, vp]
    lib.oracle_sample_faces.argtypes = [i64, i64, i64, vp, vp, i64, vp, vp, vp]
    lib.oracle_sample_points.argtypes = [i64, i64, i64, vp, vp, i64, vp, vp, vp, vp]
    lib.oracle_sample_backward.argtypes = [i64, i64, i64, vp, i64, vp, vp, vp, vp, vp, vp, vp]
    lib.oracle_point_triangle_batch.argtypes = [i64, vp, vp, vp, vp, vp, vp]
    lib.oracle_p2s_forward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp]
    lib.oracle_p2s_backward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _cloud(a) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    if a.ndim != 3 or a.shape[2] != 3:
        raise ValueError(f"expected a [B, N, 3] cloud, got shape {a.shape}")
    return a


def threads() -> int:
    """OpenMP threads the oracle's nearest-neighbour loop uses."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Threads for the oracle's later parallel loops (timing only: results do
    not depend on the thread count)."""
    _load().oracle_set_threads(int(n))


def nn_one_way(P, Q, fused: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """For each query p in P[b]: min_j d(p, Q[b, j]) and the lowest j attaining it."""
    P, Q = _cloud(P), _cloud(Q)
    if P.shape[0] != Q.shape[0]:
        raise ValueError("batch sizes differ")
    B, NP, NQ = P.shape[0], P.shape[1], Q.shape[1]
    if NQ < 1:
        raise ValueError("nearest neighbour over an empty target set is undefined")
    dist = np.empty((B, NP), np.float32)
    idx = np.empty((B, NP), np.int32)
    _load().oracle_nn(B, NP, NQ, _ptr(P), _ptr(Q), int(bool(fused)), _ptr(dist), _ptr(idx))
    return dist, idx


def nn(X, Y, fused: bool = False):
    """Both directions: (dist_xy [B,N], idx_xy [B,N], dist_yx [B,M], idx_yx [B,M])."""
    dxy, ixy = nn_one_way(X, Y, fused)
    dyx, iyx = nn_one_way(Y, X, fused)
    return dxy, ixy, dyx, iyx


def chamfer(dist_xy, dist_yx, w1: float = 1.0, w2: float = 1.0) -> np.ndarray:
    """Per-item Chamfer distance [B] in float64: w1*mean(dist_xy) + w2*mean(dist_yx)."""
    dxy = np.ascontiguousarray(dist_xy, np.float32)
    dyx = np.ascontiguousarray(dist_yx, np.float32)
    B, N, M = dxy.shape[0], dxy.shape[1], dyx.shape[1]
    out = np.empty(B, np.float64)
    _load().oracle_chamfer(B, N, M, _ptr(dxy), _ptr(dyx), float(w1), float(w2), _ptr(out))
    return out


def fscore(dist_xy, dist_yx, tau: float):
    """F-score@tau per item: (F, P, R, cnt_p, cnt_r); tau is taken as float32."""
    dxy = np.ascontiguousarray(dist_xy, np.float32)
    dyx = np.ascontiguousarray(dist_yx, np.float32)
    B, N, M = dxy.shape[0], dxy.shape[1], dyx.shape[1]
    f, p, r = (np.empty(B, np.float64) for _ in range(3))
    cp, cr = np.empty(B, np.int64), np.empty(B, np.int64)
    _load().oracle_fscore(B, N, M, _ptr(dxy), _ptr(dyx), ctypes.c_float(tau),
                          _ptr(f), _ptr(p), _ptr(r), _ptr(cp), _ptr(cr))
    return f, p, r, cp, cr


def backward_pointwise(g_xy, g_yx, X, Y, idx_xy, idx_yx):
    """Gradient of sum g_xy*dist_xy + sum g_yx*dist_yx for fixed neighbours.

    Returns (gX, gY, sX, sY, nX, nY): float64 gradients, per-component sums of
    absolute contributions and per-point contribution counts.
    """
    X, Y = _cloud(X), _cloud(Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    gxy = np.ascontiguousarray(np.broadcast_to(g_xy, (B, N)), np.float64)
    gyx = np.ascontiguousarray(np.broadcast_to(g_yx, (B, M)), np.float64)
    ixy = np.ascontiguousarray(idx_xy, np.int32)
    iyx = np.ascontiguousarray(idx_yx, np.int32)
    if ixy.shape != (B, N) or iyx.shape != (B, M):
        raise ValueError("index arrays do not match the clouds")
    if ixy.min(initial=0) < 0 or ixy.max(initial=0) >= M or iyx.min(initial=0) < 0 \
            or iyx.max(initial=0) >= N:
        raise ValueError("neighbour index out of range")
    gX, sX = np.empty((B, N, 3)), np.empty((B, N, 3))
    gY, sY = np.empty((B, M, 3)), np.empty((B, M, 3))
    nX, nY = np.empty((B, N), np.int32), np.empty((B, M), np.int32)
    _load().oracle_backward_pointwise(B, N, M, _ptr(gxy), _ptr(gyx), _ptr(X), _ptr(Y),
                                      _ptr(ixy), _ptr(iyx), _ptr(gX), _ptr(gY), _ptr(sX),
                                      _ptr(sY), _ptr(nX), _ptr(nY))
    return gX, gY, sX, sY, nX, nY


def backward(grad_out, X, Y, idx_xy, idx_yx, w1: float = 1.0, w2: float = 1.0):
    """Gradient of sum_b grad_out[b] * chamfer[b]: the pointwise form with
    g_xy[b,i] = grad_out[b] * w1 / N and g_yx[b,j] = grad_out[b] * w2 / M."""
    X, Y = _cloud(X), _cloud(Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    go = np.asarray(grad_out, np.float64).reshape(B)
    g_xy = np.repeat((go * float(w1) / N)[:, None], N, axis=1)
    g_yx = np.repeat((go * float(w2) / M)[:, None], M, axis=1)
    return backward_pointwise(g_xy, g_yx, X, Y, idx_xy, idx_yx)


def forward_all(X, Y, taus=(0.01,), w1: float = 1.0, w2: float = 1.0, fused: bool = False):
    """One full pass: nearest neighbours, Chamfer and F-score at each tau."""
    dxy, ixy, dyx, iyx = nn(X, Y, fused)
    cd = chamfer(dxy, dyx, w1, w2)
    fs = {float(t): fscore(dxy, dyx, t) for t in taus}
    return dict(dist_xy=dxy, idx_xy=ixy, dist_yx=dyx, idx_yx=iyx, chamfer=cd, fscore=fs)


# ---------------------------------------------------------------- mesh sampling
# Kaolin Sec. 2.1: differentiable surface sampling (reparameterization trick).

def _mesh(V, F):
    V = np.ascontiguousarray(V, np.float32)
    F = np.ascontiguousarray(F, np.int32)
    if V.ndim != 3 or V.shape[2] != 3 or F.ndim != 3 or F.shape[2] != 3 or F.shape[0] != V.shape[0]:
        raise ValueError("expected V [B, nv, 3] float and F [B, nf, 3] int")
    if F.size and (F.min() < 0 or F.max() >= V.shape[1]):
        raise ValueError("face index out of range")
    return V, F


def face_areas(V, F) -> np.ndarray:
    """Area of every face [B, nf] in double."""
    V, F = _mesh(V, F)
    out = np.empty(F.shape[:2], np.float64)
    _load().oracle_face_areas(V.shape[0], V.shape[1], F.shape[1], _ptr(V), _ptr(F), _ptr(out))
    return out


def sample_faces(V, F, u) -> np.ndarray:
    """Area-weighted face choice for uniforms u [B, S]: first f with u*total < cdf_f."""
    V, F = _mesh(V, F)
    u = np.ascontiguousarray(u, np.float32)
    B, S = u.shape
    scratch = np.empty(F.shape[:2], np.float64)
    out = np.empty((B, S), np.int32)
    _load().oracle_sample_faces(B, V.shape[1], F.shape[1], _ptr(V), _ptr(F), S, _ptr(u),
                                _ptr(scratch), _ptr(out))
    return out


def sample_points(V, F, fidx, r1, r2) -> np.ndarray:
    """Reparameterised samples P [B, S, 3] (float64) on the chosen faces."""
    V, F = _mesh(V, F)
    fidx = np.ascontiguousarray(fidx, np.int32)
    r1 = np.ascontiguousarray(r1, np.float32)
    r2 = np.ascontiguousarray(r2, np.float32)
    B, S = fidx.shape
    if fidx.size and (fidx.min() < 0 or fidx.max() >= F.shape[1]):
        raise ValueError("face choice out of range")
    out = np.empty((B, S, 3), np.float64)
    _load().oracle_sample_points(B, V.shape[1], F.shape[1], _ptr(V), _ptr(F), S, _ptr(fidx),
                                 _ptr(r1), _ptr(r2), _ptr(out))
    return out


def sample_backward(V, F, fidx, r1, r2, gP):
    """(gV [B, nv, 3], sV, nV): gradient of sum(gP * P) w.r.t. the vertices,
    per-component absolute sums and per-vertex contribution counts."""
    V, F = _mesh(V, F)
    fidx = np.ascontiguousarray(fidx, np.int32)
    r1 = np.ascontiguousarray(r1, np.float32)
    r2 = np.ascontiguousarray(r2, np.float32)
    gP = np.ascontiguousarray(gP, np.float64)
    B, S = fidx.shape
    gV = np.empty(V.shape, np.float64)
    sV = np.empty(V.shape, np.float64)
    nV = np.empty(V.shape[:2], np.int32)
    _load().oracle_sample_backward(B, V.shape[1], F.shape[1], _ptr(F), S, _ptr(fidx), _ptr(r1),
                                   _ptr(r2), _ptr(gP), _ptr(gV), _ptr(sV), _ptr(nV))
    return gV, sV, nV


# ---------------------------------------------------------------- point to surface
# Kaolin Sec. 2.5: point-to-surface loss for meshes (squared distance from each
# point to the closest face, mean over the points).

def point_triangle(p, a, b, c):
    """(d2 [n], w [n, 3]): squared distance from p[k] to the closed triangle
    (a[k], b[k], c[k]) and the barycentric coordinates of the closest point;
    all inputs [n, 3], rounded to float32 first."""
    p, a, b, c = (np.ascontiguousarray(np.reshape(x, (-1, 3)), np.float32) for x in (p, a, b, c))
    n = p.shape[0]
    if not (a.shape[0] == b.shape[0] == c.shape[0] == n):
        raise ValueError("p, a, b, c must have the same number of rows")
    d2 = np.empty(n, np.float64)
    w = np.empty((n, 3), np.float64)
    _load().oracle_point_triangle_batch(n, _ptr(p), _ptr(a), _ptr(b), _ptr(c), _ptr(d2), _ptr(w))
    return d2, w


def p2s_forward(P, V, F):
    """(dist [B, S] float64, fidx [B, S] int32, w [B, S, 3] float64): squared
    distance from every point to the closest face (lowest index on exact
    ties) and the barycentric coordinates of the closest point."""
    V, F = _mesh(V, F)
    P = np.ascontiguousarray(P, np.float32)
    if P.ndim != 3 or P.shape[2] != 3 or P.shape[0] != V.shape[0]:
        raise ValueError("expected P [B, S, 3]")
    B, S = P.shape[:2]
    dist = np.empty((B, S), np.float64)
    fidx = np.empty((B, S), np.int32)
    w = np.empty((B, S, 3), np.float64)
    _load().oracle_p2s_forward(B, S, V.shape[1], F.shape[1], _ptr(P), _ptr(V), _ptr(F),
                               _ptr(dist), _ptr(fidx), _ptr(w))
    return dist, fidx, w


def p2s_backward(P, V, F, fidx, g):
    """(gP [B, S, 3], gV [B, nv, 3], sV, nV) for the given face choices and
    per-point weights g [B, S] = dL/d dist, in float64."""
    V, F = _mesh(V, F)
    P = np.ascontiguousarray(P, np.float32)
    fidx = np.ascontiguousarray(fidx, np.int32)
    g = np.ascontiguousarray(np.broadcast_to(g, fidx.shape), np.float64)
    B, S = fidx.shape
    if P.shape != (B, S, 3) or P.shape[0] != V.shape[0]:
        raise ValueError("P and fidx shapes disagree")
    gP = np.empty((B, S, 3), np.float64)
    gV = np.empty(V.shape, np.float64)
    sV = np.empty(V.shape, np.float64)
    nV = np.empty(V.shape[:2], np.int32)
    _load().oracle_p2s_backward(B, S, V.shape[1], F.shape[1], _ptr(P), _ptr(V), _ptr(F),
                                _ptr(fidx), _ptr(g), _ptr(gP), _ptr(gV), _ptr(sV), _ptr(nV))
    return gP, gV, sV, nV
