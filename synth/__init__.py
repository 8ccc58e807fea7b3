"""Seeded synthetic point-cloud generators for the batched Chamfer distance.

This module is shared by the parity tests, the benchmark and the CPU oracle's
callers.  It holds input generation only: none of the Chamfer / nearest-neighbour
/ F-score / gradient arithmetic lives here, so that the oracle and the HIP path
share no computation.

The paper evaluates its point-cloud metrics on ShapeNet-style mesh
reconstruction (Sec. 2.5, Sec. 2.6); those datasets are not used.  Five
workload families stand in for them, each drawn from NumPy's PCG64 stream in
float64 and then cast to float32 (the precision the path computes in):

  uniform   i.i.d. U[-1,1]^3 points.
  sphere    points on a sphere of per-item radius U(0.5,1.0) with N(0,0.01^2)
            jitter; Y is an independent sample of the same sphere under a
            uniform random rotation (mesh-reconstruction training-loss shape).
  mesh      area-weighted uniform samples on a 200-triangle soup whose
            vertices are N(0,0.3^2); X and Y are independent samples of the
            same soup (the surface-sampling step of Sec. 2.1 feeding the loss).
  gmm       a 32-component isotropic Gaussian mixture per item, means
            U[-1,1]^3, sigma U(0.01,0.1), equal weights, shared by X and Y
            (asymmetric evaluation-metric shape).
  grid_dup  coordinates quantised to a 1/256 grid in [-1,1]^3 and 30% of Y
            being exact copies of distinct X points (exact ties everywhere).

Every array is C-contiguous float32 of shape [B, N, 3] / [B, M, 3].
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Tuple

import numpy as np

__all__ = ["Workload", "WORKLOADS", "generate", "workload", "lattice_pair", "triangle_soup",
           "grid_mesh", "uniforms", "icosphere", "p2s_workload", "P2S_WORKLOAD"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """A named workload: a generator kind plus its full-size shape."""

    name: str
    kind: str
    B: int
    N: int
    M: int
    taus: Tuple[float, ...]
    seed: int

    def describe(self) -> str:
        return f"{self.name}: kind={self.kind} B={self.B} N={self.N} M={self.M} taus={self.taus}"


# The five workloads, numbered 1..5; workload k draws from seed k.
WORKLOADS: Dict[int, Workload] = {
    1: Workload("uniform_b1_n1024", "uniform", 1, 1024, 1024, (0.01,), 1),
    2: Workload("sphere_b32_n2048", "sphere", 32, 2048, 2048, (0.01,), 2),
    3: Workload("mesh_b16_n16384", "mesh", 16, 16384, 16384, (0.005, 0.01, 0.02), 3),
    4: Workload("gmm_b4_n100000_m10000", "gmm", 4, 100000, 10000, (0.01,), 4),
    5: Workload("griddup_b8_n65536", "grid_dup", 8, 65536, 65536, (0.01,), 5),
}


def _f32(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _unit_directions(rng: np.random.Generator, n: int) -> np.ndarray:
    g = rng.standard_normal((n, 3))
    nrm = np.linalg.norm(g, axis=1, keepdims=True)
    nrm[nrm == 0.0] = 1.0
    return g / nrm


def _random_rotation(rng: np.random.Generator) -> np.ndarray:
    # QR of a Gaussian matrix with the diagonal of R made positive gives a
    # Haar-distributed orthogonal matrix; flip one column to land in SO(3).
    q, r = np.linalg.qr(rng.standard_normal((3, 3)))
    q = q * np.sign(np.diag(r))
    if np.linalg.det(q) < 0:
        q[:, 0] = -q[:, 0]
    return q


def _gen_uniform(rng, B, N, M):
    return rng.uniform(-1.0, 1.0, (B, N, 3)), rng.uniform(-1.0, 1.0, (B, M, 3))


def _gen_sphere(rng, B, N, M):
    X = np.empty((B, N, 3))
    Y = np.empty((B, M, 3))
    for b in range(B):
        r = rng.uniform(0.5, 1.0)
        X[b] = r * _unit_directions(rng, N) + rng.normal(0.0, 0.01, (N, 3))
        rot = _random_rotation(rng)
        Y[b] = (r * _unit_directions(rng, M)) @ rot.T + rng.normal(0.0, 0.01, (M, 3))
    return X, Y


def _sample_soup(rng, tri: np.ndarray, n: int) -> np.ndarray:
    # tri: [T,3(vertex),3(xyz)].  Area-weighted triangle choice, then uniform
    # barycentrics (1-sqrt(r1), sqrt(r1)(1-r2), sqrt(r1) r2) (Osada et al. 2002).
    e1 = tri[:, 1] - tri[:, 0]
    e2 = tri[:, 2] - tri[:, 0]
    area = 0.5 * np.linalg.norm(np.cross(e1, e2), axis=1)
    p = area / area.sum()
    t = rng.choice(len(tri), size=n, p=p)
    r1 = np.sqrt(rng.uniform(0.0, 1.0, n))
    r2 = rng.uniform(0.0, 1.0, n)
    a = 1.0 - r1
    b = r1 * (1.0 - r2)
    c = r1 * r2
    v = tri[t]
    return a[:, None] * v[:, 0] + b[:, None] * v[:, 1] + c[:, None] * v[:, 2]


def _gen_mesh(rng, B, N, M, n_tri=200):
    X = np.empty((B, N, 3))
    Y = np.empty((B, M, 3))
    for b in range(B):
        tri = rng.normal(0.0, 0.3, (n_tri, 3, 3))
        X[b] = _sample_soup(rng, tri, N)
        Y[b] = _sample_soup(rng, tri, M)
    return X, Y


def _gen_gmm(rng, B, N, M, k=32):
    X = np.empty((B, N, 3))
    Y = np.empty((B, M, 3))
    for b in range(B):
        mu = rng.uniform(-1.0, 1.0, (k, 3))
        sig = rng.uniform(0.01, 0.1, k)
        for out, n in ((X, N), (Y, M)):
            comp = rng.integers(0, k, n)
            out[b] = mu[comp] + sig[comp, None] * rng.standard_normal((n, 3))
    return X, Y


def _quantise(v: np.ndarray) -> np.ndarray:
    return np.clip(np.round(v * 256.0) / 256.0, -1.0, 1.0)


def _gen_grid_dup(rng, B, N, M, copy_frac=0.3):
    X = np.empty((B, N, 3))
    Y = np.empty((B, M, 3))
    n_copy = min(int(np.floor(copy_frac * M)), N)
    for b in range(B):
        X[b] = _quantise(rng.uniform(-1.0, 1.0, (N, 3)))
        Y[b] = _quantise(rng.uniform(-1.0, 1.0, (M, 3)))
        pos = rng.choice(M, size=n_copy, replace=False)
        src = rng.choice(N, size=n_copy, replace=False)
        Y[b, pos] = X[b, src]
    return X, Y


_GENERATORS = {
    "uniform": _gen_uniform,
    "sphere": _gen_sphere,
    "mesh": _gen_mesh,
    "gmm": _gen_gmm,
    "grid_dup": _gen_grid_dup,
}


def generate(kind: str, B: int, N: int, M: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Draw (X [B,N,3], Y [B,M,3]) float32 clouds of the given family."""
    if kind not in _GENERATORS:
        raise ValueError(f"unknown workload kind {kind!r}")
    rng = np.random.default_rng(seed)
    X, Y = _GENERATORS[kind](rng, int(B), int(N), int(M))
    return _f32(X), _f32(Y)


def workload(k: int, *, B: int | None = None, N: int | None = None, M: int | None = None,
             seed: int | None = None) -> Tuple[np.ndarray, np.ndarray]:
    """Workload k at full size, or with B/N/M/seed overridden (same distribution)."""
    w = WORKLOADS[k]
    return generate(w.kind, w.B if B is None else B, w.N if N is None else N,
                    w.M if M is None else M, w.seed if seed is None else seed)


def lattice_pair(B: int, dims: Tuple[int, int, int], h: float, shift, seed: int):
    """A dyadic lattice X and Y = permuted (X + shift), for closed-form checks.

    X is the grid {h * (a, b, c)} (centred at the origin) with `dims` points per
    axis, repeated for each of the B items; `shift` is a 3-vector whose entries
    must be dyadic and smaller than h/2 in magnitude, so the unique nearest
    neighbour of every X point is its own shifted copy.  Y[b, perm[b, i]] =
    X[b, i] + shift.  Returns (X, Y, perm) with perm int64 [B, N].
    """
    nx, ny, nz = dims
    s = np.asarray(shift, dtype=np.float64)
    if np.any(np.abs(s) >= h / 2):
        raise ValueError("shift must be below half the lattice spacing in every axis")
    a, b_, c = np.meshgrid(np.arange(nx) - nx // 2, np.arange(ny) - ny // 2,
                           np.arange(nz) - nz // 2, indexing="ij")
    base = h * np.stack([a.ravel(), b_.ravel(), c.ravel()], axis=1).astype(np.float64)
    n = base.shape[0]
    rng = np.random.default_rng(seed)
    X = np.broadcast_to(base, (B, n, 3)).copy()
    perm = np.stack([rng.permutation(n) for _ in range(B)])
    Y = np.empty_like(X)
    for b in range(B):
        Y[b, perm[b]] = X[b] + s
    Xf, Yf = _f32(X), _f32(Y)
    if not (np.array_equal(Xf.astype(np.float64), X) and np.array_equal(Yf.astype(np.float64), Y)):
        raise ValueError("lattice is not exactly representable in float32")
    return Xf, Yf, perm


def triangle_soup(B: int, n_tri: int, seed: int, sigma: float = 0.3):
    """Independent triangles: V [B, 3*n_tri, 3] with vertices N(0, sigma^2), F [B, n_tri, 3]
    (face t uses vertices 3t, 3t+1, 3t+2) -- the meshes of the mesh workload."""
    rng = np.random.default_rng(seed)
    V = rng.normal(0.0, sigma, (B, 3 * n_tri, 3))
    F = np.broadcast_to(np.arange(3 * n_tri, dtype=np.int32).reshape(n_tri, 3), (B, n_tri, 3))
    return _f32(V), np.ascontiguousarray(F)


def grid_mesh(B: int, n: int, seed: int, amp: float = 0.1):
    """A triangulated n x n height field per item (vertices shared by up to six
    faces): V [B, n*n, 3] on [-1,1]^2 with heights amp * N(0,1), F [B, 2(n-1)^2, 3]."""
    rng = np.random.default_rng(seed)
    gx, gy = np.meshgrid(np.linspace(-1.0, 1.0, n), np.linspace(-1.0, 1.0, n), indexing="ij")
    V = np.empty((B, n * n, 3))
    for b in range(B):
        V[b, :, 0] = gx.ravel()
        V[b, :, 1] = gy.ravel()
        V[b, :, 2] = amp * rng.standard_normal(n * n)
    i, j = np.meshgrid(np.arange(n - 1), np.arange(n - 1), indexing="ij")
    v00 = (i * n + j).ravel()
    v10 = ((i + 1) * n + j).ravel()
    v01 = (i * n + j + 1).ravel()
    v11 = ((i + 1) * n + j + 1).ravel()
    faces = np.concatenate([np.stack([v00, v10, v11], 1), np.stack([v00, v11, v01], 1)])
    F = np.broadcast_to(faces.astype(np.int32), (B,) + faces.shape)
    return _f32(V), np.ascontiguousarray(F)


def uniforms(B: int, S: int, seed: int, count: int = 3):
    """`count` arrays of float32 uniforms in [0, 1), shape [B, S] each (the random
    numbers a sampler draws, drawn here and passed in)."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        u = rng.random((B, S)).astype(np.float32)
        out.append(np.minimum(u, np.float32(np.nextafter(np.float32(1), np.float32(0)))))
    return tuple(out)


def icosphere(level: int):
    """Unit icosphere: the icosahedron with each face split into 4 (edge
    midpoints pushed to the sphere) `level` times.  Returns V [nv, 3] float64,
    F [nf, 3] int32 with outward (counter-clockwise) faces; level 4 gives 2562
    vertices and 5120 faces, the initial mesh of sphere-deforming
    reconstruction networks."""
    t = (1.0 + 5.0 ** 0.5) / 2.0
    verts = [(-1, t, 0), (1, t, 0), (-1, -t, 0), (1, -t, 0), (0, -1, t), (0, 1, t),
             (0, -1, -t), (0, 1, -t), (t, 0, -1), (t, 0, 1), (-t, 0, -1), (-t, 0, 1)]
    verts = [np.array(v, dtype=np.float64) / np.linalg.norm(v) for v in verts]
    faces = [(0, 11, 5), (0, 5, 1), (0, 1, 7), (0, 7, 10), (0, 10, 11), (1, 5, 9), (5, 11, 4),
             (11, 10, 2), (10, 7, 6), (7, 1, 8), (3, 9, 4), (3, 4, 2), (3, 2, 6), (3, 6, 8),
             (3, 8, 9), (4, 9, 5), (2, 4, 11), (6, 2, 10), (8, 6, 7), (9, 8, 1)]
    for _ in range(level):
        mid = {}

        def midpoint(i, j):
            key = (min(i, j), max(i, j))
            if key not in mid:
                m = verts[i] + verts[j]
                verts.append(m / np.linalg.norm(m))
                mid[key] = len(verts) - 1
            return mid[key]

        nxt = []
        for a, b, c in faces:
            ab, bc, ca = midpoint(a, b), midpoint(b, c), midpoint(c, a)
            nxt += [(a, ab, ca), (b, bc, ab), (c, ca, bc), (ab, bc, ca)]
        faces = nxt
    return np.array(verts), np.array(faces, dtype=np.int32)


@dataclasses.dataclass(frozen=True)
class P2SWorkload:
    """Point-to-surface workload: B deformed icospheres and B point clouds."""

    name: str
    B: int
    S: int
    level: int
    seed: int


P2S_WORKLOAD = P2SWorkload("p2s_b16_s16384_f5120", 16, 16384, 4, 6)


def p2s_workload(B: int = 16, S: int = 16384, level: int = 4, seed: int = 6,
                 noise: float = 0.05, jitter: float = 0.01):
    """Point-to-surface inputs standing in for mesh reconstruction with a
    point-to-surface loss: per item, an icosphere of radius U(0.8, 1.2) whose
    vertices move radially by N(0, noise^2) (the predicted mesh), and S points
    on an independently drawn radius-U(0.8, 1.2) sphere with N(0, jitter^2)
    jitter (the target surface's samples).  Returns P [B, S, 3], V [B, nv, 3]
    float32 and F [B, nf, 3] int32."""
    V0, F0 = icosphere(level)
    rng = np.random.default_rng(seed)
    V = np.empty((B,) + V0.shape)
    P = np.empty((B, S, 3))
    for b in range(B):
        r = rng.uniform(0.8, 1.2)
        V[b] = V0 * (r + rng.normal(0.0, noise, (len(V0), 1)))
        rp = rng.uniform(0.8, 1.2)
        P[b] = rp * _unit_directions(rng, S) + rng.normal(0.0, jitter, (S, 3))
    F = np.broadcast_to(F0, (B,) + F0.shape)
    return _f32(P), _f32(V), np.ascontiguousarray(F)
