"""MI355X-native batched Chamfer distance (Kaolin, arXiv 1911.05063, Sec. 2.5).

Thin Python binding over the C ABI of ``libcd_hip.so`` (declared in
``include/cd.h``).  It only marshals arguments: torch supplies device memory
and the current stream, every step of the computation runs in the library's
HIP kernels.  There is no CPU fallback: if the library is missing or the
tensors are not on a ROCm device, the calls raise.

Functions (names follow the C ABI):
  nn_distance(X, Y)                 -> dist_xy, idx_xy, dist_yx, idx_yx
  nn_distance_noalloc(X, Y, out)    -> the same through cd_forward_noalloc (static workspace)
  chamfer_reduce(dist_xy, dist_yx)  -> chamfer [B]
  f_score(dist_xy, dist_yx, tau)    -> f, precision, recall  [B] each
  metrics(dist_xy, dist_yx, taus)   -> chamfer [B], f / precision / recall [ntau, B]
  chamfer_backward(...)             -> gX, gY
  chamfer_distance(X, Y, w1, w2)    -> chamfer [B], differentiable (autograd)
  mesh_sample_faces / mesh_sample_points / mesh_sample_backward
                                    -> differentiable mesh surface sampling (Sec. 2.1)
  p2s_forward / p2s_backward / point_to_surface
                                    -> point-to-surface distance to triangle meshes (Sec. 2.5)
  emd_forward / emd_backward / earth_movers_distance
                                    -> approximate EMD (scheduled Sinkhorn, Sec. 2.5)
  sample_points(V, F, S)            -> P [B, S, 3], differentiable in V (autograd)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

__all__ = [
    "CDError", "LIB_PATH", "library", "workspace_bytes", "nn_distance", "nn_distance_noalloc",
    "FORWARD_NOALLOC_MAX_BYTES", "chamfer_reduce",
    "f_score", "metrics", "chamfer_backward", "chamfer_backward_pointwise", "chamfer_distance",
    "ChamferDistance", "forward_step", "mesh_sample_faces", "mesh_sample_points",
    "mesh_sample_backward", "MeshSample", "sample_points", "p2s_forward", "p2s_backward",
    "PointToSurface", "point_to_surface", "emd_forward", "emd_backward", "EarthMoversDistance",
    "earth_movers_distance",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcd_hip.so")
CD_OK = 0

_lib = None


class CDError(RuntimeError):
    """A cd_* call returned a status other than CD_OK."""


def library() -> ctypes.CDLL:
    """Load libcd_hip.so (built in-tree by paper_1911_05063_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_1911_05063_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    i64, vp, f32, st = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_int
    lib.cd_status_string.restype = ctypes.c_char_p
    lib.cd_status_string.argtypes = [st]
    lib.cd_last_error.restype = ctypes.c_char_p
    lib.cd_last_error.argtypes = []
    lib.cd_version.restype = ctypes.c_char_p
    lib.cd_version.argtypes = []
    lib.cd_workspace_bytes.restype = ctypes.c_size_t
    lib.cd_workspace_bytes.argtypes = [i64, i64, i64]
    lib.cd_forward.restype = st
    lib.cd_forward.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.cd_reduce.restype = st
    lib.cd_reduce.argtypes = [i64, i64, i64, vp, vp, f32, f32, vp, vp]
    lib.cd_fscore.restype = st
    lib.cd_fscore.argtypes = [i64, i64, i64, vp, vp, f32, vp, vp, vp, vp]
    lib.cd_metrics.restype = st
    lib.cd_metrics.argtypes = [i64, i64, i64, vp, vp, f32, f32, vp, ctypes.c_int, vp, vp, vp, vp, vp]
    lib.cd_backward.restype = st
    lib.cd_backward_workspace_bytes.restype = ctypes.c_size_t
    lib.cd_backward_workspace_bytes.argtypes = [i64, i64, i64]
    lib.cd_backward.argtypes = [i64, i64, i64, vp, f32, f32, vp, vp, vp, vp, vp, vp, vp,
                                ctypes.c_size_t, vp]
    lib.cd_mesh_workspace_bytes.restype = ctypes.c_size_t
    lib.cd_mesh_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.cd_mesh_sample_faces.restype = st
    lib.cd_mesh_sample_faces.argtypes = [i64, i64, i64, vp, vp, i64, vp, vp, vp, ctypes.c_size_t, vp]
    lib.cd_mesh_sample_points.restype = st
    lib.cd_mesh_sample_points.argtypes = [i64, i64, i64, vp, vp, i64, vp, vp, vp, vp, vp]
    lib.cd_mesh_sample_backward.restype = st
    lib.cd_mesh_sample_backward.argtypes = [i64, i64, i64, vp, i64, vp, vp, vp, vp, vp, vp,
                                            ctypes.c_size_t, vp]
    lib.cd_p2s_workspace_bytes.restype = ctypes.c_size_t
    lib.cd_p2s_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.cd_p2s_forward.restype = st
    lib.cd_p2s_forward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.cd_p2s_backward.restype = st
    lib.cd_p2s_backward.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp,
                                    ctypes.c_size_t, vp]
    lib.cd_emd_workspace_bytes.restype = ctypes.c_size_t
    lib.cd_emd_workspace_bytes.argtypes = [i64, i64, i64]
    lib.cd_emd_forward.restype = st
    lib.cd_emd_forward.argtypes = [i64, i64, i64, vp, vp, f32, f32, ctypes.c_int, ctypes.c_int,
                                   vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.cd_emd_backward.restype = st
    lib.cd_emd_backward.argtypes = [i64, i64, i64, vp, vp, vp, vp, f32, vp, vp, vp, vp,
                                    ctypes.c_size_t, vp]
    lib.cd_backward_pointwise.restype = st
    lib.cd_backward_pointwise.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                          ctypes.c_size_t, vp]
    lib.cd_forward_noalloc.restype = st
    lib.cd_forward_noalloc.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
    _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != CD_OK:
        lib = library()
        raise CDError(f"{what}: {lib.cd_status_string(status).decode()}: "
                      f"{lib.cd_last_error().decode()}")


def _device_tensor(t: torch.Tensor, name: str, dtype: torch.dtype) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a ROCm GPU (got {t.device}); there is no CPU path")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    return t.contiguous()


def _cloud(t: torch.Tensor, name: str) -> torch.Tensor:
    t = _device_tensor(t, name, torch.float32)
    if t.dim() != 3 or t.shape[2] != 3:
        raise ValueError(f"{name} must have shape [B, n, 3] (got {tuple(t.shape)})")
    return t


def _expect(t: torch.Tensor, name: str, dtype: torch.dtype, shape, device: torch.device
            ) -> torch.Tensor:
    """A contiguous tensor of exactly `shape` on `device`: the kernels index
    every array by the sizes they are given, so a smaller one would be read or
    written out of bounds."""
    t = _device_tensor(t, name, dtype)
    shape = tuple(int(n) for n in shape)
    if tuple(t.shape) != shape:
        raise ValueError(f"{name} must have shape {list(shape)} (got {list(t.shape)})")
    if t.device != device:
        raise ValueError(f"{name} must be on {device} (got {t.device})")
    return t


def _clouds(X: torch.Tensor, Y: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    X, Y = _cloud(X, "X"), _cloud(Y, "Y")
    if X.device != Y.device or X.shape[0] != Y.shape[0]:
        raise ValueError("X and Y must share device and batch size")
    return X, Y


def _distances(dist_xy: torch.Tensor, dist_yx: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    dxy = _device_tensor(dist_xy, "dist_xy", torch.float32)
    if dxy.dim() != 2:
        raise ValueError(f"dist_xy must have shape [B, N] (got {list(dxy.shape)})")
    dyx = _device_tensor(dist_yx, "dist_yx", torch.float32)
    if dyx.dim() != 2:
        raise ValueError(f"dist_yx must have shape [B, M] (got {list(dyx.shape)})")
    dyx = _expect(dyx, "dist_yx", torch.float32, (dxy.shape[0], dyx.shape[1]), dxy.device)
    return dxy, dyx


def _workspace(ws: Optional[torch.Tensor], need: int, device: torch.device) -> torch.Tensor:
    """The caller's workspace if it is a large enough uint8 tensor on `device`,
    else a new one."""
    if ws is not None:
        ws = _device_tensor(ws, "workspace", torch.uint8)
        if ws.device != device:
            raise ValueError(f"workspace must be on {device} (got {ws.device})")
        if ws.numel() >= need:
            return ws
    return torch.empty(max(need, 1), dtype=torch.uint8, device=device)


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def workspace_bytes(B: int, N: int, M: int) -> int:
    """Device workspace (bytes) that cd_forward needs for this shape."""
    return int(library().cd_workspace_bytes(B, N, M))


def nn_distance(X: torch.Tensor, Y: torch.Tensor, workspace: Optional[torch.Tensor] = None
                ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """Nearest neighbours both ways: (dist_xy [B,N], idx_xy [B,N], dist_yx [B,M], idx_yx [B,M])."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    dev = X.device
    dist_xy = torch.empty((B, N), dtype=torch.float32, device=dev)
    idx_xy = torch.empty((B, N), dtype=torch.int32, device=dev)
    dist_yx = torch.empty((B, M), dtype=torch.float32, device=dev)
    idx_yx = torch.empty((B, M), dtype=torch.int32, device=dev)
    lib = library()
    workspace = _workspace(workspace, int(lib.cd_workspace_bytes(B, N, M)), dev)
    with torch.cuda.device(dev):
        _check(lib.cd_forward(B, N, M, _ptr(X), _ptr(Y), _ptr(dist_xy), _ptr(idx_xy),
                              _ptr(dist_yx), _ptr(idx_yx), _ptr(workspace), workspace.numel(),
                              ctypes.c_void_p(_stream(dev))), "cd_forward")
    return dist_xy, idx_xy, dist_yx, idx_yx


# The static workspace of cd_forward_noalloc (CD_FORWARD_NOALLOC_MAX_BYTES).
FORWARD_NOALLOC_MAX_BYTES = 64 << 20


def nn_distance_noalloc(X: torch.Tensor, Y: torch.Tensor, out=None
                        ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """nn_distance through cd_forward_noalloc: the library uses its static
    per-GPU workspace.  `out` = (dist_xy, idx_xy, dist_yx, idx_yx) preallocated
    by the caller, else allocated here."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    dev = X.device
    if out is None:
        out = (torch.empty((B, N), dtype=torch.float32, device=dev),
               torch.empty((B, N), dtype=torch.int32, device=dev),
               torch.empty((B, M), dtype=torch.float32, device=dev),
               torch.empty((B, M), dtype=torch.int32, device=dev))
    dist_xy = _expect(out[0], "dist_xy", torch.float32, (B, N), dev)
    idx_xy = _expect(out[1], "idx_xy", torch.int32, (B, N), dev)
    dist_yx = _expect(out[2], "dist_yx", torch.float32, (B, M), dev)
    idx_yx = _expect(out[3], "idx_yx", torch.int32, (B, M), dev)
    if any(o.data_ptr() != t.data_ptr() for o, t in zip(out, (dist_xy, idx_xy, dist_yx, idx_yx))):
        raise ValueError("out tensors must be contiguous")
    with torch.cuda.device(dev):
        _check(library().cd_forward_noalloc(B, N, M, _ptr(X), _ptr(Y), _ptr(dist_xy),
                                            _ptr(idx_xy), _ptr(dist_yx), _ptr(idx_yx),
                                            ctypes.c_void_p(_stream(dev))), "cd_forward_noalloc")
    return dist_xy, idx_xy, dist_yx, idx_yx


def chamfer_reduce(dist_xy: torch.Tensor, dist_yx: torch.Tensor, w1: float = 1.0,
                   w2: float = 1.0) -> torch.Tensor:
    """chamfer[b] = w1 * mean_i dist_xy[b,i] + w2 * mean_j dist_yx[b,j]."""
    dxy, dyx = _distances(dist_xy, dist_yx)
    B, N, M = dxy.shape[0], dxy.shape[1], dyx.shape[1]
    out = torch.empty(B, dtype=torch.float32, device=dxy.device)
    with torch.cuda.device(dxy.device):
        _check(library().cd_reduce(B, N, M, _ptr(dxy), _ptr(dyx), float(w1), float(w2), _ptr(out),
                                   ctypes.c_void_p(_stream(dxy.device))), "cd_reduce")
    return out


def f_score(dist_xy: torch.Tensor, dist_yx: torch.Tensor, tau: float):
    """F-score@tau per item: (f, precision, recall), each [B] float32."""
    dxy, dyx = _distances(dist_xy, dist_yx)
    B, N, M = dxy.shape[0], dxy.shape[1], dyx.shape[1]
    f, p, r = (torch.empty(B, dtype=torch.float32, device=dxy.device) for _ in range(3))
    with torch.cuda.device(dxy.device):
        _check(library().cd_fscore(B, N, M, _ptr(dxy), _ptr(dyx), float(tau), _ptr(f), _ptr(p),
                                   _ptr(r), ctypes.c_void_p(_stream(dxy.device))), "cd_fscore")
    return f, p, r


def metrics(dist_xy: torch.Tensor, dist_yx: torch.Tensor, taus, w1: float = 1.0,
            w2: float = 1.0):
    """Chamfer [B] and F-score at each tau ([ntau, B] f, precision, recall) in one launch."""
    dxy, dyx = _distances(dist_xy, dist_yx)
    B, N, M = dxy.shape[0], dxy.shape[1], dyx.shape[1]
    taus = [float(t) for t in taus]
    ntau = len(taus)
    tau_arr = (ctypes.c_float * max(ntau, 1))(*taus)
    ch = torch.empty(B, dtype=torch.float32, device=dxy.device)
    f, p, r = (torch.empty((ntau, B), dtype=torch.float32, device=dxy.device) for _ in range(3))
    with torch.cuda.device(dxy.device):
        _check(library().cd_metrics(B, N, M, _ptr(dxy), _ptr(dyx), float(w1), float(w2),
                                    ctypes.cast(tau_arr, ctypes.c_void_p), ntau, _ptr(ch), _ptr(f),
                                    _ptr(p), _ptr(r), ctypes.c_void_p(_stream(dxy.device))),
               "cd_metrics")
    return ch, f, p, r


def _backward_ws(B, N, M, device):
    need = int(library().cd_backward_workspace_bytes(B, N, M))
    return torch.empty(max(need, 1), dtype=torch.uint8, device=device)


def chamfer_backward(grad_out: torch.Tensor, X: torch.Tensor, Y: torch.Tensor,
                     idx_xy: torch.Tensor, idx_yx: torch.Tensor, w1: float = 1.0,
                     w2: float = 1.0) -> Tuple[torch.Tensor, torch.Tensor]:
    """Gradient of sum_b grad_out[b] * chamfer[b] w.r.t. X and Y."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    go = _expect(grad_out, "grad_out", torch.float32, (B,), X.device)
    ixy = _expect(idx_xy, "idx_xy", torch.int32, (B, N), X.device)
    iyx = _expect(idx_yx, "idx_yx", torch.int32, (B, M), X.device)
    gX = torch.empty_like(X)
    gY = torch.empty_like(Y)
    ws = _backward_ws(B, N, M, X.device)
    with torch.cuda.device(X.device):
        _check(library().cd_backward(B, N, M, _ptr(go), float(w1), float(w2), _ptr(X), _ptr(Y),
                                     _ptr(ixy), _ptr(iyx), _ptr(gX), _ptr(gY), _ptr(ws),
                                     ws.numel(), ctypes.c_void_p(_stream(X.device))),
               "cd_backward")
    return gX, gY


def chamfer_backward_pointwise(g_xy: torch.Tensor, g_yx: torch.Tensor, X: torch.Tensor,
                               Y: torch.Tensor, idx_xy: torch.Tensor, idx_yx: torch.Tensor
                               ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Gradient w.r.t. X and Y given dL/d dist_xy [B,N] and dL/d dist_yx [B,M]."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    gxy = _expect(g_xy, "g_xy", torch.float32, (B, N), X.device)
    gyx = _expect(g_yx, "g_yx", torch.float32, (B, M), X.device)
    ixy = _expect(idx_xy, "idx_xy", torch.int32, (B, N), X.device)
    iyx = _expect(idx_yx, "idx_yx", torch.int32, (B, M), X.device)
    gX = torch.empty_like(X)
    gY = torch.empty_like(Y)
    ws = _backward_ws(B, N, M, X.device)
    with torch.cuda.device(X.device):
        _check(library().cd_backward_pointwise(B, N, M, _ptr(gxy), _ptr(gyx), _ptr(X), _ptr(Y),
                                               _ptr(ixy), _ptr(iyx), _ptr(gX), _ptr(gY),
                                               _ptr(ws), ws.numel(),
                                               ctypes.c_void_p(_stream(X.device))),
               "cd_backward_pointwise")
    return gX, gY


class ChamferDistance(torch.autograd.Function):
    """Per-item Chamfer distance with its backward through the HIP kernels."""

    @staticmethod
    def forward(ctx, X, Y, w1: float = 1.0, w2: float = 1.0):
        dist_xy, idx_xy, dist_yx, idx_yx = nn_distance(X, Y)
        ctx.save_for_backward(X, Y, idx_xy, idx_yx)
        ctx.w = (float(w1), float(w2))
        return chamfer_reduce(dist_xy, dist_yx, w1, w2)

    @staticmethod
    def backward(ctx, grad_out):
        X, Y, idx_xy, idx_yx = ctx.saved_tensors
        gX, gY = chamfer_backward(grad_out.float(), X, Y, idx_xy, idx_yx, *ctx.w)
        return gX, gY, None, None


def chamfer_distance(X: torch.Tensor, Y: torch.Tensor, w1: float = 1.0, w2: float = 1.0
                     ) -> torch.Tensor:
    """Differentiable per-item Chamfer distance [B] (batch mean is the caller's)."""
    return ChamferDistance.apply(X, Y, w1, w2)


def forward_step(X, Y, taus=(0.01,), w1: float = 1.0, w2: float = 1.0, workspace=None):
    """One forward pass of the whole path: neighbours, Chamfer, F-score at each tau."""
    dist_xy, idx_xy, dist_yx, idx_yx = nn_distance(X, Y, workspace)
    cd = chamfer_reduce(dist_xy, dist_yx, w1, w2)
    fs = {float(t): f_score(dist_xy, dist_yx, t) for t in taus}
    return dict(dist_xy=dist_xy, idx_xy=idx_xy, dist_yx=dist_yx, idx_yx=idx_yx, chamfer=cd,
                fscore=fs)


# ---------------------------------------------------------------- mesh sampling

def _mesh(V: torch.Tensor, F: torch.Tensor):
    V = _device_tensor(V, "V", torch.float32)
    F = _device_tensor(F, "F", torch.int32)
    if V.dim() != 3 or V.shape[2] != 3 or F.dim() != 3 or F.shape[2] != 3 or F.shape[0] != V.shape[0]:
        raise ValueError("expected V [B, nv, 3] float32 and F [B, nf, 3] int32")
    if V.device != F.device:
        raise ValueError("V and F must share a device")
    return V, F


def _mesh_ws(B, nv, nf, S, device):
    need = int(library().cd_mesh_workspace_bytes(B, nv, nf, S))
    return torch.empty(max(need, 1), dtype=torch.uint8, device=device)


def mesh_sample_faces(V: torch.Tensor, F: torch.Tensor, u: torch.Tensor) -> torch.Tensor:
    """Area-weighted face choice fidx [B, S] for uniforms u [B, S] (Sec. 2.1)."""
    V, F = _mesh(V, F)
    u = _device_tensor(u, "u", torch.float32)
    if u.dim() != 2:
        raise ValueError(f"u must have shape [B, S] (got {list(u.shape)})")
    u = _expect(u, "u", torch.float32, (V.shape[0], u.shape[1]), V.device)
    B, nv, nf, S = V.shape[0], V.shape[1], F.shape[1], u.shape[1]
    lib = library()
    ws = _mesh_ws(B, nv, nf, S, V.device)
    fidx = torch.empty((B, S), dtype=torch.int32, device=V.device)
    with torch.cuda.device(V.device):
        _check(lib.cd_mesh_sample_faces(B, nv, nf, _ptr(V), _ptr(F), S, _ptr(u), _ptr(fidx),
                                        _ptr(ws), ws.numel(), ctypes.c_void_p(_stream(V.device))),
               "cd_mesh_sample_faces")
    return fidx


def mesh_sample_points(V, F, fidx, r1, r2) -> torch.Tensor:
    """Reparameterised surface samples P [B, S, 3] on the faces fidx."""
    V, F = _mesh(V, F)
    fidx = _device_tensor(fidx, "fidx", torch.int32)
    if fidx.dim() != 2:
        raise ValueError(f"fidx must have shape [B, S] (got {list(fidx.shape)})")
    B, nv, nf, S = V.shape[0], V.shape[1], F.shape[1], fidx.shape[1]
    fidx = _expect(fidx, "fidx", torch.int32, (B, S), V.device)
    r1 = _expect(r1, "r1", torch.float32, (B, S), V.device)
    r2 = _expect(r2, "r2", torch.float32, (B, S), V.device)
    P = torch.empty((B, S, 3), dtype=torch.float32, device=V.device)
    with torch.cuda.device(V.device):
        _check(library().cd_mesh_sample_points(B, nv, nf, _ptr(V), _ptr(F), S, _ptr(fidx), _ptr(r1),
                                               _ptr(r2), _ptr(P), ctypes.c_void_p(_stream(V.device))),
               "cd_mesh_sample_points")
    return P


def mesh_sample_backward(nv: int, F, fidx, r1, r2, gP) -> torch.Tensor:
    """gV [B, nv, 3]: gradient of sum(gP * P) with respect to the vertices."""
    F = _device_tensor(F, "F", torch.int32)
    fidx = _device_tensor(fidx, "fidx", torch.int32)
    if F.dim() != 3 or F.shape[2] != 3 or fidx.dim() != 2:
        raise ValueError("expected F [B, nf, 3] int32 and fidx [B, S] int32")
    B, nf, S = F.shape[0], F.shape[1], fidx.shape[1]
    fidx = _expect(fidx, "fidx", torch.int32, (B, S), F.device)
    r1 = _expect(r1, "r1", torch.float32, (B, S), F.device)
    r2 = _expect(r2, "r2", torch.float32, (B, S), F.device)
    gP = _expect(gP, "gP", torch.float32, (B, S, 3), F.device)
    gV = torch.empty((B, int(nv), 3), dtype=torch.float32, device=F.device)
    ws = _mesh_ws(B, int(nv), nf, S, F.device)
    with torch.cuda.device(F.device):
        _check(library().cd_mesh_sample_backward(B, int(nv), nf, _ptr(F), S, _ptr(fidx), _ptr(r1),
                                                 _ptr(r2), _ptr(gP), _ptr(gV), _ptr(ws), ws.numel(),
                                                 ctypes.c_void_p(_stream(F.device))),
               "cd_mesh_sample_backward")
    return gV


class MeshSample(torch.autograd.Function):
    """P = sample(V) for fixed faces and uniforms, differentiable in V."""

    @staticmethod
    def forward(ctx, V, F, fidx, r1, r2):
        ctx.save_for_backward(F, fidx, r1, r2)
        ctx.nv = V.shape[1]
        return mesh_sample_points(V, F, fidx, r1, r2)

    @staticmethod
    def backward(ctx, gP):
        F, fidx, r1, r2 = ctx.saved_tensors
        return mesh_sample_backward(ctx.nv, F, fidx, r1, r2, gP.float()), None, None, None, None


def sample_points(V: torch.Tensor, F: torch.Tensor, num_samples: int, generator=None):
    """Differentiable surface sampling of B meshes: returns (P [B, S, 3], fidx).
    The uniforms are drawn with torch on the device (input generation); the
    face choice and the samples are computed by the library's kernels."""
    B = V.shape[0]
    u, r1, r2 = (torch.rand((B, int(num_samples)), device=V.device, generator=generator)
                 for _ in range(3))
    fidx = mesh_sample_faces(V.detach(), F, u)
    return MeshSample.apply(V, F, fidx, r1, r2), fidx


# ---------------------------------------------------------------- point to surface

def _p2s_args(P, V, F):
    V, F = _mesh(V, F)
    P = _device_tensor(P, "P", torch.float32)
    if P.dim() != 3 or P.shape[2] != 3 or P.shape[0] != V.shape[0] or P.device != V.device:
        raise ValueError("expected P [B, S, 3] float32 on the mesh's device")
    return P, V, F


def _p2s_ws(B, S, nv, nf, device):
    need = int(library().cd_p2s_workspace_bytes(B, S, nv, nf))
    return torch.empty(max(need, 1), dtype=torch.uint8, device=device)


def p2s_forward(P, V, F):
    """(dist [B, S], fidx [B, S]): squared distance from every point to the
    nearest face of its item's mesh, and that face (Sec. 2.5)."""
    P, V, F = _p2s_args(P, V, F)
    B, S, nv, nf = P.shape[0], P.shape[1], V.shape[1], F.shape[1]
    dist = torch.empty((B, S), dtype=torch.float32, device=P.device)
    fidx = torch.empty((B, S), dtype=torch.int32, device=P.device)
    ws = _p2s_ws(B, S, nv, nf, P.device)
    with torch.cuda.device(P.device):
        _check(library().cd_p2s_forward(B, S, nv, nf, _ptr(P), _ptr(V), _ptr(F), _ptr(dist),
                                        _ptr(fidx), _ptr(ws), ws.numel(),
                                        ctypes.c_void_p(_stream(P.device))), "cd_p2s_forward")
    return dist, fidx


def p2s_backward(P, V, F, fidx, g, want_points: bool = True, want_vertices: bool = True):
    """(gP [B, S, 3] or None, gV [B, nv, 3] or None) for g [B, S] = dL/d dist."""
    P, V, F = _p2s_args(P, V, F)
    B, S, nv, nf = P.shape[0], P.shape[1], V.shape[1], F.shape[1]
    fidx = _expect(fidx, "fidx", torch.int32, (B, S), P.device)
    g = _expect(g, "g", torch.float32, (B, S), P.device)
    gP = torch.empty((B, S, 3), dtype=torch.float32, device=P.device) if want_points else None
    gV = torch.empty((B, nv, 3), dtype=torch.float32, device=P.device) if want_vertices else None
    ws = _p2s_ws(B, S, nv, nf, P.device)
    with torch.cuda.device(P.device):
        _check(library().cd_p2s_backward(B, S, nv, nf, _ptr(P), _ptr(V), _ptr(F), _ptr(fidx),
                                         _ptr(g), _ptr(gP) if gP is not None else None,
                                         _ptr(gV) if gV is not None else None, _ptr(ws),
                                         ws.numel(), ctypes.c_void_p(_stream(P.device))),
               "cd_p2s_backward")
    return gP, gV


class PointToSurface(torch.autograd.Function):
    """dist [B, S] = squared distance of each point to the nearest face,
    differentiable in the points and the vertices (the face choice is not)."""

    @staticmethod
    def forward(ctx, P, V, F):
        dist, fidx = p2s_forward(P, V, F)
        ctx.save_for_backward(P, V, F, fidx)
        ctx.mark_non_differentiable(fidx)
        return dist, fidx

    @staticmethod
    def backward(ctx, g_dist, _g_fidx):
        P, V, F, fidx = ctx.saved_tensors
        gP, gV = p2s_backward(P, V, F, fidx, g_dist.contiguous().float(),
                              want_points=ctx.needs_input_grad[0],
                              want_vertices=ctx.needs_input_grad[1])
        return gP, gV, None


def point_to_surface(P, V, F):
    """Per-point squared distances [B, S] (autograd); the point-to-surface loss
    of Sec. 2.5 is their mean over the points."""
    return PointToSurface.apply(P, V, F)[0]


# ---------------------------------------------------------------- approximate EMD

def _emd_ws(B, N, M, device):
    need = int(library().cd_emd_workspace_bytes(B, N, M))
    return torch.empty(max(need, 1), dtype=torch.uint8, device=device)


def emd_forward(X, Y, eps_start: float = 0.5, eps_end: float = 0.01, n_iters: int = 50,
                g_init: Optional[torch.Tensor] = None):
    """(cost [B], f [B, N], g [B, M]): approximate EMD by scheduled log-domain
    Sinkhorn iterations (the schedule and updates are documented in cd.h)."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    f = torch.empty((B, N), dtype=torch.float32, device=X.device)
    if g_init is None:
        g = torch.empty((B, M), dtype=torch.float32, device=X.device)
    else:
        g = _expect(g_init, "g_init", torch.float32, (B, M), X.device).clone()
    cost = torch.empty(B, dtype=torch.float32, device=X.device)
    ws = _emd_ws(B, N, M, X.device)
    with torch.cuda.device(X.device):
        _check(library().cd_emd_forward(B, N, M, _ptr(X), _ptr(Y), float(eps_start),
                                        float(eps_end), int(n_iters), int(g_init is not None),
                                        _ptr(f), _ptr(g), _ptr(cost), _ptr(ws), ws.numel(),
                                        ctypes.c_void_p(_stream(X.device))), "cd_emd_forward")
    return cost, f, g


def emd_backward(X, Y, f, g, eps: float, grad_out):
    """(gX, gY) of sum_b grad_out[b] cost[b] with the plan held fixed."""
    X, Y = _clouds(X, Y)
    B, N, M = X.shape[0], X.shape[1], Y.shape[1]
    f = _expect(f, "f", torch.float32, (B, N), X.device)
    g = _expect(g, "g", torch.float32, (B, M), X.device)
    go = _expect(grad_out, "grad_out", torch.float32, (B,), X.device)
    gX = torch.empty_like(X)
    gY = torch.empty_like(Y)
    ws = _emd_ws(B, N, M, X.device)
    with torch.cuda.device(X.device):
        _check(library().cd_emd_backward(B, N, M, _ptr(X), _ptr(Y), _ptr(f), _ptr(g), float(eps),
                                         _ptr(go), _ptr(gX), _ptr(gY), _ptr(ws), ws.numel(),
                                         ctypes.c_void_p(_stream(X.device))), "cd_emd_backward")
    return gX, gY


class EarthMoversDistance(torch.autograd.Function):
    """Approximate EMD per item [B]; the backward holds the transport plan fixed."""

    @staticmethod
    def forward(ctx, X, Y, eps_start, eps_end, n_iters):
        cost, f, g = emd_forward(X, Y, eps_start, eps_end, n_iters)
        ctx.save_for_backward(X, Y, f, g)
        ctx.eps = eps_end
        return cost

    @staticmethod
    def backward(ctx, grad_out):
        X, Y, f, g = ctx.saved_tensors
        gX, gY = emd_backward(X, Y, f, g, ctx.eps, grad_out.contiguous().float())
        return gX, gY, None, None, None


def earth_movers_distance(X, Y, eps_start: float = 0.5, eps_end: float = 0.01, n_iters: int = 50):
    """Approximate EMD [B] between X [B, N, 3] and Y [B, M, 3] (autograd)."""
    return EarthMoversDistance.apply(X, Y, eps_start, eps_end, n_iters)
