"""cd_forward_noalloc (static per-GPU workspace) against cd_forward, through
the C ABI: two calls in a row, the second on a smaller problem, each bitwise
equal to cd_forward on the same inputs (and to the oracle in the kernel's
precision)."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
import synth
import gpu_checks as gc

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no ROCm GPU visible")
    import paper_1911_05063_amd as cd
    assert os.path.exists(cd.LIB_PATH), "libcd_hip.so missing: build before running GPU tests"
    return cd.library()


def _outputs(B, N, M):
    dev = "cuda:0"
    return (torch.empty((B, N), dtype=torch.float32, device=dev),
            torch.empty((B, N), dtype=torch.int32, device=dev),
            torch.empty((B, M), dtype=torch.float32, device=dev),
            torch.empty((B, M), dtype=torch.int32, device=dev))


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def test_noalloc_forward_matches_forward_twice(lib):
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # Larger first, then smaller: the second call must not see the first's keys.
    for kind, B, N, M, seed in (("mesh", 3, 5000, 7001, 21), ("grid_dup", 2, 1000, 300, 22)):
        print(f"[noalloc] {kind} B={B} N={N} M={M}", flush=True)
        X, Y = synth.generate(kind, B, N, M, seed)
        Xg, Yg = gc.to_gpu(X), gc.to_gpu(Y)
        ws_bytes = int(lib.cd_workspace_bytes(B, N, M))
        assert 0 < ws_bytes <= (64 << 20)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda:0")
        ref = _outputs(B, N, M)
        got = _outputs(B, N, M)
        st = lib.cd_forward(B, N, M, _p(Xg), _p(Yg), *[_p(t) for t in ref], _p(ws), ws_bytes,
                            stream)
        assert st == 0, lib.cd_last_error()
        st = lib.cd_forward_noalloc(B, N, M, _p(Xg), _p(Yg), *[_p(t) for t in got], stream)
        assert st == 0, lib.cd_last_error()
        torch.cuda.synchronize()
        for a, b in zip(got, ref):
            assert torch.equal(a, b)
        gc.assert_nn_bitwise(tuple(gc.to_np(t) for t in got), oracle.nn(X, Y, fused=True),
                             f"noalloc {kind}")
