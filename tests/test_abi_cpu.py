"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/cd.h declares, and rejects bad arguments before it
enqueues anything (these calls never reach the HIP runtime)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cd.h")

CD_OK, CD_ERR_INVALID_ARG, CD_ERR_WORKSPACE, CD_ERR_HIP = 0, 1, 2, 3


@pytest.fixture(scope="module")
def lib():
    import paper_1911_05063_amd as cd
    if not os.path.exists(cd.LIB_PATH):
        from paper_1911_05063_amd import build
        build.build()
    return cd.library()


def declared_functions():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cd_[a-z_]+)\s*\(", text)))


def test_header_declares_the_path():
    names = declared_functions()
    for n in ("cd_forward", "cd_reduce", "cd_fscore", "cd_metrics", "cd_backward", "cd_backward_pointwise",
              "cd_workspace_bytes", "cd_status_string", "cd_last_error", "cd_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in cd.h but not exported"


def test_exported_symbols_are_unmangled_c():
    import subprocess
    import paper_1911_05063_amd as cd
    out = subprocess.run(["nm", "-D", "--defined-only", cd.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    for name in declared_functions():
        assert name in exported


def test_status_strings(lib):
    assert lib.cd_status_string(CD_OK) == b"CD_OK"
    assert lib.cd_status_string(CD_ERR_INVALID_ARG) == b"CD_ERR_INVALID_ARG"
    assert lib.cd_status_string(CD_ERR_WORKSPACE) == b"CD_ERR_WORKSPACE"
    assert lib.cd_status_string(CD_ERR_HIP) == b"CD_ERR_HIP"
    assert lib.cd_version().count(b".") == 2


def test_workspace_bytes(lib):
    ws = lib.cd_workspace_bytes(16, 16384, 16384)
    assert ws >= 8 * 16 * (16384 + 16384) and ws % 256 == 0
    assert lib.cd_workspace_bytes(0, 10, 10) == 0
    assert lib.cd_workspace_bytes(1, 0, 10) == 0
    assert lib.cd_workspace_bytes(-1, 10, 10) == 0
    assert lib.cd_workspace_bytes(1, 2 ** 31, 10) == 0
    assert lib.cd_workspace_bytes(3, 7, 5) >= 8 * 3 * 12


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails its checks


def fwd(lib, B, N, M, ptrs=(FAKE,) * 6, ws=FAKE, ws_bytes=1 << 30):
    return lib.cd_forward(B, N, M, *ptrs, ws, ws_bytes, None)


def test_noalloc_forward_checks_before_any_launch(lib):
    # cd_forward_noalloc takes no workspace: its static per-GPU array holds
    # CD_FORWARD_NOALLOC_MAX_BYTES.  Shapes whose keys need more are refused
    # before anything is launched (here without a GPU), with the sizes.
    assert lib.cd_workspace_bytes(1, 2 ** 22, 2 ** 22) == 64 << 20
    n = 2 ** 22 + 1
    assert lib.cd_forward_noalloc(1, n, n, *([FAKE] * 6), None) == CD_ERR_WORKSPACE
    err = lib.cd_last_error()
    assert b"cd_forward_noalloc" in err and b"67108864" in err
    assert lib.cd_forward_noalloc(3, 2 ** 21, 2 ** 21, *([FAKE] * 6), None) == CD_ERR_WORKSPACE
    assert lib.cd_forward_noalloc(1, 0, 5, *([FAKE] * 6), None) == CD_ERR_INVALID_ARG
    assert lib.cd_forward_noalloc(1, 5, 5, FAKE, None, *([FAKE] * 4), None) == CD_ERR_INVALID_ARG
    assert lib.cd_forward_noalloc(0, 5, 5, *([FAKE] * 6), None) == CD_OK
    with open(HEADER) as f:
        assert "#define CD_FORWARD_NOALLOC_MAX_BYTES ((size_t)64 << 20)" in f.read()


def test_forward_rejects_bad_shapes(lib):
    assert fwd(lib, -1, 4, 4) == CD_ERR_INVALID_ARG
    assert fwd(lib, 1, 0, 4) == CD_ERR_INVALID_ARG
    assert fwd(lib, 1, 4, 0) == CD_ERR_INVALID_ARG
    assert fwd(lib, 1, 2 ** 31, 4) == CD_ERR_INVALID_ARG
    assert fwd(lib, 1, 4, 2 ** 31) == CD_ERR_INVALID_ARG
    assert b"invalid argument" in lib.cd_last_error()


def test_forward_rejects_null_pointers(lib):
    for k in range(6):
        ptrs = [FAKE] * 6
        ptrs[k] = None
        assert fwd(lib, 2, 4, 4, ptrs=tuple(ptrs)) == CD_ERR_INVALID_ARG
    # B == 0 is a no-op even with NULL pointers.
    assert fwd(lib, 0, 4, 4, ptrs=(None,) * 6, ws=None, ws_bytes=0) == CD_OK


def test_forward_checks_workspace(lib):
    need = lib.cd_workspace_bytes(2, 100, 50)
    assert fwd(lib, 2, 100, 50, ws_bytes=need - 1) == CD_ERR_WORKSPACE
    assert b"workspace too small" in lib.cd_last_error()
    assert fwd(lib, 2, 100, 50, ws=None) == CD_ERR_WORKSPACE
    assert fwd(lib, 2, 100, 50, ws=ctypes.c_void_p(0x1010)) == CD_ERR_INVALID_ARG  # unaligned


def test_reduce_fscore_backward_reject_bad_args(lib):
    assert lib.cd_reduce(1, 0, 3, FAKE, FAKE, 1.0, 1.0, FAKE, None) == CD_ERR_INVALID_ARG
    assert lib.cd_reduce(1, 3, 3, None, FAKE, 1.0, 1.0, FAKE, None) == CD_ERR_INVALID_ARG
    assert lib.cd_reduce(0, 3, 3, None, None, 1.0, 1.0, None, None) == CD_OK
    assert lib.cd_fscore(1, 3, 3, FAKE, FAKE, -0.5, FAKE, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_fscore(1, 3, 3, FAKE, FAKE, float("nan"), FAKE, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_fscore(1, 3, 3, FAKE, FAKE, 0.1, None, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_fscore(0, 3, 3, None, None, 0.1, None, None, None, None) == CD_OK
    args = [FAKE] * 7
    for k in range(7):
        a = list(args)
        a[k] = None
        go, X, Y, ixy, iyx, gX, gY = a
        assert lib.cd_backward(1, 3, 3, go, 1.0, 1.0, X, Y, ixy, iyx, gX, gY, FAKE, 1 << 30,
                               None) == CD_ERR_INVALID_ARG
    assert lib.cd_backward(-2, 3, 3, *([FAKE] * 1), 1.0, 1.0, *([FAKE] * 6), FAKE, 1 << 30,
                           None) == CD_ERR_INVALID_ARG
    for k in range(8):
        a = [FAKE] * 8
        a[k] = None
        assert lib.cd_backward_pointwise(1, 3, 3, *a, FAKE, 1 << 30, None) == CD_ERR_INVALID_ARG
    need = lib.cd_backward_workspace_bytes(16, 16384, 16384)
    assert need > 0 and need % 256 == 0
    assert lib.cd_backward(16, 16384, 16384, *([FAKE] * 1), 1.0, 1.0, *([FAKE] * 6), FAKE,
                           need - 1, None) == CD_ERR_WORKSPACE
    assert lib.cd_backward_pointwise(4, 100000, 10000, *([FAKE] * 8), FAKE, 8,
                                     None) == CD_ERR_WORKSPACE
    assert lib.cd_backward_workspace_bytes(0, 3, 3) == 0
    assert lib.cd_backward_workspace_bytes(2, 0, 3) == 0
    # Bounded partials: a few hundred MB at most for the largest workloads.
    for B, N, M in ((16, 16384, 16384), (4, 100000, 10000), (8, 65536, 65536), (1, 10 ** 6, 10 ** 6)):
        assert lib.cd_backward_workspace_bytes(B, N, M) <= 400 << 20, (B, N, M)


def test_metrics_rejects_bad_args(lib):
    taus = (ctypes.c_float * 17)(*([0.1] * 17))
    tp = ctypes.cast(taus, ctypes.c_void_p)
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, tp, 0, FAKE, FAKE, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, tp, 17, FAKE, FAKE, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, None, 2, FAKE, FAKE, None, None, None) == CD_ERR_INVALID_ARG
    bad = (ctypes.c_float * 2)(0.1, float("nan"))
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, ctypes.cast(bad, ctypes.c_void_p), 2, FAKE, FAKE,
                          None, None, None) == CD_ERR_INVALID_ARG
    neg = (ctypes.c_float * 1)(-1.0)
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, ctypes.cast(neg, ctypes.c_void_p), 1, FAKE, FAKE,
                          None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, tp, 3, None, FAKE, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_metrics(1, 3, 3, FAKE, FAKE, 1.0, 1.0, tp, 3, FAKE, None, None, None, None) == CD_ERR_INVALID_ARG
    assert lib.cd_metrics(0, 3, 3, None, None, 1.0, 1.0, tp, 3, None, None, None, None, None) == CD_OK


def test_mesh_entry_points_reject_bad_args(lib):
    assert lib.cd_mesh_workspace_bytes(2, 30, 10, 100) >= 2 * 10 * 8
    assert lib.cd_mesh_workspace_bytes(2, 30, 0, 100) == 0
    assert lib.cd_mesh_workspace_bytes(-1, 30, 10, 100) == 0
    # Chunked backward: partial sums for every chunk, bounded whatever S is.
    assert lib.cd_mesh_workspace_bytes(16, 600, 200, 16384) >= 16 * 2 * 600 * 24
    for nv in (1, 600, 2048, 2049, 10 ** 6):
        for B in (1, 3, 16):
            w = lib.cd_mesh_workspace_bytes(B, nv, 10, (2 ** 31 - 1) // B)
            assert 0 < w <= (48 << 20) + 256 and w % 256 == 0
    assert lib.cd_mesh_workspace_bytes(2, 30, 10, 2 ** 30 + 1) == 0      # B * S > 2^31
    # The backward's chunks (24 B per vertex and chunk when an item has more
    # than one): about one workgroup per CU, up to two where the chunks then
    # hold at most 2048 samples, chunk lengths a multiple of 512.
    assert lib.cd_mesh_workspace_bytes(16, 600, 200, 16384) == 16 * 16 * 600 * 24   # 16 x 1024
    assert lib.cd_mesh_workspace_bytes(64, 300, 200, 16000) == 64 * 8 * 300 * 24   # 8 x 2048
    assert lib.cd_mesh_workspace_bytes(4, 3000, 5000, 100000) == 4 * 49 * 3000 * 24  # 2 slices, 49 x 2048
    assert lib.cd_mesh_workspace_bytes(1, 100, 50, 300000) == (196 * 100 * 24 + 255) // 256 * 256
    assert lib.cd_mesh_workspace_bytes(600, 50, 30, 3000) == (600 * 30 * 8 + 255) // 256 * 256  # one chunk
    ws = FAKE
    assert lib.cd_mesh_sample_faces(1, 0, 4, FAKE, FAKE, 5, FAKE, FAKE, ws, 1 << 20, None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_faces(1, 3, 0, FAKE, FAKE, 5, FAKE, FAKE, ws, 1 << 20, None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_faces(1, 3, 4, FAKE, FAKE, -1, FAKE, FAKE, ws, 1 << 20, None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_faces(4, 3, 4, FAKE, FAKE, 2 ** 29 + 1, FAKE, FAKE, ws, 1 << 40,
                                    None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_faces(1, 3, 4, None, FAKE, 5, FAKE, FAKE, ws, 1 << 20, None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_faces(1, 3, 4, FAKE, FAKE, 5, FAKE, FAKE, ws, 8, None) == CD_ERR_WORKSPACE
    assert lib.cd_mesh_sample_faces(0, 3, 4, None, None, 5, None, None, None, 0, None) == CD_OK
    for k in range(6):
        a = [FAKE] * 6
        a[k] = None
        V, F, fi, r1, r2, P = a
        assert lib.cd_mesh_sample_points(1, 3, 4, V, F, 5, fi, r1, r2, P, None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_points(1, 3, 4, None, None, 0, None, None, None, None, None) == CD_OK
    for k in range(6):
        a = [FAKE] * 6
        a[k] = None
        F, fi, r1, r2, gP, gV = a
        assert lib.cd_mesh_sample_backward(1, 3, 4, F, 5, fi, r1, r2, gP, gV, ws, 1 << 20,
                                           None) == CD_ERR_INVALID_ARG
    need = lib.cd_mesh_workspace_bytes(4, 600, 200, 16384)
    assert lib.cd_mesh_sample_backward(4, 600, 200, FAKE, 16384, FAKE, FAKE, FAKE, FAKE, FAKE, ws,
                                       need - 1, None) == CD_ERR_WORKSPACE


def test_binding_refuses_cpu_tensors():
    import torch
    import paper_1911_05063_amd as cd
    X = torch.zeros(1, 4, 3)
    with pytest.raises(ValueError, match="ROCm GPU"):
        cd.nn_distance(X, X)
    with pytest.raises(ValueError, match="ROCm GPU"):
        cd.chamfer_distance(X, X)


def test_product_path_does_not_touch_the_oracle():
    # The package sources never import, load or execute anything under oracle/.
    pkg = os.path.join(ROOT, "paper_1911_05063_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".cpp", ".h")):
                with open(os.path.join(dirpath, fn)) as f:
                    src = f.read()
                assert "oracle" not in src.replace("oracle-free", ""), fn


def test_p2s_entry_points_reject_bad_args(lib):
    assert lib.cd_p2s_workspace_bytes(2, 100, 30, 10) > 0
    assert lib.cd_p2s_workspace_bytes(2, 100, 30, 0) == 0
    assert lib.cd_p2s_workspace_bytes(2, -1, 30, 10) == 0
    assert lib.cd_p2s_workspace_bytes(2, 2 ** 30 + 1, 30, 10) == 0       # B * S > 2^31
    assert lib.cd_p2s_workspace_bytes(16, 16384, 2562, 5120) % 256 == 0
    ws = FAKE
    for k in range(5):
        a = [FAKE] * 5
        a[k] = None
        P, V, F, d, fi = a
        assert lib.cd_p2s_forward(1, 5, 3, 1, P, V, F, d, fi, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_p2s_forward(1, 5, 0, 1, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_p2s_forward(1, 5, 3, 1, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 8, None) == CD_ERR_WORKSPACE
    assert lib.cd_p2s_forward(0, 5, 3, 1, None, None, None, None, None, None, 0, None) == CD_OK
    assert lib.cd_p2s_forward(2, 0, 3, 1, None, None, None, None, None, None, 0, None) == CD_OK
    assert lib.cd_p2s_backward(1, 5, 3, 1, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, ws, 1 << 30,
                               None) == CD_OK                                  # nothing asked
    assert lib.cd_p2s_backward(1, 5, 3, 1, FAKE, FAKE, FAKE, None, FAKE, FAKE, None, ws, 1 << 30,
                               None) == CD_ERR_INVALID_ARG
    assert lib.cd_p2s_backward(1, 5, 3, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 8,
                               None) == CD_ERR_WORKSPACE


def test_emd_entry_points_reject_bad_args(lib):
    assert lib.cd_emd_workspace_bytes(2, 100, 50) > 0
    assert lib.cd_emd_workspace_bytes(0, 100, 50) == 0
    assert lib.cd_emd_workspace_bytes(2, 0, 50) == 0
    ws = FAKE
    ok_args = (FAKE, FAKE, 0.5, 0.01, 10, 0, FAKE, FAKE, FAKE, ws, 1 << 30, None)
    assert lib.cd_emd_forward(1, 5, 5, FAKE, FAKE, 0.0, 0.01, 10, 0, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_forward(1, 5, 5, FAKE, FAKE, 0.5, float("nan"), 10, 0, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_forward(1, 5, 5, FAKE, FAKE, 0.5, 0.01, 0, 0, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_forward(1, 0, 5, *ok_args) == CD_ERR_INVALID_ARG
    for k in (0, 1, 6, 7, 8):
        a = list(ok_args)
        a[k] = None
        assert lib.cd_emd_forward(1, 5, 5, *a) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_forward(1, 5, 5, FAKE, FAKE, 0.5, 0.01, 10, 0, FAKE, FAKE, FAKE, ws, 8, None) == CD_ERR_WORKSPACE
    assert lib.cd_emd_forward(0, 5, 5, None, None, 0.5, 0.01, 10, 0, None, None, None, None, 0, None) == CD_OK
    assert lib.cd_emd_backward(1, 5, 5, FAKE, FAKE, FAKE, FAKE, -1.0, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_backward(1, 5, 5, FAKE, FAKE, FAKE, None, 0.1, FAKE, FAKE, FAKE, ws, 1 << 30, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_backward(1, 5, 5, FAKE, FAKE, FAKE, FAKE, 0.1, FAKE, FAKE, FAKE, ws, 8, None) == CD_ERR_WORKSPACE


def test_launch_size_limits(lib):
    # One thread per point of both clouds must fit a launch.
    assert lib.cd_workspace_bytes(1, 2 ** 30, 2 ** 30) > 0
    assert lib.cd_workspace_bytes(2, 2 ** 30, 2 ** 30) == 0
    assert lib.cd_workspace_bytes(4, 2 ** 29, 2 ** 29 + 1) == 0
    assert lib.cd_backward_workspace_bytes(2, 2 ** 30, 2 ** 30) == 0
    assert lib.cd_forward(2, 2 ** 30, 2 ** 30, *([FAKE] * 6), FAKE, 1 << 40, None) == CD_ERR_INVALID_ARG
    # The EMD gradient merge: one thread per component, 3 B max(N, M) < 2^32.
    assert lib.cd_emd_forward(1, 2 ** 30 + 2 ** 29, 10, FAKE, FAKE, 0.5, 0.01, 1, 0, FAKE, FAKE, FAKE,
                              FAKE, 1 << 40, None) == CD_ERR_INVALID_ARG


C_CLIENT = r"""
#include <stdio.h>
#include "cd.h"
int main(void)
{
    /* Pure argument checks and sizes: no device work, so no GPU is needed. */
    size_t ws = cd_workspace_bytes(16, 16384, 16384);
    cd_status s = cd_forward(1, 0, 5, 0, 0, 0, 0, 0, 0, 0, 0, 0);
    printf("%s %s %d %s\n", cd_version(), cd_status_string(s), ws > 0, cd_last_error());
    return s == CD_ERR_INVALID_ARG && ws > 0 ? 0 : 1;
}
"""


@pytest.mark.parametrize("compiler,std", [("gcc", "-std=c99"), ("g++", "-std=c++17")])
def test_header_builds_a_c_and_cpp_client(lib, tmp_path, compiler, std):
    """include/cd.h compiles as C and C++, and a client linked against the
    library calls it (argument checks only)."""
    import shutil
    import subprocess
    import paper_1911_05063_amd as cd
    if shutil.which(compiler) is None:
        pytest.skip(f"{compiler} not available")
    src = tmp_path / ("client.c" if compiler == "gcc" else "client.cpp")
    src.write_text(C_CLIENT)
    exe = tmp_path / "client"
    libdir = os.path.dirname(cd.LIB_PATH)
    cmd = [compiler, std, "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
           str(src), "-o", str(exe), f"-L{libdir}", "-lcd_hip", f"-Wl,-rpath,{libdir}"]
    if compiler == "gcc":
        cmd.insert(1, "-x")
        cmd.insert(2, "c")
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "CD_ERR_INVALID_ARG" in r.stdout and "N < 1" in r.stdout


def test_huge_batch_counts_are_rejected_without_overflow(lib):
    # B * S (and the like) would wrap around int64 here; the checks must not form it.
    big = 2 ** 62
    assert lib.cd_workspace_bytes(big, 2 ** 30, 2 ** 30) == 0
    assert lib.cd_mesh_workspace_bytes(big, 30, 10, 2 ** 31 - 1) == 0
    assert lib.cd_mesh_workspace_bytes(big, 2 ** 31 - 1, 10, 0) == 0
    assert lib.cd_p2s_workspace_bytes(big, 2 ** 31 - 1, 30, 10) == 0
    assert lib.cd_p2s_workspace_bytes(big, 0, 30, 2 ** 31 - 1) == 0
    assert lib.cd_emd_workspace_bytes(big, 2 ** 30, 4) == 0
    assert lib.cd_emd_forward(big, 4, 2 ** 31 - 1, FAKE, FAKE, 0.5, 0.01, 1, 0, FAKE, FAKE, FAKE,
                              FAKE, 1 << 40, None) == CD_ERR_INVALID_ARG
    assert lib.cd_emd_backward(big, 4, 2 ** 31 - 1, FAKE, FAKE, FAKE, FAKE, 0.1, FAKE, FAKE, FAKE,
                               FAKE, 1 << 40, None) == CD_ERR_INVALID_ARG
    assert lib.cd_p2s_forward(big, 2 ** 31 - 1, 3, 1, *([FAKE] * 5), FAKE, 1 << 40,
                              None) == CD_ERR_INVALID_ARG
    assert lib.cd_mesh_sample_points(big, 3, 4, FAKE, FAKE, 2 ** 31 - 1, FAKE, FAKE, FAKE, FAKE,
                                     None) == CD_ERR_INVALID_ARG


def _backward_plan_bytes(B, N, M):
    """The backward's workspace for its plan, restated: the direct scan (slices
    of up to 2048 receivers that scan all senders; per-block bounds, shifts
    and chunk partials) or, where the direct scan would need the bound pass
    (senders beyond one pass of 16384) or its repeated index scans would read
    64 MB or more, senders bucketed by slice (4 bytes per sender slot in
    chunks of 2048, and each chunk's slice offsets)."""
    import math
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    s = 2048
    while s > 256 and 2 * B * (math.ceil(N / s) + math.ceil(M / s)) <= 256:
        s //= 2
    n_recv, n_send = (N, M), (M, N)
    ns = [math.ceil(r / s) for r in n_recv]
    nch = [math.ceil(q / 2048) for q in n_send]
    feasible = all(n <= 1024 and c <= 1024 and math.ceil(q / n) <= 16384
                   for n, c, q in zip(ns, nch, n_send))
    rounds = [math.ceil(q / 16384) for q in n_send]
    target = min(rounds)
    nc, local = [], []
    for r, q in zip(rounds, n_send):
        chunk = math.ceil(r / math.ceil(r / target)) * 16384
        nc.append(math.ceil(q / chunk))
        local.append(nc[-1] == 1 and q <= 16384)
    scan = 4 * B * (ns[0] * n_send[0] + ns[1] * n_send[1])
    bucketed = feasible and (not all(local) or scan >= 64 << 20)
    if bucketed:
        return True, up(4 * B * 2048 * sum(nch)) + up(4 * B * sum(c * (n + 1) for c, n in zip(nch, ns)))
    nblk = math.ceil(max(N, M) / 1024)
    parts = sum(B * c * r * 3 for c, r in zip(nc, n_recv) if c > 1)
    return False, up(B * nblk * 8 * 4) + up(B * 2 * 4) + up(parts * 8)


def test_backward_workspace_follows_its_plan(lib):
    # Bucketed where the direct scan would need the bound pass or would re-read
    # 64 MB or more of indices (and every slice's share stays small); the
    # direct scan otherwise.  Either way the workspace is what the plan needs.
    cases = {(8, 65536, 65536): True, (4, 65536, 65536): True, (1, 200000, 180000): True,
             (4, 70000, 65536): True, (1, 2 ** 20, 2 ** 20): True, (2, 2 ** 21, 2 ** 21): True,
             (4, 20000, 30000): True, (16, 16385, 16384): True, (16, 20000, 20000): True,
             (16, 16384, 16384): False, (4, 100000, 10000): False, (32, 2048, 2048): False,
             (1, 1024, 1024): False, (1, 300000, 700): False, (2, 5000, 90000): False,
             (32, 4096, 40000): False}
    import random
    rng = random.Random(9)
    for _ in range(200):
        cases.setdefault((rng.randint(1, 32), rng.randint(1, 120000), rng.randint(1, 120000)), None)
    for (B, N, M), want_bucketed in cases.items():
        bucketed, want = _backward_plan_bytes(B, N, M)
        if want_bucketed is not None:
            assert bucketed == want_bucketed, (B, N, M)
        assert lib.cd_backward_workspace_bytes(B, N, M) == want, (B, N, M, bucketed)


def test_forward_workspace_is_linear_in_the_clouds(lib):
    # The forward keeps one 8-byte key per point of each cloud (tiles fold
    # into them with atomic minima), whatever the planner's tiling: 8 B N and
    # 8 B M bytes, each rounded up to 256.  The backward's workspace is
    # nonzero and aligned for the same shapes.
    import random
    rng = random.Random(5)
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    shapes = [(1, 1, 1), (1, 1024, 1024), (32, 2048, 2048), (16, 16384, 16384),
              (4, 100000, 10000), (8, 65536, 65536), (600, 40, 50), (1, 300000, 1),
              (1, 2 ** 20, 2 ** 20), (1, 2 ** 22, 2 ** 22), (1, 2 ** 30, 2 ** 30)]
    shapes += [(rng.randint(1, 64), rng.randint(1, 70000), rng.randint(1, 70000)) for _ in range(300)]
    for B, N, M in shapes:
        ws = lib.cd_workspace_bytes(B, N, M)
        assert ws == up(8 * B * N) + up(8 * B * M), (B, N, M, ws)
        assert ws <= 8 * B * (N + M) + 512
        bw = lib.cd_backward_workspace_bytes(B, N, M)
        assert bw > 0 and bw % 256 == 0, (B, N, M, bw)
