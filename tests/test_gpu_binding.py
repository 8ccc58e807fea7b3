"""The Python binding refuses arrays whose shapes do not match the problem
(the kernels index every array by the sizes they are given), before any
launch."""
import pytest
import torch

import paper_1911_05063_amd as cd

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def f32(*shape):
    return torch.zeros(shape, dtype=torch.float32, device=DEV)


def i32(*shape):
    return torch.zeros(shape, dtype=torch.int32, device=DEV)


def test_chamfer_calls_check_shapes():
    X, Y = f32(2, 5, 3), f32(2, 7, 3)
    with pytest.raises(ValueError):
        cd.nn_distance(X, f32(3, 7, 3))
    with pytest.raises(ValueError):
        cd.nn_distance(X, Y, workspace=torch.zeros(64, dtype=torch.uint8, device="cpu"))
    with pytest.raises(ValueError):
        cd.chamfer_reduce(f32(2, 5), f32(3, 7))
    with pytest.raises(ValueError):
        cd.f_score(f32(2, 5), f32(14), 0.1)
    with pytest.raises(ValueError):
        cd.metrics(f32(10), f32(2, 7), [0.1])
    good = dict(grad_out=f32(2), idx_xy=i32(2, 5), idx_yx=i32(2, 7))
    for key, bad in (("grad_out", f32(1)), ("idx_xy", i32(2, 4)), ("idx_yx", i32(2, 5, 1))):
        args = dict(good, **{key: bad})
        with pytest.raises(ValueError):
            cd.chamfer_backward(args["grad_out"], X, Y, args["idx_xy"], args["idx_yx"])
    with pytest.raises(ValueError):
        cd.chamfer_backward_pointwise(f32(2, 5), f32(2, 6), X, Y, i32(2, 5), i32(2, 7))
    with pytest.raises(ValueError):
        cd.chamfer_backward(f32(2), X, f32(1, 7, 3), i32(2, 5), i32(2, 7))


def test_mesh_p2s_emd_calls_check_shapes():
    V, F = f32(2, 4, 3), i32(2, 2, 3)
    with pytest.raises(ValueError):
        cd.mesh_sample_faces(V, F, f32(1, 10))
    with pytest.raises(ValueError):
        cd.mesh_sample_points(V, F, i32(2, 10), f32(2, 10), f32(2, 9))
    with pytest.raises(ValueError):
        cd.mesh_sample_backward(4, F, i32(2, 10), f32(2, 10), f32(2, 10), f32(2, 10, 2))
    P = f32(2, 6, 3)
    with pytest.raises(ValueError):
        cd.p2s_backward(P, V, F, i32(2, 6), f32(2, 5))
    with pytest.raises(ValueError):
        cd.p2s_backward(P, V, F, i32(1, 6), f32(2, 6))
    X, Y = f32(2, 5, 3), f32(2, 7, 3)
    with pytest.raises(ValueError):
        cd.emd_forward(X, Y, g_init=f32(2, 5))
    with pytest.raises(ValueError):
        cd.emd_backward(X, Y, f32(2, 5), f32(2, 7), 0.1, f32(3))
    with pytest.raises(ValueError):
        cd.emd_backward(X, Y, f32(2, 7), f32(2, 7), 0.1, f32(2))
