"""The Python example of README.md runs as written on the GPU."""
import os
import re

import pytest
import torch

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_readme_example_runs():
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, flags=re.S)
    assert blocks, "no python example in README.md"
    scope = {}
    exec(compile(blocks[0], "README.md", "exec"), scope)
    torch.cuda.synchronize()
    B = 16
    assert scope["loss"].shape == (B,) and scope["X"].grad.shape == (B, 16384, 3)
    assert scope["f"].shape == (3, B) and scope["P"].shape == (B, 16384, 3)
    assert scope["d"].shape == (B, 16384) and scope["emd"].shape == (B,)
    for k in ("loss", "chamfer", "d", "emd"):
        assert bool(torch.isfinite(scope[k]).all()), k
