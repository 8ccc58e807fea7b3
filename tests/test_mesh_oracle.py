"""The mesh-sampling oracle against its pins, and pin strength by mutation."""
import importlib.util
import os
import subprocess

import numpy as np
import pytest

import oracle
import mesh_pins


@pytest.mark.parametrize("pin", mesh_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_mesh_oracle_pin(pin):
    pin(oracle)


def test_mesh_oracle_rejects_bad_input():
    V = np.zeros((1, 3, 3), np.float32)
    with pytest.raises(ValueError):
        oracle.face_areas(V, np.array([[[0, 1, 3]]], np.int32))
    with pytest.raises(ValueError):
        oracle.sample_points(V, np.array([[[0, 1, 2]]], np.int32), np.array([[1]]),
                             np.zeros((1, 1)), np.zeros((1, 1)))


MUTATIONS = [
    ("weights of b and c swapped", "w[1] = s1 * (1.0 - r2);\n    w[2] = s1 * r2;",
     "w[1] = s1 * r2;\n    w[2] = s1 * (1.0 - r2);"),
    ("no square root", "const double s1 = sqrt(r1);", "const double s1 = r1;"),
    ("non-strict face choice", "if (target < cdf) {", "if (target <= cdf) {"),
    ("area without the half", "area[b * nf + f] = 0.5 * sqrt(cx * cx + cy * cy + cz * cz);",
     "area[b * nf + f] = sqrt(cx * cx + cy * cy + cz * cz);"),
    ("cross product sign slip", "const double cy = e1[2] * e2[0] - e1[0] * e2[2];",
     "const double cy = e1[2] * e2[0] + e1[0] * e2[2];"),
    ("gradient to the wrong vertex", "const int64_t v = b * nv + tri[i];",
     "const int64_t v = b * nv + tri[(i + 1) % 3];"),
    ("gradient without the weight", "const double term = w[i] * gP[k * 3 + c];",
     "const double term = gP[k * 3 + c];"),
]


@pytest.mark.parametrize("desc,orig,mut", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mesh_mutant_is_caught(tmp_path, desc, orig, mut):
    here = os.path.dirname(oracle.__file__)
    with open(os.path.join(here, "mesh_oracle.c")) as f:
        src = f.read()
    assert src.count(orig) == 1, f"mutation site for {desc!r} not unique"
    c_path = tmp_path / "mesh_mut.c"
    c_path.write_text(src.replace(orig, mut))
    so_path = tmp_path / "mut.so"
    srcs = [str(c_path) if os.path.basename(x) == "mesh_oracle.c" else x for x in oracle.SOURCES]
    subprocess.run(["gcc", "-O1", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    *srcs, "-o", str(so_path), "-lm"], check=True)
    spec = importlib.util.spec_from_file_location("oracle_mesh_mut", oracle.__file__)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod.LIB_PATH = str(so_path)
    mod._lib = None
    caught = []
    for pin in mesh_pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {desc}"
