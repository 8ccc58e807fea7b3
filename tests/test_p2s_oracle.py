"""Point-to-surface oracle against its pins, and planted mistakes caught."""
import importlib.util
import os
import subprocess

import pytest

import oracle
import p2s_pins


@pytest.mark.parametrize("pin", p2s_pins.ALL_PINS, ids=[p.__name__ for p in p2s_pins.ALL_PINS])
def test_p2s_oracle_pin(pin):
    pin(oracle)


MUTATIONS = [
    ("first sub-triangle oriented the wrong way", "        sub3(c, b, x);\n        sub3(q, b, y);",
     "        sub3(b, c, x);\n        sub3(q, b, y);"),
    ("plane distance without |n|^2", "return h * h * nn;", "return h * h;"),
    ("segment not clamped at its end", "    if (s > 1.0) s = 1.0;\n", ""),
    ("edge bc parameters swapped", "        w[1] = 1.0 - t;\n        w[2] = t;",
     "        w[1] = t;\n        w[2] = 1.0 - t;"),
    ("barycentric of c from the wrong edge", "        sub3(b, a, x);\n        sub3(q, a, y);",
     "        sub3(c, a, x);\n        sub3(q, a, y);"),
    ("ties to the last face", "                if (d < best) {\n                    best = d;\n                    arg",
     "                if (d <= best) {\n                    best = d;\n                    arg"),
    ("point gradient sign", "gP[3 * k + i] = 2.0 * g[k] * (p[i] - q[i]);",
     "gP[3 * k + i] = 2.0 * g[k] * (q[i] - p[i]);"),
    ("vertex gradient to the wrong corner", "const double term = -2.0 * g[k] * w[j] * (p[i] - q[i]);",
     "const double term = -2.0 * g[k] * w[(j + 1) % 3] * (p[i] - q[i]);"),
    ("edge ca skipped", "    d = seg_dist2(p, c, a, &t);\n    if (d < best) {",
     "    d = seg_dist2(p, c, a, &t);\n    if (0) {"),
]


@pytest.mark.parametrize("desc,orig,mut", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_p2s_mutant_is_caught(tmp_path, desc, orig, mut):
    here = os.path.dirname(oracle.__file__)
    with open(os.path.join(here, "p2s_oracle.c")) as f:
        src = f.read()
    assert src.count(orig) == 1, f"mutation site for {desc!r} not unique"
    c_path = tmp_path / "p2s_mut.c"
    c_path.write_text(src.replace(orig, mut))
    so_path = tmp_path / "mut.so"
    srcs = [str(c_path) if os.path.basename(x) == "p2s_oracle.c" else x for x in oracle.SOURCES]
    subprocess.run(["gcc", "-O1", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    *srcs, "-o", str(so_path), "-lm"], check=True)
    spec = importlib.util.spec_from_file_location("oracle_p2s_mut", oracle.__file__)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod.LIB_PATH = str(so_path)
    mod._lib = None
    caught = []
    for pin in p2s_pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {desc}"
