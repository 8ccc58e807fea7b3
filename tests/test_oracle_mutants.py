"""Pin strength: plant plausible mistakes in a copy of the C oracle and check
that at least one pin catches each of them.  Mutants are built on the CPU in
a temporary directory; the real oracle is never modified."""
import importlib.util
import os
import subprocess

import pytest

import oracle
import oracle_pins

# (description, original text, mutated text); each original must occur once.
MUTATIONS = [
    ("wrong sign in dx", "float dx = p[0] - q[0];", "float dx = p[0] + q[0];"),
    ("wrong coordinate index", "float dz = p[2] - q[2];", "float dz = p[2] - q[1];"),
    ("dropped z term", "return sxy + dz * dz;", "return sxy;"),
    ("unsquared term", "float sxy = dx * dx + dy * dy;", "float sxy = dx * dx + dy;"),
    ("transposed product in fused form", "fmaf(dy, dy, dx * dx)", "fmaf(dy, dx, dx * dx)"),
    ("tie keeps the last index", "if (d < best) {", "if (d <= best) {"),
    ("target stride uses the query count", "const float *qb = Q + 3 * b * NQ;",
     "const float *qb = Q + 3 * b * NP;"),
    ("means swapped", "out[b] = w1 * (sx / (double)N) + w2 * (sy / (double)M);",
     "out[b] = w1 * (sx / (double)M) + w2 * (sy / (double)N);"),
    ("one direction dropped", "out[b] = w1 * (sx / (double)N) + w2 * (sy / (double)M);",
     "out[b] = w1 * (sx / (double)N);"),
    ("non-strict threshold", "cp += ((double)dist_xy[b * N + i] < t2) ? 1 : 0;",
     "cp += ((double)dist_xy[b * N + i] <= t2) ? 1 : 0;"),
    ("harmonic mean without the 2", "f[b] = (P + R > 0.0) ? (2.0 * P * R) / (P + R) : 0.0;",
     "f[b] = (P + R > 0.0) ? (P * R) / (P + R) : 0.0;"),
    ("precision and recall swapped", "double P = (double)cp / (double)N;",
     "double P = (double)cp / (double)M;"),
    ("scatter sign flipped", "gY[(b * M + j) * 3 + c] -= term;", "gY[(b * M + j) * 3 + c] += term;"),
    ("missing factor 2", "double diff = (double)Y[(b * M + j) * 3 + c] - (double)X[(b * N + i) * 3 + c];\n"
     "                double term = 2.0 * g * diff;",
     "double diff = (double)Y[(b * M + j) * 3 + c] - (double)X[(b * N + i) * 3 + c];\n"
     "                double term = g * diff;"),
    ("scatter to the wrong point", "gX[(b * N + i) * 3 + c] -= term;", "gX[(b * N + j % N) * 3 + c] -= term;"),
]


def _mutant_module(tmp_path, name, src):
    c_path = tmp_path / f"{name}.c"
    so_path = tmp_path / f"{name}.so"
    c_path.write_text(src)
    srcs = [str(c_path) if os.path.basename(x) == "cd_oracle.c" else x for x in oracle.SOURCES]
    subprocess.run(["gcc", "-O1", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    *srcs, "-o", str(so_path), "-lm"], check=True)
    spec = importlib.util.spec_from_file_location(f"oracle_{name}", oracle.__file__)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod.LIB_PATH = str(so_path)
    mod._lib = None
    return mod


@pytest.mark.parametrize("desc,orig,mut", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutant_is_caught(tmp_path, desc, orig, mut):
    with open(os.path.join(os.path.dirname(oracle.__file__), "cd_oracle.c")) as f:
        src = f.read()
    assert src.count(orig) == 1, f"mutation site for {desc!r} not unique"
    mod = _mutant_module(tmp_path, "m", src.replace(orig, mut))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {desc}"


def test_unmutated_copy_passes(tmp_path):
    with open(os.path.join(os.path.dirname(oracle.__file__), "cd_oracle.c")) as f:
        mod = _mutant_module(tmp_path, "same", f.read())
    for pin in oracle_pins.ALL_PINS:
        pin(mod)
