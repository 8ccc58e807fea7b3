"""Approximate-EMD oracle against its pins, and planted mistakes caught."""
import importlib.util
import os

import pytest

import emd_pins
from oracle import emd_oracle


@pytest.mark.parametrize("pin", emd_pins.ALL_PINS, ids=[p.__name__ for p in emd_pins.ALL_PINS])
def test_emd_oracle_pin(pin):
    pin(emd_oracle)


MUTATIONS = [
    ("squared instead of Euclidean cost", "return np.sqrt(((x[:, None, :] - y[None, :, :]) ** 2).sum(-1))",
     "return ((x[:, None, :] - y[None, :, :]) ** 2).sum(-1)"),
    ("masses swapped", "la, lb = -np.log(N), -np.log(M)", "la, lb = -np.log(M), -np.log(N)"),
    ("potential sign", "f = -e * _lse((g[None, :] - C) / e + lb, axis=1)",
     "f = e * _lse((g[None, :] - C) / e + lb, axis=1)"),
    ("plan without the masses", "return np.exp((np.asarray(f)[:, None] + np.asarray(g)[None, :] - C) / eps) / (N * M)",
     "return np.exp((np.asarray(f)[:, None] + np.asarray(g)[None, :] - C) / eps)"),
    ("schedule reversed", "return float(eps_start) * (float(eps_end) / float(eps_start)) ** t",
     "return float(eps_end) * (float(eps_start) / float(eps_end)) ** t"),
    ("gradient of Y with the wrong sign", "gY[b] = -grad_out[b] * (W[..., None] * diff).sum(0)",
     "gY[b] = grad_out[b] * (W[..., None] * diff).sum(0)"),
    ("gradient not divided by the distance", "W = np.divide(P, C, out=np.zeros_like(P), where=C > 0)",
     "W = P"),
    ("last g-update skipped", "            g = -e * _lse((f[:, None] - C) / e + la, axis=0)\n",
     "            g = g if e == eps[-1] else -e * _lse((f[:, None] - C) / e + la, axis=0)\n"),
]


# A planted mistake may overflow (the reversed schedule ends at the large eps
# with potentials of the small one): that is part of what makes it fail.
@pytest.mark.filterwarnings("ignore:overflow encountered:RuntimeWarning")
@pytest.mark.parametrize("desc,orig,mut", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_emd_mutant_is_caught(tmp_path, desc, orig, mut):
    with open(emd_oracle.__file__) as f:
        src = f.read()
    assert src.count(orig) == 1, f"mutation site for {desc!r} not unique"
    path = tmp_path / "emd_mut.py"
    path.write_text(src.replace(orig, mut))
    spec = importlib.util.spec_from_file_location("emd_mut", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    caught = []
    for pin in emd_pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches: {desc}"
