"""The CPU oracle against its pins (hand-worked values, closed forms,
invariants, float64 brute force, float64 finite differences)."""
import pytest

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle)


def test_backward_matches_independent_numpy_scatter():
    # A second, independently written float64 backward (np.add.at scatters).
    import numpy as np
    import synth
    from oracle import check64
    X, Y = synth.generate("grid_dup", 2, 120, 90, 7)
    dxy, ixy, dyx, iyx = oracle.nn(X, Y)
    go = np.array([0.5, -2.0])
    gX, gY, *_ = oracle.backward(go, X, Y, ixy, iyx, 1.25, 0.5)
    rX, rY = check64.backward64(go, X, Y, ixy, iyx, 1.25, 0.5)
    assert np.allclose(gX, rX, rtol=1e-12, atol=1e-15)
    assert np.allclose(gY, rY, rtol=1e-12, atol=1e-15)


def test_oracle_rejects_bad_input():
    import numpy as np
    with pytest.raises(ValueError):
        oracle.nn_one_way(np.zeros((1, 3, 3), np.float32), np.zeros((1, 0, 3), np.float32))
    with pytest.raises(ValueError):
        oracle.nn_one_way(np.zeros((1, 3, 2), np.float32), np.zeros((1, 3, 2), np.float32))
    with pytest.raises(ValueError):
        oracle.backward([1.0], np.zeros((1, 2, 3), np.float32), np.zeros((1, 2, 3), np.float32),
                        np.array([[0, 2]]), np.array([[0, 0]]))
