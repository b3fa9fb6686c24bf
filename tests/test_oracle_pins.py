"""The CPU oracle against the paper's fixed facts and independent routines."""
import pytest

import oracle
import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.default())


def test_inverse_triangular_solve_full_image():
    """One 16x16x12 image (N = 3072 unknowns) against scipy solve_triangular."""
    pins.pin_inverse_triangular_solve(oracle.default(), big=True)


def test_golden_regression():
    """The oracle still reproduces the committed 8x8x3 fixture (written by
    tests/golden/make_golden.py from the oracle alone)."""
    import json
    import os

    import numpy as np

    from paper_2301_09266_amd import synth

    rec = json.load(open(os.path.join(pins.GOLDEN, "layer_c3_8x8_b1_k3_tl.json")))
    c = synth.make("layer_c3_8x8_b1_k3")
    assert np.array_equal(np.array(rec["x"]), c["x"].ravel())
    assert np.array_equal(np.array(rec["K"]), c["K"].ravel())
    o = oracle.default()
    np.testing.assert_allclose(o.forward(c["x"], c["K"], 0).ravel(), rec["y"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(o.inverse(c["z"], c["K"], 0).ravel(), rec["inv_z"], rtol=0,
                               atol=1e-12)
    assert abs(o.logdet(c["K"], 0, 8, 8) - rec["logdet"]) < 1e-12
