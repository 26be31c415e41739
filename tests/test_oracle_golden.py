"""The oracle still reproduces its committed regression anchor (written by
``tests/golden/make_golden.py`` from the oracle alone). Float64 BLAS results
may differ in the last bits between CPUs, hence the tight relative bound."""

import json
import os

import numpy as np
import pytest

from tests.golden.make_golden import compute

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_dense784x100_seed0_anchor():
    with open(os.path.join(HERE, "dense784x100_seed0.json")) as f:
        want = json.load(f)
    got = compute()
    assert got.keys() == want.keys()
    assert got["relu_active"] == want["relu_active"]
    assert got["loss"] == pytest.approx(want["loss"], rel=1e-12)
    for k in ("h", "db", "dw", "dx", "new_w"):
        np.testing.assert_allclose(np.array(got[k]), np.array(want[k]), rtol=1e-6, atol=0)
