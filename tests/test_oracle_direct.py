"""The fp64 direct-convolution oracle against its pins (CPU only)."""
import numpy as np
import pytest

import pins_direct
import pins_direct_rs
from oracle import direct


@pytest.mark.parametrize("check", pins_direct.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(check):
    check(direct.conv2d)


@pytest.mark.parametrize("check", pins_direct_rs.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin_rs(check):
    check(direct.conv2d)


def test_absval_bounds_the_output():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 3, 6, 7))
    g = rng.standard_normal((4, 3, 3, 3))
    y = direct.conv2d(x, g, 1)
    b = direct.conv2d(x, g, 1, absval=True)
    assert np.array_equal(b, direct.conv2d(np.abs(x), np.abs(g), 1))
    assert np.all(np.abs(y) <= b * (1 + 1e-15))


def test_rejects_bad_shapes():
    x = np.zeros((1, 2, 4, 4))
    with pytest.raises(ValueError):
        direct.conv2d(x, np.zeros((1, 3, 3, 3)), 1)      # channel mismatch
    with pytest.raises(ValueError):
        direct.conv2d(np.zeros((1, 1, 1, 1)), np.zeros((1, 1, 3, 3)), 0)   # Ho < 1
    with pytest.raises(ValueError):
        direct.conv2d(np.zeros((1, 1, 4, 4)), np.zeros((1, 1, 5, 5)), 0)   # Ho < 1 (5x5)
