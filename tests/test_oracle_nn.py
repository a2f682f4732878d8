"""Pins for the oracle's stack glue (``oracle/nn.py``): ReLU and 2x2/2 max-pool.

These are the references for the max-pool kernel and for every layer-stack
check (the VGG-16 and ResNet-style stacks stand in for the networks of the
paper's evaluation, Sec. 3).  Each check below uses hand-worked values, not the
oracle's own formula; plausible mistakes planted in copies of the source must
fail at least one check (CPU only).
"""
import os
import types

import numpy as np
import pytest

from oracle import nn

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "nn.py")


def check_relu_signs(relu, maxpool):
    x = np.array([-3.5, -1e-300, -0.0, 0.0, 1e-300, 2.25, np.inf, -np.inf])
    y = relu(x)
    assert y.shape == x.shape
    assert np.array_equal(y, [0.0, 0.0, 0.0, 0.0, 1e-300, 2.25, np.inf, 0.0])


def check_relu_keeps_shape_and_positives(relu, maxpool):
    x = np.arange(-12.0, 12.0).reshape(1, 2, 3, 4)
    y = relu(x)
    assert y.shape == (1, 2, 3, 4)
    assert np.array_equal(y.ravel(), [0.0] * 13 + list(range(1, 12)))


def check_pool_hand_4x4(relu, maxpool):
    # four windows, the maximum in a different corner of each
    x = np.array([[9, 1, 2, 3],
                  [4, 5, 6, 8],
                  [0, 1, 7, 4],
                  [6, 2, 5, 3]], dtype=np.float64)[None, None]
    assert np.array_equal(maxpool(x)[0, 0], [[9, 8], [6, 7]])


def check_pool_each_corner(relu, maxpool):
    # a single 5.0 moved through the four positions of the first window of a
    # 2x4 image; the second window holds 1.0 everywhere
    for a in range(2):
        for b in range(2):
            x = np.zeros((1, 1, 2, 4))
            x[0, 0, :, 2:] = 1.0
            x[0, 0, a, b] = 5.0
            assert np.array_equal(maxpool(x)[0, 0], [[5.0, 1.0]]), (a, b)


def check_pool_all_negative(relu, maxpool):
    # the result is the least negative value of the window, not zero
    x = np.array([[-4, -3, -9, -8],
                  [-2, -7, -1.5, -6]], dtype=np.float64)[None, None]
    assert np.array_equal(maxpool(x)[0, 0], [[-2.0, -1.5]])


def check_pool_odd_sizes_floor(relu, maxpool):
    # 5x7 -> 2x3: the last row and column are dropped (floor), even when they
    # hold the largest values
    x = np.arange(35, dtype=np.float64).reshape(1, 1, 5, 7)
    x[0, 0, 4, :] = 1000.0
    x[0, 0, :, 6] = 1000.0
    y = maxpool(x)
    assert y.shape == (1, 1, 2, 3)
    assert np.array_equal(y[0, 0], [[8, 10, 12], [22, 24, 26]])


def check_pool_one_pixel_and_one_row(relu, maxpool):
    assert maxpool(np.ones((1, 1, 1, 1))).shape == (1, 1, 0, 0)
    y = maxpool(np.array([[[[3.0, -1.0, 2.0]], [[0.0, 0.0, 0.0]]]]).reshape(1, 2, 1, 3))
    assert y.shape == (1, 2, 0, 1)


def check_pool_channels_and_images_independent(relu, maxpool):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 4, 6, 8))
    y = maxpool(x)
    for n in range(3):
        for c in range(4):
            want = np.array([[x[n, c, 2 * i:2 * i + 2, 2 * j:2 * j + 2].max() for j in range(4)]
                             for i in range(3)])
            assert np.array_equal(y[n, c], want), (n, c)


ALL_CHECKS = [check_relu_signs, check_relu_keeps_shape_and_positives, check_pool_hand_4x4,
              check_pool_each_corner, check_pool_all_negative, check_pool_odd_sizes_floor,
              check_pool_one_pixel_and_one_row, check_pool_channels_and_images_independent]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_nn_pin(check):
    check(nn.relu, nn.maxpool2x2)


# (name, original text, mutated text) in a copy of oracle/nn.py
MUTANTS = [
    ("pool_stride_one", "x[:, :, a:2 * Ho:2, b:2 * Wo:2]", "x[:, :, a:a + Ho, b:b + Wo]"),
    ("pool_init_zero", "-np.inf, dtype", "0.0, dtype"),
    ("pool_one_window_row", "for a in range(2):", "for a in range(1):"),
    ("pool_one_window_col", "for b in range(2):", "for b in range(1):"),
    ("pool_min", "y = np.maximum(y, x", "y = np.minimum(y, x"),
    ("pool_ceil", "Ho, Wo = H // 2, W // 2", "Ho, Wo = (H + 1) // 2, (W + 1) // 2"),
    ("pool_window_offset", "x[:, :, a:2 * Ho:2, b:2 * Wo:2]", "x[:, :, a + 1:2 * Ho + 1:2, b:2 * Wo:2]"),
    ("relu_abs", "return np.maximum(x, 0.0)", "return np.abs(x)"),
    ("relu_leaky", "return np.maximum(x, 0.0)", "return np.maximum(x, 0.01 * x)"),
    ("relu_min", "return np.maximum(x, 0.0)", "return np.minimum(x, 0.0)"),
]


def _mutant_module(name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, (name, old)
    mod = types.ModuleType("nn_" + name)
    exec(compile(src.replace(old, new), "nn_" + name, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_nn_pins_catch_mutant(mutant):
    mod = _mutant_module(*mutant)
    caught = []
    for check in ALL_CHECKS:
        try:
            check(mod.relu, mod.maxpool2x2)
        except (AssertionError, ValueError, IndexError):
            caught.append(check.__name__)
    assert caught, f"no pin caught mutant {mutant[0]}"
