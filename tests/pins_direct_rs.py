"""Pins of the oracle's general R x S direct convolution (the 5x5 filters of the
paper's Table 2 layers) against facts fixed by mathematics.

Each check takes ``conv(x, g, pad) -> y`` (fp64 [N, K, Ho, Wo], g [K, C, R, S])
and raises AssertionError on a mismatch; ``test_oracle_mutants.py`` plants
plausible mistakes in a copy of the oracle and checks that one of them fails.
"""
import numpy as np
from numpy.lib.stride_tricks import sliding_window_view


def check_single_dot_product_5x5(conv):
    # C = K = 1, 5x5 input, pad 0: one output = sum of the 25 elementwise products.
    x = np.arange(1, 26, dtype=np.float64).reshape(1, 1, 5, 5)
    y = conv(x, x.copy(), 0)
    assert y.shape == (1, 1, 1, 1)
    assert y[0, 0, 0, 0] == 5525.0           # 1^2 + ... + 25^2 = 25*26*51/6


def check_hand_example_5x5_pad2(conv):
    # 3x3 input, 5x5 filter with +1 at (0,0) and -1 at (4,4), pad 2:
    # y[i,j] = x~[i-2, j-2] - x~[i+2, j+2]; with Ho = Wo = 3 only the corner
    # outputs see data (worked by hand).
    x = np.arange(1, 10, dtype=np.float64).reshape(1, 1, 3, 3)
    g = np.zeros((1, 1, 5, 5))
    g[0, 0, 0, 0] = 1.0
    g[0, 0, 4, 4] = -1.0
    want = np.array([[-9, 0, 0],
                     [0, 0, 0],
                     [0, 0, 1]], dtype=np.float64)
    y = conv(x, g, 2)
    assert y.shape == (1, 1, 3, 3)
    assert np.array_equal(y[0, 0], want), y[0, 0]


def _sliding_window_reference(x, g, pad):
    R, S = g.shape[2:]
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    win = sliding_window_view(xp, (R, S), axis=(2, 3))      # n, c, i, j, r, s
    return np.einsum("ncijrs,kcrs->nkij", win, g)


def check_against_sliding_window_rs(conv, seed=11):
    rng = np.random.default_rng(seed)
    for (N, C, H, W, K, R, S, pad) in [(2, 3, 9, 7, 4, 5, 5, 0), (1, 5, 8, 9, 2, 5, 5, 2),
                                       (3, 2, 6, 6, 3, 5, 5, 1), (1, 2, 7, 8, 2, 5, 3, 2),
                                       (2, 4, 1, 1, 5, 5, 5, 2), (1, 1, 4, 9, 1, 1, 7, 3)]:
        x = rng.standard_normal((N, C, H, W))
        g = rng.standard_normal((K, C, R, S))
        want = _sliding_window_reference(x, g, pad)
        y = conv(x, g, pad)
        assert y.shape == want.shape, (y.shape, want.shape)
        scale = np.abs(x).max() * np.abs(g).sum(axis=(1, 2, 3)).max()
        assert np.abs(y - want).max() <= 1e-12 * scale, np.abs(y - want).max()


def check_textbook_correlate2d_5x5(conv, seed=12):
    from scipy.signal import correlate2d
    rng = np.random.default_rng(seed)
    for (H, W, pad) in [(7, 7, 0), (6, 5, 2), (5, 9, 3)]:
        x = rng.standard_normal((H, W))
        g = rng.standard_normal((5, 5))
        want = correlate2d(np.pad(x, pad), g, mode="valid")
        y = conv(x.reshape(1, 1, H, W), g.reshape(1, 1, 5, 5), pad)[0, 0]
        assert np.allclose(y, want, rtol=0, atol=1e-12), np.abs(y - want).max()


def check_one_hot_orientation_5x5(conv):
    # One-hot filters at every tap: y[i,j] = x~[i + r - pad, j + s - pad] exactly.
    rng = np.random.default_rng(13)
    x = rng.integers(-9, 10, (1, 1, 6, 7)).astype(np.float64)
    for pad in (0, 2, 3):
        xp = np.pad(x[0, 0], pad)
        for r in range(5):
            for s in range(5):
                g = np.zeros((1, 1, 5, 5))
                g[0, 0, r, s] = 1.0
                y = conv(x, g, pad)[0, 0]
                Ho, Wo = y.shape
                assert np.array_equal(y, xp[r:r + Ho, s:s + Wo]), (pad, r, s)


def check_linearity_5x5(conv, seed=14):
    rng = np.random.default_rng(seed)
    x1, x2 = (rng.integers(-5, 6, (2, 3, 8, 7)).astype(np.float64) for _ in range(2))
    g1, g2 = (rng.integers(-5, 6, (4, 3, 5, 5)).astype(np.float64) for _ in range(2))
    a, b = 3.0, -2.0
    assert np.array_equal(conv(a * x1 + b * x2, g1, 2), a * conv(x1, g1, 2) + b * conv(x2, g1, 2))
    assert np.array_equal(conv(x1, a * g1 + b * g2, 2), a * conv(x1, g1, 2) + b * conv(x1, g2, 2))


def check_zero_pad_invariance_5x5(conv, seed=15):
    rng = np.random.default_rng(seed)
    x = rng.integers(-7, 8, (2, 3, 6, 8)).astype(np.float64)
    g = rng.integers(-7, 8, (2, 3, 5, 5)).astype(np.float64)
    for p in (1, 2, 3):
        xp = np.pad(x, ((0, 0), (0, 0), (p, p), (p, p)))
        assert np.array_equal(conv(x, g, p), conv(xp, g, 0)), p


def check_channel_and_batch_independence_5x5(conv, seed=16):
    rng = np.random.default_rng(seed)
    x = rng.integers(-5, 6, (3, 4, 7, 7)).astype(np.float64)
    g = rng.integers(-5, 6, (2, 4, 5, 5)).astype(np.float64)
    y = conv(x, g, 2)
    for n in range(3):
        assert np.array_equal(y[n:n + 1], conv(x[n:n + 1], g, 2)), n
    acc = sum(conv(x[:, c:c + 1], g[:, c:c + 1], 2) for c in range(4))
    assert np.array_equal(y, acc)


ALL_CHECKS = [check_single_dot_product_5x5, check_hand_example_5x5_pad2, check_against_sliding_window_rs,
              check_textbook_correlate2d_5x5, check_one_hot_orientation_5x5, check_linearity_5x5,
              check_zero_pad_invariance_5x5, check_channel_and_batch_independence_5x5]
