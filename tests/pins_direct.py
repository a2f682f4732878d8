"""Pins of the direct-convolution oracle against facts fixed by mathematics.

Each check takes ``conv(x, g, pad) -> y`` (fp64 [N, K, Ho, Wo]) and raises
AssertionError on a mismatch.  They are written so that a plausible mistake in
the oracle (a dropped term, a wrong sign, an index off by one, a flipped or
transposed filter, a wrong padding offset, a skipped channel) fails at least
one of them; ``test_oracle_mutants.py`` plants such mistakes and checks that.

Definition pinned (the paper's Eq. 1 reaches it exactly, Sec. 2): the
multi-channel 3x3 stride-1 cross-correlation with symmetric zero padding.
"""
import numpy as np
from numpy.lib.stride_tricks import sliding_window_view


def check_single_dot_product(conv):
    # C = K = 1, 3x3 input, pad 0: one output = sum of the 9 elementwise products.
    x = np.arange(1, 10, dtype=np.float64).reshape(1, 1, 3, 3)
    g = np.arange(1, 10, dtype=np.float64).reshape(1, 1, 3, 3)
    y = conv(x, g, 0)
    assert y.shape == (1, 1, 1, 1)
    assert y[0, 0, 0, 0] == 285.0            # 1^2 + 2^2 + ... + 9^2


def check_hand_example_pad1(conv):
    # x = [[1,2,3],[4,5,6],[7,8,9]], g has +1 at (0,0) and -1 at (2,2), pad 1:
    # y[i,j] = x~[i-1, j-1] - x~[i+1, j+1] (x~ zero outside).  Worked by hand.
    x = np.arange(1, 10, dtype=np.float64).reshape(1, 1, 3, 3)
    g = np.zeros((1, 1, 3, 3))
    g[0, 0, 0, 0] = 1.0
    g[0, 0, 2, 2] = -1.0
    want = np.array([[-5, -6, 0],
                     [-8, -8, 2],
                     [0, 4, 5]], dtype=np.float64)
    y = conv(x, g, 1)
    assert y.shape == (1, 1, 3, 3)
    assert np.array_equal(y[0, 0], want), y[0, 0]


def check_matvec_special_case(conv):
    # H = W = 1, pad 1: only the centre tap sees data, so y[n,k] = sum_c g[k,c,1,1] x[n,c].
    # C=2, K=3, g[k,c,1,1] = 10k + c, x[n,c] = c + 1:  y = [2, 32, 62] (by hand).
    x = np.array([1.0, 2.0]).reshape(1, 2, 1, 1)
    g = np.full((3, 2, 3, 3), 1000.0)        # off-centre taps must not contribute
    for k in range(3):
        for c in range(2):
            g[k, c, 1, 1] = 10 * k + c
    y = conv(x, g, 1)
    assert y.shape == (1, 3, 1, 1)
    assert np.array_equal(y[0, :, 0, 0], [2.0, 32.0, 62.0]), y[0, :, 0, 0]


def _sliding_window_reference(x, g, pad):
    xp = np.pad(x, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    win = sliding_window_view(xp, (3, 3), axis=(2, 3))      # n, c, i, j, r, s
    return np.einsum("ncijrs,kcrs->nkij", win, g)


def check_against_sliding_window(conv, seed=1):
    rng = np.random.default_rng(seed)
    for (N, C, H, W, K, pad) in [(2, 3, 7, 5, 4, 0), (1, 5, 6, 9, 2, 1), (3, 2, 4, 4, 3, 2),
                                 (1, 1, 3, 8, 1, 1), (2, 4, 1, 1, 5, 1)]:
        x = rng.standard_normal((N, C, H, W))
        g = rng.standard_normal((K, C, 3, 3))
        want = _sliding_window_reference(x, g, pad)
        y = conv(x, g, pad)
        assert y.shape == want.shape, (y.shape, want.shape)
        scale = np.abs(x).max() * np.abs(g).sum(axis=(1, 2, 3)).max()
        assert np.abs(y - want).max() <= 1e-12 * scale, np.abs(y - want).max()


def check_textbook_correlate2d(conv, seed=2):
    from scipy.signal import correlate2d
    rng = np.random.default_rng(seed)
    for (H, W, pad) in [(5, 5, 0), (6, 4, 1), (3, 7, 2)]:
        x = rng.standard_normal((H, W))
        g = rng.standard_normal((3, 3))
        want = correlate2d(np.pad(x, pad), g, mode="valid")
        y = conv(x.reshape(1, 1, H, W), g.reshape(1, 1, 3, 3), pad)[0, 0]
        assert np.allclose(y, want, rtol=0, atol=1e-12), np.abs(y - want).max()


def check_one_hot_orientation(conv):
    # Asymmetric one-hot filters: y[i,j] = x~[i + r - pad, j + s - pad] exactly.
    rng = np.random.default_rng(3)
    x = rng.integers(-9, 10, (1, 1, 5, 6)).astype(np.float64)
    for pad in (0, 1, 2):
        xp = np.pad(x[0, 0], pad)
        for r in range(3):
            for s in range(3):
                g = np.zeros((1, 1, 3, 3))
                g[0, 0, r, s] = 1.0
                y = conv(x, g, pad)[0, 0]
                Ho, Wo = y.shape
                assert np.array_equal(y, xp[r:r + Ho, s:s + Wo]), (pad, r, s)


def check_linearity(conv, seed=4):
    rng = np.random.default_rng(seed)
    x1, x2 = (rng.integers(-5, 6, (2, 3, 6, 5)).astype(np.float64) for _ in range(2))
    g1, g2 = (rng.integers(-5, 6, (4, 3, 3, 3)).astype(np.float64) for _ in range(2))
    a, b = 3.0, -2.0
    assert np.array_equal(conv(a * x1 + b * x2, g1, 1), a * conv(x1, g1, 1) + b * conv(x2, g1, 1))
    assert np.array_equal(conv(x1, a * g1 + b * g2, 1), a * conv(x1, g1, 1) + b * conv(x1, g2, 1))


def check_zero_pad_invariance(conv, seed=5):
    rng = np.random.default_rng(seed)
    x = rng.integers(-7, 8, (2, 3, 5, 7)).astype(np.float64)
    g = rng.integers(-7, 8, (2, 3, 3, 3)).astype(np.float64)
    for p in (1, 2):
        xp = np.pad(x, ((0, 0), (0, 0), (p, p), (p, p)))
        assert np.array_equal(conv(x, g, p), conv(xp, g, 0)), p


def check_channel_and_batch_independence(conv, seed=6):
    rng = np.random.default_rng(seed)
    x = rng.integers(-5, 6, (3, 4, 5, 5)).astype(np.float64)
    g = rng.integers(-5, 6, (2, 4, 3, 3)).astype(np.float64)
    y = conv(x, g, 1)
    # Batch: each image on its own.
    for n in range(3):
        assert np.array_equal(y[n:n + 1], conv(x[n:n + 1], g, 1)), n
    # Channels: the layer is the sum of its single-channel layers (Eq. 1's sum over c).
    acc = sum(conv(x[:, c:c + 1], g[:, c:c + 1], 1) for c in range(4))
    assert np.array_equal(y, acc)


ALL_CHECKS = [check_single_dot_product, check_hand_example_pad1, check_matvec_special_case,
              check_against_sliding_window, check_textbook_correlate2d, check_one_hot_orientation,
              check_linearity, check_zero_pad_invariance, check_channel_and_batch_independence]
