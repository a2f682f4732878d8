"""The 1-D variants F(1xm, 1xr, 1x8) of the oracle (1x3/1x5/1x7 and 3x1/5x1/7x1
layers), pinned against the bilinear identity and the direct definition (CPU)."""
from fractions import Fraction as Q

import numpy as np
import pytest

from oracle import cooktoom as ct
from oracle import direct

VARIANTS = list(ct.SUPPORTED_1D)


def direct_1d(x, g, pad, axis):
    """The direct definition with padding along the filtered axis only: pad x
    there and take the valid correlation (zero-pad invariance is pinned)."""
    pw = ((0, 0), (0, 0), (0, 0), (pad, pad)) if axis == "w" else ((0, 0), (0, 0), (pad, pad), (0, 0))
    return direct.conv2d(np.pad(np.asarray(x, dtype=np.float64), pw), np.asarray(g, dtype=np.float64), 0)


@pytest.mark.parametrize("m,r", VARIANTS)
def test_bilinear_identity(m, r):
    # F(m, r) with alpha = 8: y[i] = sum_k g[k] d[i+k] for every basis pair.
    AT, G, BT = ct.cook_toom_1d(m, r)
    assert len(AT) == m and len(G) == 8 and len(BT) == 8
    for kk in range(r):
        for aa in range(8):
            for i in range(m):
                s = sum((AT[i][j] * G[j][kk] * BT[j][aa] for j in range(8)), Q(0))
                assert s == (1 if aa == i + kk else 0), (m, r, i, kk, aa)


def test_shared_input_transform_and_dyadic_entries():
    bts = [ct.cook_toom_1d(m, r)[2] for m, r in VARIANTS]
    assert bts[0] == bts[1] == bts[2]                      # the same points: the same B^T
    for m, r in VARIANTS:
        AT, _, BT = ct.cook_toom_1d(m, r)
        for v in (v for row in AT + BT for v in row):      # powers of two only: exact in fp32
            d = v.denominator
            assert d & (d - 1) == 0, v


@pytest.mark.parametrize("m,r", VARIANTS)
@pytest.mark.parametrize("axis", ["w", "h"])
def test_listing1_over_rationals_equals_direct(m, r, axis):
    rng = np.random.default_rng(m * 10 + r + (axis == "h"))
    for pad in (0, (r - 1) // 2, r - 1):
        shape = (2, 2, 4, 11) if axis == "w" else (2, 2, 11, 4)
        x = rng.integers(-5, 6, shape)
        g = rng.integers(-4, 5, (3, 2, 1, r) if axis == "w" else (3, 2, r, 1))
        yq = ct.conv1d_exact(x, g, pad, m, axis)
        yd = direct_1d(x, g, pad, axis)
        assert yq.shape == yd.shape
        assert all(Q(int(v)) == v for v in yq.ravel())
        assert np.array_equal(yq.astype(np.float64), yd), pad


@pytest.mark.parametrize("m,r", VARIANTS)
@pytest.mark.parametrize("axis", ["w", "h"])
def test_fp64_stages_compose_to_direct(m, r, axis):
    rng = np.random.default_rng(100 + m + r)
    for (N, C, H, W, K, pad) in [(2, 5, 9, 17, 6, (r - 1) // 2), (1, 3, 1, 1, 2, r // 2 + 1), (3, 4, 8, 13, 7, 0)]:
        if axis == "h":
            H, W = W, H
        Ho, Wo, th, tw, P = ct.geometry_1d(N, H, W, pad, m, r, axis)
        if Ho < 1 or Wo < 1:
            continue
        x = rng.standard_normal((N, C, H, W))
        g = rng.standard_normal((K, C, 1, r) if axis == "w" else (K, C, r, 1))
        yw = ct.winograd_conv1d_f64(x, g, pad, m, axis)
        yd = direct_1d(x, g, pad, axis)
        bound = direct_1d(np.abs(x), np.abs(g), pad, axis)
        assert yw.shape == yd.shape == (N, K, Ho, Wo)
        assert np.all(np.abs(yw - yd) <= 1e-12 * (bound + 1e-300))
        V = ct.input_transform_1d(x, pad, m, r, axis)
        assert V.shape == (8, C, P)


def test_geometry_1d():
    # 1 x 7 'same' layer on 17 x 17 (Inception-v3): pad 3 along W only.
    assert ct.geometry_1d(2, 17, 17, 3, 2, 7, "w") == (17, 17, 17, 9, 2 * 17 * 9)
    assert ct.geometry_1d(2, 17, 17, 3, 2, 7, "h") == (17, 17, 9, 17, 2 * 9 * 17)
    assert ct.geometry_1d(1, 5, 10, 0, 6, 3, "w") == (5, 8, 5, 2, 10)
    with pytest.raises(ValueError):
        ct.cook_toom_1d(4, 3)
