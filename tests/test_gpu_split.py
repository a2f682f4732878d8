"""The split path (input transform into blocks of 16 consecutive tiles, then
the T GEMMs with the output transform in their epilogue) against the fp64
direct oracle, on layers whose GEMM work items leave a short last round: those
items run as units of one tile block and one filter block, with the channel
parts of a unit summed in a fixed order.  The shapes also end the batch in a
partial tile block, have K not a multiple of 16 and C not a multiple of 4."""
import numpy as np
import pytest

import gpu_helpers as h
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl
from test_gpu_conv import _exact_bound

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}
ELEM = {2: 2e-5, 4: 2e-4}
CUS = 256


def split_items(N, C, H, W, K, pad, m):
    """(items, tail items, units per item) of the GEMM kernel, by the rule the
    library documents: items = tile-block pairs x filter groups (4 filter
    blocks per group for m = 4, 8 for m = 2); the items past the last whole
    round of 256 run as units when they number at most 256 / units."""
    _, _, _, _, P = h.geometry(N, H, W, pad, m)
    kgw = 4 if m == 4 else 8
    items = (-(-P // 16) + 1) // 2 * -(-(-(-K // 16)) // kgw)
    rem, units = items % CUS, 2 * kgw
    tail = rem if items > CUS and 0 < rem and rem * units <= CUS else 0
    return items, tail, units


# (N, C, H, W, K, pad, m)
SHAPES = [
    (11, 16, 56, 56, 256, 1, 4),    # 2156 tiles: 135 blocks (last one 12 tiles), 272 items, 16 of them as units
    (11, 13, 56, 56, 250, 1, 4),    # C, K ragged
    (11, 8, 56, 56, 128, 1, 2),     # 8624 tiles: 539 blocks, 270 items, 14 as units
    (5, 24, 58, 62, 144, 1, 2),     # ragged tiles at both edges: 29 x 31 per image
    (6, 36, 61, 61, 200, 1, 4),     # 15 x 15 tiles per image, several channel steps
]


def _check(shape, flags, seed):
    N, C, H, W, K, pad, m = shape
    rng = np.random.default_rng(seed)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = direct.conv2d(x, g, pad, absval=True)
    U = h.filter_transform(g, m)
    y = h.host(h.conv2d(x, U, K, pad, m, flags))
    assert np.all(np.isfinite(y))
    err = h.normwise_err(y, ref)
    print(f"  normwise err {err:.2e}", flush=True)
    assert err <= TOL[m], err
    # elementwise against 16 x the largest |x|*|g| of the layer (a tile's own
    # bound can be smaller; a misplaced or missing output fails this by far)
    assert np.all(np.abs(y - ref) <= ELEM[m] * 16 * bound.max()), "elementwise"
    return x, g, U, y


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_split_tail_units(shape):
    items, tail, units = split_items(*shape)
    print(f"split shape={shape} items={items} tail={tail} units={units}", flush=True)
    if shape[3] in (56,):
        assert tail > 0, "the shape exercises the tail units"
    _check(shape, B.WINO_ALGO_SPLIT, seed=sum(shape))


@pytest.mark.parametrize("shape", SHAPES[:3], ids=lambda s: "x".join(map(str, s)))
def test_split_relu_and_repeatable(shape):
    N, C, H, W, K, pad, m = shape
    print(f"split relu shape={shape}", flush=True)
    rng = np.random.default_rng(7 + sum(shape))
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = np.maximum(direct.conv2d(x, g, pad), 0.0)
    U = h.filter_transform(g, m)
    y1 = h.host(h.conv2d(x, U, K, pad, m, B.WINO_ALGO_SPLIT | B.WINO_FLAG_RELU))
    y2 = h.host(h.conv2d(x, U, K, pad, m, B.WINO_ALGO_SPLIT | B.WINO_FLAG_RELU))
    assert np.all(y1 >= 0)
    assert h.normwise_err(y1, ref) <= TOL[m]
    assert np.array_equal(y1, y2)          # bitwise run to run


def test_split_exact_on_integers():
    # Integer x and g a multiple of 576 (S*G integer for m = 4): every partial
    # sum is an integer below 2^24, so the tail units' summation order and the
    # main items' must both give the oracle's result bit for bit.
    N, C, H, W, K, pad, m = 11, 8, 56, 56, 256, 1, 4
    assert split_items(N, C, H, W, K, pad, m)[1] > 0
    rng = np.random.default_rng(3)
    x = rng.integers(-1, 2, (N, C, H, W)).astype(np.float32)
    g = (rng.integers(-1, 2, (K, C, 3, 3)) * 576).astype(np.float32)
    big, u_int = _exact_bound(x[:2].astype(np.float64), g.astype(np.float64), pad, m)
    assert u_int and big < 2 ** 23, "precondition of the exact regime (bound on two images, margin 2x)"
    ref = direct.conv2d(x, g, pad)
    U = h.filter_transform(g, m)
    y = h.host(h.conv2d(x, U, K, pad, m, B.WINO_ALGO_SPLIT))
    assert np.array_equal(y.astype(np.float64), ref)
