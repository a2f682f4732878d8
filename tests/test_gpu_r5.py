"""F(2x2,5x5) -- the method on 5x5 filters (the 5x5 layers of the paper's
Table 2) -- through wino_filter_transform_r / wino_conv2d_r, against the fp64
oracle: the filter transform, whole layers on the fused and three-stage
algorithms (ragged, padded, several tile and filter blocks, every fused
variant, ReLU), exact integer results, and a sampled full-size layer."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import cooktoom as ct
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

M_, R_ = 2, 5
# Same region size and points as F(4x4,3x3): its gates.
TOL, ELEM = 1e-3, 2e-4
U32 = 2.0 ** -24


def filter_transform(g):
    K, C = g.shape[:2]
    U = h.empty_bytes(B.wino_filter_bytes_r(C, K, M_, R_))
    B.check(B.wino_filter_transform_r(h.dev(g), U, C, K, M_, R_), "wino_filter_transform_r")
    return U


def conv(x, U, K, pad, flags=0, y=None):
    xt = h.dev(x) if isinstance(x, np.ndarray) else x
    N, C, H, W = xt.shape
    Ho, Wo = H + 2 * pad - 4, W + 2 * pad - 4
    if y is None:
        y = torch.full((N, K, Ho, Wo), float("nan"), dtype=torch.float32, device=h.DEV)
    wsb = B.wino_workspace_bytes_r(N, C, H, W, K, pad, M_, R_, flags)
    assert wsb != 2**64 - 1
    ws = h.empty_bytes(wsb)
    B.check(B.wino_conv2d_r(xt, U, y, N, C, H, W, K, pad, M_, R_, flags, ws, wsb), "wino_conv2d_r")
    return y


def random_layer(rng, N, C, H, W, K):
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    g = (rng.standard_normal((K, C, 5, 5)) * np.sqrt(2.0 / (25.0 * C))).astype(np.float32)
    return x, g


def tile_bound(bound):
    N, K, Ho, Wo = bound.shape
    th, tw = -(-Ho // 2), -(-Wo // 2)
    b = np.zeros((N, K, th * 2, tw * 2))
    b[:, :, :Ho, :Wo] = bound
    t = b.reshape(N, K, th, 2, tw, 2).max(axis=(3, 5))
    return np.repeat(np.repeat(t, 2, axis=2), 2, axis=3)[:, :, :Ho, :Wo]


@pytest.mark.parametrize("C,K", [(3, 20), (16, 16), (37, 5), (130, 250), (128, 64)])
def test_filter_transform_5x5(C, K):
    rng = np.random.default_rng(500 + C + K)
    _, g = random_layer(rng, 1, C, 4, 4, K)
    print(f"filter_transform_r C={C} K={K}", flush=True)
    U = h.host(filter_transform(g))
    full = h.unpack_U(U, C, K, M_, crop=False, r=R_)
    got = full[:, :C, :K].astype(np.float64)
    ref = ct.filter_transform(g.astype(np.float64), M_)
    assert got.shape == ref.shape == (36, C, K)
    assert np.all(np.abs(got - ref) <= 2 * U32 * np.abs(ref) + 1e-45)     # fp64 inside, one rounding
    pad_mask = np.ones(full.shape, bool)
    pad_mask[:, :C, :K] = False
    assert np.all(full[pad_mask] == 0)


# (N, C, H, W, K, pad): the 'same' 5x5 layer (pad 2), valid, ragged (odd sizes),
# one-pixel images, C not a multiple of 4, K not a multiple of 16, several tile
# blocks, and rows wider than 64 tiles.
SHAPES = [
    (1, 3, 6, 6, 4, 0),
    (2, 5, 9, 11, 7, 2),
    (1, 16, 17, 23, 20, 2),
    (3, 8, 5, 5, 33, 1),
    (1, 1, 1, 1, 1, 2),
    (1, 24, 35, 35, 48, 2),
    (2, 32, 14, 14, 64, 2),
    (1, 4, 6, 140, 8, 2),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv2d_5x5(shape):
    N, C, H, W, K, pad = shape
    print(f"conv2d_r shape={shape}", flush=True)
    rng = np.random.default_rng(sum(shape) + 55)
    x, g = random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True))
    U = filter_transform(g)
    for flags in (0, B.WINO_ALGO_STAGED | B.WINO_FLAG_RELU):
        y = h.host(conv(x, U, K, pad, flags))
        r = np.maximum(ref, 0.0) if flags & B.WINO_FLAG_RELU else ref
        assert np.all(np.isfinite(y))
        assert h.normwise_err(y, r) <= TOL
        assert np.all(np.abs(y - r) <= ELEM * (bound + 1e-30))


# The fused kernel's variants: tile block (1 x 16 or 4 x 4) x channel split.
FUSED = [(f"b{bn}c{c}", B.WINO_ALGO_FUSED | bf | B.WINO_CSPLIT(c))
         for bn, bf in (("16", B.WINO_BLOCK_1x16), ("4", B.WINO_BLOCK_4x4)) for c in (1, 2, 4)]


@pytest.mark.parametrize("variant", FUSED, ids=lambda v: v[0])
@pytest.mark.parametrize("shape", [(2, 5, 9, 11, 7, 2), (1, 16, 17, 23, 20, 2), (1, 1, 1, 1, 1, 2),
                                   (2, 37, 14, 37, 40, 2), (1, 4, 6, 140, 8, 2), (3, 8, 5, 5, 33, 1),
                                   (2, 40, 20, 28, 36, 2), (1, 64, 13, 16, 80, 0)],
                         ids=lambda s: "x".join(map(str, s)))
def test_conv2d_5x5_fused_variants(shape, variant):
    # Every variant against the oracle: several channel steps, ragged tile
    # blocks and filter groups, odd widths (one float per patch load) and
    # W % 4 == 0 (16-byte patch loads).
    name, flags = variant
    N, C, H, W, K, pad = shape
    print(f"conv2d_r fused {name} shape={shape}", flush=True)
    rng = np.random.default_rng(sum(shape) + 5)
    x, g = random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True))
    U = filter_transform(g)
    assert B.wino_workspace_bytes_r(N, C, H, W, K, pad, M_, R_, flags) == 0
    y = h.host(conv(x, U, K, pad, flags))
    assert np.all(np.isfinite(y))
    assert h.normwise_err(y, ref) <= TOL
    assert np.all(np.abs(y - ref) <= ELEM * (bound + 1e-30))
    yr = h.host(conv(x, U, K, pad, flags | B.WINO_FLAG_RELU))
    assert np.array_equal(yr, np.maximum(y, 0.0))


def test_conv2d_5x5_fused_matches_staged():
    # Same U and V arithmetic (fp32 transforms, fp32 accumulation in a different
    # order): the two algorithms agree to rounding.
    N, C, H, W, K, pad = 2, 48, 35, 35, 64, 2
    rng = np.random.default_rng(35)
    x, g = random_layer(rng, N, C, H, W, K)
    U = filter_transform(g)
    yf = h.host(conv(x, U, K, pad, B.WINO_ALGO_FUSED))
    ys = h.host(conv(x, U, K, pad, B.WINO_ALGO_STAGED))
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True))
    assert np.all(np.abs(yf - ys) <= 2 * ELEM * (bound + 1e-30))


@pytest.mark.parametrize("shape", [(2, 4, 9, 11, 20, 2), (1, 8, 12, 12, 16, 0), (1, 3, 7, 16, 40, 1)])
def test_conv2d_5x5_exact_on_integers(shape):
    # Integer x in {-1, 0, 1} and g a multiple of 24^2 (S*G is an integer matrix
    # with S = 24): U, V, M and every partial sum are integers below 2^24, so the
    # result is the oracle's bit for bit.
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(sum(shape))
    x = rng.integers(-1, 2, (N, C, H, W)).astype(np.float32)
    g = (rng.integers(-1, 2, (K, C, 5, 5)) * 576).astype(np.float32)
    AT, _, BT = ct.matrices_f64(M_, R_)
    Uo = ct.filter_transform(g.astype(np.float64), M_)
    Vo = ct.input_transform(x.astype(np.float64), pad, M_, R_)
    Mabs = ct.batched_gemm(np.abs(Uo), np.abs(Vo))
    assert np.all(Uo == np.round(Uo)) and Mabs.max() < 2 ** 24 and np.abs(Vo).max() < 2 ** 24
    assert (np.abs(AT).sum(axis=1).max() ** 2) * Mabs.max() < 2 ** 24
    ref = direct.conv2d(x, g, pad)
    U = filter_transform(g)
    for flags in (B.WINO_ALGO_FUSED, B.WINO_ALGO_STAGED):
        y = h.host(conv(x, U, K, pad, flags))
        assert np.array_equal(y.astype(np.float64), ref)


def test_conv2d_5x5_repeatable_and_guarded():
    N, C, H, W, K, pad = 2, 12, 19, 21, 24, 2
    rng = np.random.default_rng(77)
    x, g = random_layer(rng, N, C, H, W, K)
    U = filter_transform(g)
    Ho, Wo = H + 2 * pad - 4, W + 2 * pad - 4
    n_out = N * K * Ho * Wo
    guard = 1024
    buf = torch.full((guard + n_out + guard,), float("nan"), dtype=torch.float32, device=h.DEV)
    conv(x, U, K, pad, y=buf[guard:guard + n_out].view(N, K, Ho, Wo))
    a = h.host(buf)
    assert np.all(np.isnan(a[:guard])) and np.all(np.isnan(a[guard + n_out:]))
    y2 = h.host(conv(x, U, K, pad))
    assert np.array_equal(a[guard:guard + n_out].reshape(N, K, Ho, Wo), y2)


def test_conv2d_5x5_sampled_at_full_size():
    # An Inception-style 5x5 layer at its full size (32 images of 48 x 35 x 35,
    # 64 filters, pad 2): outputs sampled across the batch, each against the
    # direct sum.
    w = wl.WORKLOADS["f2r5_n32_c48_k64_35x35"]
    L = w.first
    x, gs = wl.generate(w)
    g = gs[0]
    N, C, H, W, K, pad = w.N, L.C, L.H, L.W, L.K, L.pad
    y = h.host(conv(x, filter_transform(g), K, pad))
    rng = np.random.default_rng(9)
    idx = np.stack([rng.integers(0, s, 2048) for s in (N, K, H, W)], axis=1)
    idx[:4] = [[0, 0, 0, 0], [N - 1, K - 1, H - 1, W - 1], [0, K - 1, 0, W - 1], [N - 1, 0, H - 1, 0]]
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    g64 = g.astype(np.float64)
    for n, k, i, j in idx:
        ref = np.sum(xp[n, :, i:i + 5, j:j + 5] * g64[k])
        ti, tj = i // 2 * 2, j // 2 * 2
        scale = max(np.sum(np.abs(xp[n, :, a:a + 5, b:b + 5]) * np.abs(g64[k]))
                    for a in range(ti, min(ti + 2, H)) for b in range(tj, min(tj + 2, W)))
        assert abs(y[n, k, i, j] - ref) <= ELEM * (scale + 1e-30), (n, k, i, j)
