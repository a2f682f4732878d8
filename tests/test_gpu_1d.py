"""1-D layers -- 1 x r and r x 1 filters with F(1x6,1x3,1x8), F(1x4,1x5,1x8) and
F(1x2,1x7,1x8) -- through wino_filter_transform_1d / wino_conv2d_1d, against
the fp64 oracle: the filter transform, layers along both axes (ragged, padded,
several tile and filter blocks, ReLU), exact results, and a sampled full-size
Inception-style 1x7 / 7x1 layer."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import cooktoom as ct
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL, ELEM = 1e-3, 2e-4          # the F(4x4,3x3) gates (see the readings)
U32 = 2.0 ** -24
VARIANTS = [(6, 3), (4, 5), (2, 7)]
AXES = {"w": B.WINO_AXIS_W, "h": B.WINO_AXIS_H}


def direct_1d(x, g, pad, axis, absval=False):
    pw = ((0, 0), (0, 0), (0, 0), (pad, pad)) if axis == "w" else ((0, 0), (0, 0), (pad, pad), (0, 0))
    return direct.conv2d(np.pad(np.asarray(x, dtype=np.float64), pw), np.asarray(g, dtype=np.float64), 0,
                         absval=absval)


def filt_shape(K, C, r, axis):
    return (K, C, 1, r) if axis == "w" else (K, C, r, 1)


def filter_transform(g, m, r):
    K, C = g.shape[:2]
    U = h.empty_bytes(B.wino_filter_bytes_1d(C, K, m, r))
    B.check(B.wino_filter_transform_1d(h.dev(g), U, C, K, m, r), "wino_filter_transform_1d")
    return U


def conv(x, U, K, pad, m, r, axis, flags=0, y=None):
    xt = h.dev(x) if isinstance(x, np.ndarray) else x
    N, C, H, W = xt.shape
    Ho, Wo, *_ = ct.geometry_1d(N, H, W, pad, m, r, axis)
    if y is None:
        y = torch.full((N, K, Ho, Wo), float("nan"), dtype=torch.float32, device=h.DEV)
    ax = AXES[axis]
    wsb = B.wino_workspace_bytes_1d(N, C, H, W, K, pad, m, r, ax, flags)
    assert wsb != 2**64 - 1
    ws = h.empty_bytes(wsb)
    B.check(B.wino_conv2d_1d(xt, U, y, N, C, H, W, K, pad, m, r, ax, flags, ws, wsb), "wino_conv2d_1d")
    return y


def tile_bound(bound, m, axis):
    """Max of |x|*|g| over each tile (1 x m along W, m x 1 along H)."""
    b = np.asarray(bound)
    if axis == "h":
        b = np.swapaxes(b, 2, 3)
    N, K, A, L = b.shape
    nt = -(-L // m)
    e = np.zeros((N, K, A, nt * m))
    e[..., :L] = b
    t = np.repeat(e.reshape(N, K, A, nt, m).max(axis=4), m, axis=3)[..., :L]
    return np.swapaxes(t, 2, 3) if axis == "h" else t


@pytest.mark.parametrize("m,r", VARIANTS)
@pytest.mark.parametrize("C,K", [(3, 20), (37, 5), (64, 48)])
def test_filter_transform_1d(m, r, C, K):
    rng = np.random.default_rng(600 + 7 * m + C + K)
    g = (rng.standard_normal((K, C, 1, r)) * np.sqrt(2.0 / (r * C))).astype(np.float32)
    print(f"filter_transform_1d m={m} r={r} C={C} K={K}", flush=True)
    U = h.host(filter_transform(g, m, r))
    T = 8
    CQ, KB = -(-C // 4), -(-K // 16)
    a = U[:KB * CQ * T * 64].reshape(KB, CQ, T // 4, 4, 16, 4).transpose(2, 5, 1, 3, 0, 4)
    full = a.reshape(T, CQ * 4, KB * 16)
    ref = ct.filter_transform_1d(g.astype(np.float64), m)
    got = full[:, :C, :K].astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2 * U32 * np.abs(ref) + 1e-45)      # fp64 inside, one rounding
    mask = np.ones(full.shape, bool)
    mask[:, :C, :K] = False
    assert np.all(full[mask] == 0)


# (N, C, H, W, K): ragged and one-pixel images, C not a multiple of 4, K not a
# multiple of 16, several tile blocks; for axis 'h' H and W are swapped.
SHAPES = [(1, 3, 5, 9, 4), (2, 5, 7, 23, 7), (1, 16, 17, 17, 20), (3, 8, 1, 1, 33), (1, 24, 12, 70, 48)]


@pytest.mark.parametrize("m,r", VARIANTS)
@pytest.mark.parametrize("axis", ["w", "h"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv2d_1d(m, r, axis, shape):
    N, C, H, W, K = shape
    if axis == "h":
        H, W = W, H
    rng = np.random.default_rng(sum(shape) + 31 * m + (axis == "h"))
    for pad in ((r - 1) // 2, r - 1):
        Ho, Wo, *_ = ct.geometry_1d(N, H, W, pad, m, r, axis)
        if Ho < 1 or Wo < 1:
            continue
        print(f"conv2d_1d m={m} r={r} axis={axis} shape={shape} pad={pad}", flush=True)
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        g = (rng.standard_normal(filt_shape(K, C, r, axis)) * np.sqrt(2.0 / (r * C))).astype(np.float32)
        ref = direct_1d(x, g, pad, axis)
        bound = tile_bound(direct_1d(x, g, pad, axis, absval=True), m, axis)
        U = filter_transform(g, m, r)
        for flags in (0, B.WINO_FLAG_RELU):
            y = h.host(conv(x, U, K, pad, m, r, axis, flags))
            want = np.maximum(ref, 0.0) if flags else ref
            assert y.shape == want.shape
            assert np.all(np.isfinite(y))
            assert h.normwise_err(y, want) <= TOL
            assert np.all(np.abs(y - want) <= ELEM * (bound + 1e-30))


@pytest.mark.parametrize("m,r", VARIANTS)
@pytest.mark.parametrize("axis", ["w", "h"])
def test_conv2d_1d_exact(m, r, axis):
    # x in {-1, 0, 1}, g a multiple of 90 (90 G is an integer matrix): U is an
    # integer, V and M multiples of 1/4, every A^T partial sum a multiple of
    # 2^-7 far below 2^17 -- all exact in fp32, so the result is the oracle's.
    N, C, H, W, K, pad = 2, 6, 5, 19, 20, (r - 1) // 2
    if axis == "h":
        H, W = W, H
    rng = np.random.default_rng(40 + m + r)
    x = rng.integers(-1, 2, (N, C, H, W)).astype(np.float32)
    g = (rng.integers(-1, 2, filt_shape(K, C, r, axis)) * 90).astype(np.float32)
    Uo = ct.filter_transform_1d(g.astype(np.float64), m)
    Vo = ct.input_transform_1d(x.astype(np.float64), pad, m, r, axis)
    Mabs = ct.batched_gemm(np.abs(Uo), np.abs(Vo))
    assert np.all(Uo == np.round(Uo)) and np.all(Vo * 4 == np.round(Vo * 4))
    assert Mabs.max() * 128 < 2 ** 24
    y = h.host(conv(x, filter_transform(g, m, r), K, pad, m, r, axis))
    assert np.array_equal(y.astype(np.float64), direct_1d(x, g, pad, axis))


@pytest.mark.parametrize("axis", ["w", "h"])
def test_conv2d_1d_sampled_at_full_size(axis):
    # Inception-v3's 1x7 / 7x1 layers: 32 images of 192 x 17 x 17, 160 filters.
    w = wl.WORKLOADS["f2r7%s_n32_c192_k160_17x17" % axis]
    L = w.first
    x, gs = wl.generate(w)
    g = gs[0]
    N, C, H, W, K, pad = w.N, L.C, L.H, L.W, L.K, L.pad
    y = h.host(conv(x, filter_transform(g, 2, 7), K, pad, 2, 7, axis))
    rng = np.random.default_rng(3)
    idx = np.stack([rng.integers(0, s, 2048) for s in (N, K, H, W)], axis=1)
    idx[:4] = [[0, 0, 0, 0], [N - 1, K - 1, H - 1, W - 1], [0, K - 1, 0, W - 1], [N - 1, 0, H - 1, 0]]
    x64, g64 = x.astype(np.float64), g.astype(np.float64).reshape(K, C, 7)
    pw = ((0, 0), (0, 0), (0, 0), (pad, pad)) if axis == "w" else ((0, 0), (0, 0), (pad, pad), (0, 0))
    xp = np.pad(x64, pw)
    for n, k, i, j in idx:
        win = xp[n, :, i, j:j + 7] if axis == "w" else xp[n, :, i:i + 7, j]
        ref = np.sum(win * g64[k])
        # tile-local bound: the largest |x|*|g| over the output's 1 x 2 (2 x 1) tile
        t0 = (j if axis == "w" else i) // 2 * 2
        lim = W if axis == "w" else H
        sc = max(np.sum(np.abs(xp[n, :, i, q:q + 7] if axis == "w" else xp[n, :, q:q + 7, j]) * np.abs(g64[k]))
                 for q in range(t0, min(t0 + 2, lim)))
        assert abs(y[n, k, i, j] - ref) <= ELEM * (sc + 1e-30), (n, k, i, j)
