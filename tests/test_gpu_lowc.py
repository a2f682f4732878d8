"""The low-channel kernel (WINO_ALGO_LOWC, C <= 4) against the fp64 direct
oracle: every channel count and tile size, ragged tiles, filter ranges split
over workgroups, ReLU, exact integer results and guard bands."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl
from test_gpu_conv import _exact_bound

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}
ELEM = {2: 2e-5, 4: 2e-4}
L = B.WINO_ALGO_LOWC

# (N, C, H, W, K, pad): one channel up to four; widths that are and are not a
# multiple of the tile size (vector and scalar stores); a few tiles with many
# filters (the filter range split over workgroups); several tile groups with a
# ragged last one; K not a multiple of 16.
SHAPES = [
    (1, 1, 1, 1, 1, 1),
    (1, 3, 6, 6, 4, 0),
    (2, 2, 9, 11, 7, 1),
    (1, 4, 17, 23, 20, 1),
    (1, 3, 8, 8, 130, 1),
    (3, 1, 37, 29, 33, 2),
    (2, 3, 56, 56, 64, 1),
    (1, 4, 30, 18, 17, 3),
    (4, 3, 32, 32, 16, 1),
]


def tile_bound(bound, m):
    N, K, Ho, Wo = bound.shape
    th, tw = -(-Ho // m), -(-Wo // m)
    b = np.zeros((N, K, th * m, tw * m))
    b[:, :, :Ho, :Wo] = bound
    t = b.reshape(N, K, th, m, tw, m).max(axis=(3, 5))
    return np.repeat(np.repeat(t, m, axis=2), m, axis=3)[:, :, :Ho, :Wo]


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_lowc_matches_oracle(m, shape):
    N, C, H, W, K, pad = shape
    print(f"lowc m={m} shape={shape}", flush=True)
    rng = np.random.default_rng(sum(shape) + 31 * m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), m)
    U = h.filter_transform(g, m)
    for flags in (L, L | B.WINO_FLAG_RELU):
        y = h.host(h.conv2d(x, U, K, pad, m, flags))
        r = np.maximum(ref, 0.0) if flags & B.WINO_FLAG_RELU else ref
        assert np.all(np.isfinite(y))
        assert h.normwise_err(y, r) <= TOL[m]
        assert np.all(np.abs(y - r) <= ELEM[m] * (bound + 1e-30))
    # the planner takes this kernel for C <= 4: same bits as the explicit flag
    ya = h.host(h.conv2d(x, U, K, pad, m, 0))
    yl = h.host(h.conv2d(x, U, K, pad, m, L))
    assert np.array_equal(ya, yl)


@pytest.mark.parametrize("m,scale", [(2, 4), (4, 576)])
@pytest.mark.parametrize("shape", [(2, 3, 13, 11, 20, 1), (1, 4, 12, 16, 40, 0), (1, 1, 9, 9, 16, 2)])
def test_lowc_exact_on_integers(m, scale, shape):
    # Integer inputs and filters scaled so that U, V, M and every partial sum are
    # integers below 2^24 (C <= 4 keeps them small): the result is the oracle's
    # bit for bit.
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(sum(shape) + m)
    x = rng.integers(-1, 2, (N, C, H, W)).astype(np.float32)
    g = (rng.integers(-1, 2, (K, C, 3, 3)) * scale).astype(np.float32)
    big, u_int = _exact_bound(x.astype(np.float64), g.astype(np.float64), pad, m)
    assert u_int and big < 2 ** 24, "precondition of the exact regime"
    ref = direct.conv2d(x, g, pad)
    U = h.filter_transform(g, m)
    y = h.host(h.conv2d(x, U, K, pad, m, L))
    assert np.array_equal(y.astype(np.float64), ref)


@pytest.mark.parametrize("m", [2, 4])
def test_lowc_guard_bands_and_repeatability(m):
    N, C, H, W, K, pad = 2, 3, 19, 21, 24, 1
    rng = np.random.default_rng(90 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    Ho, Wo, *_ = h.geometry(N, H, W, pad, m)
    n_out = N * K * Ho * Wo
    guard = 1024
    buf = torch.full((guard + n_out + guard,), float("nan"), dtype=torch.float32, device=h.DEV)
    h.conv2d(x, U, K, pad, m, L, y=buf[guard:guard + n_out].view(N, K, Ho, Wo))
    a = h.host(buf)
    assert np.all(np.isnan(a[:guard])) and np.all(np.isnan(a[guard + n_out:]))
    assert np.all(np.isfinite(a[guard:guard + n_out]))
    y2 = h.host(h.conv2d(x, U, K, pad, m, L))
    assert np.array_equal(a[guard:guard + n_out].reshape(N, K, Ho, Wo), y2)
    # batch independence: image n alone gives the same bits as inside the batch
    for n in range(N):
        yn = h.host(h.conv2d(x[n:n + 1], U, K, pad, m, L))
        assert np.array_equal(y2[n:n + 1], yn)


@pytest.mark.parametrize("m", [2, 4])
def test_lowc_sampled_at_full_size(m):
    # A network's first layer at its full size (64 images of 3 x 224 x 224, 64
    # filters): outputs sampled across the batch and compared one by one with
    # the direct sum.
    N, C, H, W, K, pad = 64, 3, 224, 224, 64, 1
    rng = np.random.default_rng(5 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    y = h.host(h.conv2d(x, U, K, pad, m, 0))
    idx = np.stack([rng.integers(0, s, 4096) for s in (N, K, H, W)], axis=1)
    idx[:8] = [[0, 0, 0, 0], [N - 1, K - 1, H - 1, W - 1], [0, K - 1, 0, W - 1], [N - 1, 0, H - 1, 0],
               [1, 2, 223, 3], [2, 3, 4, 223], [63, 63, 111, 112], [32, 1, 0, 1]]
    xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    g64 = g.astype(np.float64)
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    for n, k, i, j in idx:
        ref = np.sum(xp[n, :, i:i + 3, j:j + 3] * g64[k])
        # Winograd rounding is tile-local: scale by the largest |x|*|g| in the tile
        ti, tj = i // m * m, j // m * m
        scale = max(np.sum(np.abs(xp[n, :, a:a + 3, b:b + 3]) * np.abs(g64[k]))
                    for a in range(ti, min(ti + m, Ho)) for b in range(tj, min(tj + m, Wo)))
        assert abs(y[n, k, i, j] - ref) <= ELEM[m] * (scale + 1e-30), (n, k, i, j)
