"""End-to-end wino_conv2d on the GPU against the fp64 direct oracle: every kernel
variant, small/ragged/degenerate shapes, exact integer results, invariants."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import cooktoom as ct
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}   # normwise max relative error gate per tile size
# elementwise error scaled by (|x| * |g|): far below fp32 Winograd's typical 1e-6 .. 3e-6
ELEM = {2: 2e-5, 4: 2e-4}

F = B.WINO_ALGO_FUSED
BLOCKS = (("16", B.WINO_BLOCK_1x16), ("4x4", B.WINO_BLOCK_4x4))
VARIANTS = {
    2: [("auto", 0), ("staged", B.WINO_ALGO_STAGED)]
       + [(f"split_b{bn}", B.WINO_ALGO_SPLIT | bf) for bn, bf in BLOCKS]
       + [(f"f_b{bn}c{c}", F | bf | B.WINO_CSPLIT(c))
          for bn, bf in (("16", B.WINO_BLOCK_1x16), ("4x4", B.WINO_BLOCK_4x4)) for c in (1, 2, 4, 8)],
    4: [("auto", 0), ("staged", B.WINO_ALGO_STAGED)]
       + [(f"split_b{bn}", B.WINO_ALGO_SPLIT | bf) for bn, bf in BLOCKS]
       + [(f"f_b{bn}c{c}", F | bf | B.WINO_CSPLIT(c))
          for bn, bf in (("16", B.WINO_BLOCK_1x16), ("4x4", B.WINO_BLOCK_4x4)) for c in (1, 2, 4)],
}

# (N, C, H, W, K, pad): the worked example's shape (3x6x6 input, 4 filters, valid
# convolution), ragged tiles, one-pixel images, K not a multiple of 16, C not a
# multiple of 4, several tile blocks and workgroups.
SHAPES = [
    (1, 3, 6, 6, 4, 0),
    (2, 5, 9, 11, 7, 1),
    (1, 16, 17, 23, 20, 1),
    (3, 8, 5, 5, 33, 2),
    (1, 1, 1, 1, 1, 1),
    (1, 4, 3, 3, 4, 0),
    (1, 24, 57, 57, 48, 1),
    (2, 64, 30, 30, 64, 1),
    # widths that are multiples of 4 (16-byte patch loads), every padding phase
    (1, 8, 16, 16, 20, 0),
    (2, 12, 12, 20, 17, 1),
    (1, 8, 9, 8, 16, 2),
    (1, 4, 7, 12, 8, 3),
    (1, 40, 24, 72, 32, 1),
]


def tile_bound(bound, m):
    """Max of |x|*|g| over each m x m output tile, broadcast to the tile's outputs.
    Winograd rounding error is tile-local: an output whose own window sees only
    padding is still a cancellation of its tile's nonzero terms."""
    N, K, Ho, Wo = bound.shape
    th, tw = -(-Ho // m), -(-Wo // m)
    b = np.zeros((N, K, th * m, tw * m))
    b[:, :, :Ho, :Wo] = bound
    t = b.reshape(N, K, th, m, tw, m).max(axis=(3, 5))
    return np.repeat(np.repeat(t, m, axis=2), m, axis=3)[:, :, :Ho, :Wo]


def _run_case(shape, m, flags, kind="normal", seed=0):
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(seed + sum(shape) + m)
    x, g = wl.random_layer(rng, N, C, H, W, K, kind)
    U = h.filter_transform(g, m)
    y = h.host(h.conv2d(x, U, K, pad, m, flags))
    return x, g, y


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv2d_all_variants(m, shape):
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(sum(shape) + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), m)
    U = h.filter_transform(g, m)
    for name, flags in VARIANTS[m]:
        print(f"conv2d m={m} shape={shape} variant={name}", flush=True)
        y = h.host(h.conv2d(x, U, K, pad, m, flags))
        assert np.all(np.isfinite(y)), name
        err = h.normwise_err(y, ref)
        assert err <= TOL[m], (name, err)
        # elementwise, scaled by the tile's |x|*|g|: catches a wrong value hidden by a large max
        assert np.all(np.abs(y - ref) <= ELEM[m] * (bound + 1e-30)), name


@pytest.mark.parametrize("m", [2, 4])
def test_relu_flag(m):
    shape = (2, 12, 14, 10, 20, 1)
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(42 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = np.maximum(direct.conv2d(x, g, pad), 0.0)
    U = h.filter_transform(g, m)
    for name, flags in VARIANTS[m]:
        y = h.host(h.conv2d(x, U, K, pad, m, flags | B.WINO_FLAG_RELU))
        assert np.all(y >= 0), name
        assert h.normwise_err(y, ref) <= TOL[m], name


def _exact_bound(x, g, pad, m):
    """Largest magnitude any fp32 intermediate can take, in any evaluation order."""
    AT, _, BT = ct.matrices_f64(m)
    U = ct.filter_transform(g, m)
    V = ct.input_transform(x, pad, m)
    Mabs = ct.batched_gemm(np.abs(U), np.abs(V))
    N, C, H, W = x.shape
    Ho, Wo, th, tw, P = ct.geometry(N, H, W, pad, m)
    a, K = m + 2, g.shape[0]
    s1 = np.einsum("iu,uvkp->ivkp", np.abs(AT), Mabs.reshape(a, a, K, P))
    s2 = np.einsum("ivkp,jv->ijkp", s1, np.abs(AT))
    d = ct.extract_regions(np.abs(x), pad, m)
    vb = np.einsum("au,nctjuv,bv->abcntj", np.abs(BT), d, np.abs(BT))
    return max(Mabs.max(), s1.max(), s2.max(), vb.max()), np.all(U == np.round(U))


@pytest.mark.parametrize("m,scale", [(2, 4), (4, 576)])
@pytest.mark.parametrize("shape", [(2, 8, 13, 11, 20, 1), (1, 20, 9, 9, 16, 0), (1, 24, 30, 30, 40, 1),
                                   (1, 20, 9, 12, 16, 1), (2, 8, 12, 16, 20, 2)])
def test_exact_on_integers(m, scale, shape):
    # Integer x and g with g a multiple of S^2 (S*G is an integer matrix), so U,
    # V, M and every partial sum are integers below 2^24: each variant must
    # reproduce the oracle bit for bit, whatever its summation order.
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(sum(shape) + m)
    x = rng.integers(-1, 2, (N, C, H, W)).astype(np.float32)
    g = (rng.integers(-1, 2, (K, C, 3, 3)) * scale).astype(np.float32)
    big, u_int = _exact_bound(x.astype(np.float64), g.astype(np.float64), pad, m)
    assert u_int and big < 2 ** 24, "precondition of the exact regime"
    ref = direct.conv2d(x, g, pad)
    U = h.filter_transform(g, m)
    for name, flags in VARIANTS[m]:
        print(f"exact m={m} shape={shape} variant={name}", flush=True)
        y = h.host(h.conv2d(x, U, K, pad, m, flags))
        assert np.array_equal(y.astype(np.float64), ref), name


@pytest.mark.parametrize("m", [2, 4])
def test_determinism_and_guard_bands(m):
    N, C, H, W, K, pad = 2, 20, 19, 21, 24, 1
    rng = np.random.default_rng(9)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    Ho, Wo, *_ = h.geometry(N, H, W, pad, m)
    n_out = N * K * Ho * Wo
    guard = 1024
    for name, flags in VARIANTS[m]:
        buf = torch.full((guard + n_out + guard,), float("nan"), dtype=torch.float32, device=h.DEV)
        y1 = buf[guard:guard + n_out].view(N, K, Ho, Wo)
        h.conv2d(x, U, K, pad, m, flags, y=y1)
        a = h.host(buf)
        assert np.all(np.isnan(a[:guard])) and np.all(np.isnan(a[guard + n_out:])), name
        assert np.all(np.isfinite(a[guard:guard + n_out])), name
        y2 = h.host(h.conv2d(x, U, K, pad, m, flags))
        assert np.array_equal(a[guard:guard + n_out].reshape(N, K, Ho, Wo), y2), name   # bitwise repeatable


@pytest.mark.parametrize("m", [2, 4])
def test_batch_independence_and_pad_invariance(m):
    N, C, H, W, K = 3, 12, 15, 17, 20
    rng = np.random.default_rng(10 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    for name, flags in VARIANTS[m]:
        if name == "auto":
            continue            # the planner may pick different variants for N=1 and N=3
        yb = h.host(h.conv2d(x, U, K, 1, m, flags))
        for n in range(N):
            yn = h.host(h.conv2d(x[n:n + 1], U, K, 1, m, flags))
            assert np.array_equal(yb[n:n + 1], yn), (name, n)
        xp = np.pad(x, ((0, 0), (0, 0), (1, 1), (1, 1)))
        y0 = h.host(h.conv2d(xp, U, K, 0, m, flags))
        assert np.array_equal(yb, y0), name


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", [(1, 12, 16, 16, 20, 1), (2, 8, 10, 24, 16, 2), (1, 20, 9, 12, 24, 0),
                                   (2, 100, 18, 64, 24, 1)],
                         ids=lambda s: "x".join(map(str, s)))
def test_patch_load_paths_agree(m, shape):
    # With W % 4 == 0 and a 16-byte aligned input the fused kernel loads its
    # patches in 16-byte chunks; an input one float off that alignment takes the
    # one-float path.  Both feed the same arithmetic: bit-identical outputs.
    # The 100-channel case runs several channel steps through the per-wave
    # patch regions of the one-row-group F(2x2,3x3) variants (1x16 blocks).
    N, C, H, W, K, pad = shape
    rng = np.random.default_rng(sum(shape) + 17 * m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    U = h.filter_transform(g, m)
    buf = torch.zeros(x.size + 1, dtype=torch.float32, device=h.DEV)
    xs = buf[1:].view(N, C, H, W)                 # 4-byte aligned, not 16-byte aligned
    xs.copy_(h.dev(x))
    for name, flags in VARIANTS[m]:
        ya = h.host(h.conv2d(x, U, K, pad, m, flags))
        yu = h.host(h.conv2d(xs, U, K, pad, m, flags))
        assert np.array_equal(ya, yu), name
        assert h.normwise_err(ya, ref) <= TOL[m], name
