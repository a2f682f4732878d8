"""Channel-last tensors (x [N][H][W][C], y [N][Ho][Wo][K]) through
wino_conv2d_nhwc: against the fp64 oracle, and bit for bit against the NCHW
path of the same algorithm on the same data (three stages: the two share V, M
and the GEMM; split: the same blocked V and GEMM kernel; only the layout of x
and y differs)."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}
ELEM = {2: 2e-5, 4: 2e-4}


def conv_nhwc(x_nhwc, U, K, pad, m, flags=0, y=None):
    xt = h.dev(x_nhwc) if isinstance(x_nhwc, np.ndarray) else x_nhwc
    N, H, W, C = xt.shape
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    if y is None:
        y = torch.full((N, Ho, Wo, K), float("nan"), dtype=torch.float32, device=h.DEV)
    wsb = B.wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, flags)
    assert wsb != 2**64 - 1
    ws = h.empty_bytes(wsb)
    B.check(B.wino_conv2d_nhwc(xt, U, y, N, C, H, W, K, pad, m, flags, ws, wsb), "wino_conv2d_nhwc")
    return y


def tile_bound(bound, m):
    N, K, Ho, Wo = bound.shape
    th, tw = -(-Ho // m), -(-Wo // m)
    b = np.zeros((N, K, th * m, tw * m))
    b[:, :, :Ho, :Wo] = bound
    t = b.reshape(N, K, th, m, tw, m).max(axis=(3, 5))
    return np.repeat(np.repeat(t, m, axis=2), m, axis=3)[:, :, :Ho, :Wo]


SHAPES = [(1, 3, 6, 6, 4, 0), (2, 5, 9, 11, 7, 1), (1, 16, 17, 23, 20, 1), (3, 8, 5, 5, 33, 2),
          (1, 1, 1, 1, 1, 1), (1, 24, 30, 30, 48, 1), (2, 64, 28, 28, 64, 1)]


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv2d_nhwc(m, shape):
    N, C, H, W, K, pad = shape
    print(f"conv2d_nhwc m={m} shape={shape}", flush=True)
    rng = np.random.default_rng(sum(shape) + 70 * m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), m)
    U = h.filter_transform(g, m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    y_nchw = h.host(h.conv2d(x, U, K, pad, m, B.WINO_ALGO_STAGED))
    for flags in (0, B.WINO_FLAG_RELU):
        y = h.host(conv_nhwc(x_nhwc, U, K, pad, m, flags)).transpose(0, 3, 1, 2)
        want = np.maximum(ref, 0.0) if flags else ref
        assert np.all(np.isfinite(y))
        assert h.normwise_err(y, want) <= TOL[m]
        assert np.all(np.abs(y - want) <= ELEM[m] * (bound + 1e-30))
        if not flags:
            assert np.array_equal(y, y_nchw)          # same arithmetic as the NCHW three stages


@pytest.mark.parametrize("m", [2, 4])
def test_conv2d_nhwc_unaligned_output_and_guards(m):
    # y one float off 16-byte alignment: the kernel falls back to 4-byte stores
    # and must give the same bits; nothing outside y is written.
    N, C, H, W, K, pad = 2, 12, 13, 10, 24, 1
    rng = np.random.default_rng(5 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    n_out = N * Ho * Wo * K
    buf = torch.full((1 + n_out + 1024,), float("nan"), dtype=torch.float32, device=h.DEV)
    conv_nhwc(x_nhwc, U, K, pad, m, y=buf[1:1 + n_out].view(N, Ho, Wo, K))
    a = h.host(buf)
    assert np.isnan(a[0]) and np.all(np.isnan(a[1 + n_out:]))
    y_al = h.host(conv_nhwc(x_nhwc, U, K, pad, m))
    assert np.array_equal(a[1:1 + n_out].reshape(N, Ho, Wo, K), y_al)


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("wide", [False, True])
def test_conv2d_nhwc_input_paths_agree(m, wide):
    # C % 4 == 0 with x 16-byte aligned takes the input transform by tile rows
    # through LDS, or, for an image too wide for one tile row of one channel
    # quad in its LDS budget, the 16-byte channel-quad loads per tile block; the
    # same x one float off that alignment takes the 4-byte loads: same bits,
    # on both the three stages and the split path.
    N, C, H, W, K, pad = (1, 4, 5, 444 if m == 4 else 556, 8, 1) if wide else (2, 20, 11, 14, 18, 1)
    print(f"nhwc input paths m={m} shape={(N, C, H, W, K, pad)}", flush=True)
    rng = np.random.default_rng(41 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    xb = torch.empty(1 + x_nhwc.size, dtype=torch.float32, device=h.DEV)
    xb[1:] = torch.from_numpy(x_nhwc.ravel()).to(h.DEV)
    ref = direct.conv2d(x, g, pad)
    for algo in (B.WINO_ALGO_STAGED, B.WINO_ALGO_SPLIT):
        y_al = h.host(conv_nhwc(x_nhwc, U, K, pad, m, algo))
        y_un = h.host(conv_nhwc(xb[1:].view(N, H, W, C), U, K, pad, m, algo))
        assert np.array_equal(y_al, y_un)
        assert h.normwise_err(y_al.transpose(0, 3, 1, 2), ref) <= TOL[m]


# (N, C, H, W, K, pad): ragged tiles, K and C not multiples of 4 or 16, several
# tile-block pairs and filter groups, a batch whose last block is partial
SPLIT_SHAPES = [(1, 16, 17, 23, 20, 1), (3, 8, 13, 11, 33, 2), (2, 5, 9, 11, 7, 1), (2, 40, 30, 30, 80, 1),
                (1, 1, 1, 1, 1, 1)]


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", SPLIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv2d_nhwc_split(m, shape):
    N, C, H, W, K, pad = shape
    print(f"conv2d_nhwc split m={m} shape={shape}", flush=True)
    rng = np.random.default_rng(sum(shape) + 90 * m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), m)
    U = h.filter_transform(g, m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    for flags in (0, B.WINO_FLAG_RELU):
        f = B.WINO_ALGO_SPLIT | flags
        y = h.host(conv_nhwc(x_nhwc, U, K, pad, m, f)).transpose(0, 3, 1, 2)
        want = np.maximum(ref, 0.0) if flags else ref
        assert np.all(np.isfinite(y))
        assert h.normwise_err(y, want) <= TOL[m]
        assert np.all(np.abs(y - want) <= ELEM[m] * (bound + 1e-30))
        y_nchw = h.host(h.conv2d(x, U, K, pad, m, f))
        assert np.array_equal(y, y_nchw)              # same V, GEMM and output transform


@pytest.mark.parametrize("m", [2, 4])
def test_conv2d_nhwc_split_paths_and_auto(m):
    # A layer with more than two rounds of split items: AUTO takes split (same
    # bits as explicit SPLIT); x and y one float off 16-byte alignment take the
    # 4-byte input loads and output stores: same bits again; and the NCHW
    # split path on the same data gives the same bits.
    N, C, H, W, K, pad = 16, 8, 64, 64, 256, 1
    rng = np.random.default_rng(77 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    assert B.wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, 0) == \
        B.wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, B.WINO_ALGO_SPLIT)
    y_split = h.host(conv_nhwc(x_nhwc, U, K, pad, m, B.WINO_ALGO_SPLIT))
    assert np.array_equal(h.host(conv_nhwc(x_nhwc, U, K, pad, m, 0)), y_split)
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    xb = torch.empty(1 + x_nhwc.size, dtype=torch.float32, device=h.DEV)
    xb[1:] = torch.from_numpy(x_nhwc.ravel()).to(h.DEV)
    n_out = N * Ho * Wo * K
    yb = torch.full((1 + n_out + 256,), float("nan"), dtype=torch.float32, device=h.DEV)
    conv_nhwc(xb[1:].view(N, H, W, C), U, K, pad, m, B.WINO_ALGO_SPLIT, y=yb[1:1 + n_out].view(N, Ho, Wo, K))
    a = h.host(yb)
    assert np.isnan(a[0]) and np.all(np.isnan(a[1 + n_out:]))
    assert np.array_equal(a[1:1 + n_out].reshape(N, Ho, Wo, K), y_split)
    y_nchw = h.host(h.conv2d(x, U, K, pad, m, B.WINO_ALGO_SPLIT))
    assert np.array_equal(y_split.transpose(0, 3, 1, 2), y_nchw)
    # sampled outputs against the fp64 oracle
    ref = direct.conv2d(x[:1], g[:16], pad)
    assert h.normwise_err(y_split[:1, :, :, :16].transpose(0, 3, 1, 2), ref) <= TOL[m]
