"""A seeded sweep over random small layers: every algorithm the library accepts
for the layer (AUTO, fused, staged, split, low-C), in NCHW and channel-last
layout, with and without ReLU, against the fp64 direct oracle; and the 16-bit
operand paths against the oracle's reduced-precision reference.  The shapes
lean on the edges: images of one or two pixels, odd channel and filter counts,
C <= 4 (the low-C kernel), padding up to 3, ragged tiles.  Layers with Ho or
Wo below 1 must be refused as invalid arguments by every entry point.  The
same over F(2x2,5x5) layers and the 1-D layers of both axes."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import direct
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl
from test_gpu_nhwc import tile_bound
from test_gpu_prec16 import PRECS, conv16, filter16, reference_and_bound

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}
ELEM = {2: 2e-5, 4: 2e-4}
BAD = 2**64 - 1
ALGOS = {"auto": B.WINO_ALGO_AUTO, "fused": B.WINO_ALGO_FUSED, "staged": B.WINO_ALGO_STAGED,
         "split": B.WINO_ALGO_SPLIT, "lowc": B.WINO_ALGO_LOWC}


def _cases(n=120, seed=2026):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        N = int(rng.integers(1, 4))
        C = int(rng.choice([1, 2, 3, 4, 5]) if rng.random() < 0.3 else rng.integers(1, 73))
        K = int(rng.integers(1, 73))
        H = int(rng.choice([1, 2, 3]) if rng.random() < 0.15 else rng.integers(1, 41))
        W = int(rng.choice([1, 2, 3]) if rng.random() < 0.15 else rng.integers(1, 41))
        pad = int(rng.choice([0, 1, 1, 1, 2, 3]))
        m = int(rng.choice([2, 4]))
        relu = bool(rng.random() < 0.5)
        out.append((N, C, H, W, K, pad, m, relu))
    return out


CASES = _cases()


def _valid(N, C, H, W, K, pad, m):
    return H + 2 * pad - 2 >= 1 and W + 2 * pad - 2 >= 1


def test_sweep_has_edges():
    # the generator reaches the edges it is meant to: invalid layers, tiny and
    # low-C layers, both m, padding 0 and 3
    assert any(not _valid(*c[:7]) for c in CASES)
    assert any(c[1] <= 4 and _valid(*c[:7]) for c in CASES)
    assert {2, 4} <= {c[6] for c in CASES}
    assert {0, 3} <= {c[5] for c in CASES}


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[:7])) + ("r" if c[7] else ""))
def test_sweep_fp32(case):
    N, C, H, W, K, pad, m, relu = case
    print(f"sweep fp32 {case}", flush=True)
    rng = np.random.default_rng(sum(case[:7]) * 7 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U = h.filter_transform(g, m)
    rf = B.WINO_FLAG_RELU if relu else 0
    if not _valid(N, C, H, W, K, pad, m):
        for fl in ALGOS.values():
            assert B.wino_workspace_bytes(N, C, H, W, K, pad, m, fl | rf) == BAD
            assert B.wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, fl | rf) == BAD
        y = torch.zeros(1, dtype=torch.float32, device=h.DEV)
        assert B.wino_conv2d(h.dev(x), U, y, N, C, H, W, K, pad, m, rf, None, 0) == B.WINO_ERR_INVALID_ARG
        return
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), m)
    if relu:
        ref = np.maximum(ref, 0.0)
    nonzero = np.abs(ref).max() > 0        # (ReLU can zero a tiny layer's whole output)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    ran = []
    for name, fl in ALGOS.items():
        if B.wino_workspace_bytes(N, C, H, W, K, pad, m, fl | rf) == BAD:
            assert name not in ("auto", "fused", "staged"), name   # these take every valid small layer
            continue
        y = h.host(h.conv2d(x, U, K, pad, m, fl | rf))
        assert np.all(np.isfinite(y)), name
        assert nonzero or np.all(y == 0), name
        assert not nonzero or h.normwise_err(y, ref) <= TOL[m], name
        assert np.all(np.abs(y - ref) <= ELEM[m] * (bound + 1e-30)), name
        if relu:
            assert np.all(y >= 0), name
        ran.append(name)
        wsn = B.wino_workspace_bytes_nhwc(N, C, H, W, K, pad, m, fl | rf)
        if wsn == BAD:
            continue
        yn = torch.full((N, Ho, Wo, K), float("nan"), dtype=torch.float32, device=h.DEV)
        ws = h.empty_bytes(wsn)
        B.check(B.wino_conv2d_nhwc(h.dev(x_nhwc), U, yn, N, C, H, W, K, pad, m, fl | rf, ws, wsn),
                "wino_conv2d_nhwc")
        yn = h.host(yn).transpose(0, 3, 1, 2)
        assert not nonzero or h.normwise_err(yn, ref) <= TOL[m], name + " nhwc"
        assert np.all(np.abs(yn - ref) <= ELEM[m] * (bound + 1e-30)), name + " nhwc"
        ran.append(name + "_nhwc")
    print(f"  ran {ran}", flush=True)
    assert {"auto", "fused", "staged"} <= set(ran)
    if C <= 4:
        assert "lowc" in ran


@pytest.mark.parametrize("prec", list(PRECS))
@pytest.mark.parametrize("case", [c for c in CASES if _valid(*c[:7])][::3],
                         ids=lambda c: "x".join(map(str, c[:7])) + ("r" if c[7] else ""))
def test_sweep_16bit(case, prec):
    N, C, H, W, K, pad, m, relu = case
    print(f"sweep {prec} {case}", flush=True)
    flag, u, rnd = PRECS[prec]
    rng = np.random.default_rng(sum(case[:7]) * 11 + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    U16, _ = filter16(g, m, flag)
    y16, bound = reference_and_bound(x, g, pad, m, rnd)
    if relu:
        y16 = np.maximum(y16, 0.0)           # 1-Lipschitz: the bound still holds
    tol = (2 * u + 4 * C * 2.0 ** -24 + 2.0 ** -20) * bound + 1e-30
    for algo in (B.WINO_ALGO_AUTO, B.WINO_ALGO_STAGED, B.WINO_ALGO_SPLIT):
        y = conv16(x, U16, K, pad, m, flag | algo, relu=relu)
        assert np.all(np.isfinite(y)), algo
        assert np.all(np.abs(y - y16) <= tol), algo


def _cases_rs(n, seed, rmin):
    """(N, C, H, W, K, pad, relu) for layers of an r x r or 1 x r filter."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        N = int(rng.integers(1, 4))
        C = int(rng.choice([1, 2, 3, 5]) if rng.random() < 0.25 else rng.integers(1, 73))
        K = int(rng.integers(1, 73))
        H = int(rng.integers(1, 41))
        W = int(rng.integers(1, 41))
        pad = int(rng.integers(0, rmin))
        out.append((N, C, H, W, K, pad, bool(rng.random() < 0.5)))
    return out


CASES_R5 = _cases_rs(40, 2027, 4)


@pytest.mark.parametrize("case", CASES_R5, ids=lambda c: "x".join(map(str, c[:6])) + ("r" if c[6] else ""))
def test_sweep_5x5(case):
    # F(2x2,5x5): every algorithm the library accepts for the layer (AUTO at least)
    import test_gpu_r5 as r5
    N, C, H, W, K, pad, relu = case
    print(f"sweep 5x5 {case}", flush=True)
    rng = np.random.default_rng(sum(case[:6]) * 13)
    x, g = r5.random_layer(rng, N, C, H, W, K)
    U = r5.filter_transform(g)
    rf = B.WINO_FLAG_RELU if relu else 0
    Ho, Wo = H + 2 * pad - 4, W + 2 * pad - 4
    if Ho < 1 or Wo < 1:
        assert B.wino_workspace_bytes_r(N, C, H, W, K, pad, 2, 5, rf) == BAD
        return
    ref = direct.conv2d(x, g, pad)
    bound = tile_bound(direct.conv2d(x, g, pad, absval=True), 2)
    if relu:
        ref = np.maximum(ref, 0.0)
    ran = []
    for name, fl in ALGOS.items():
        if B.wino_workspace_bytes_r(N, C, H, W, K, pad, 2, 5, fl | rf) == BAD:
            continue
        y = h.host(r5.conv(x, U, K, pad, fl | rf))
        assert np.all(np.isfinite(y)), name
        assert np.all(np.abs(y - ref) <= r5.ELEM * (bound + 1e-30)), name
        ran.append(name)
    print(f"  ran {ran}", flush=True)
    assert "auto" in ran


CASES_1D = [c + (v, ax) for c, v, ax in zip(_cases_rs(48, 2028, 4),
                                          [(6, 3), (4, 5), (2, 7)] * 16, ["w", "h"] * 24)]


@pytest.mark.parametrize("case", CASES_1D,
                         ids=lambda c: "x".join(map(str, c[:6])) + ("r" if c[6] else "") + f"-F{c[7][0]}r{c[7][1]}{c[8]}")
def test_sweep_1d(case):
    # F(1xm,1xr,1x8) along W or H: every algorithm the library accepts (AUTO at least)
    import test_gpu_1d as d1
    N, C, H, W, K, pad, relu, (m, r), axis = case
    print(f"sweep 1-D {case}", flush=True)
    rng = np.random.default_rng(sum(case[:6]) * 17 + m)
    x = rng.standard_normal((N, C, H, W)).astype(np.float32)
    g = (rng.standard_normal(d1.filt_shape(K, C, r, axis)) * np.sqrt(2.0 / (r * C))).astype(np.float32)
    U = d1.filter_transform(g, m, r)
    rf = B.WINO_FLAG_RELU if relu else 0
    ax = d1.AXES[axis]
    L = (W if axis == "w" else H) + 2 * pad - (r - 1)
    if L < 1:
        assert B.wino_workspace_bytes_1d(N, C, H, W, K, pad, m, r, ax, rf) == BAD
        return
    ref = d1.direct_1d(x, g, pad, axis)
    bound = d1.tile_bound(d1.direct_1d(x, g, pad, axis, absval=True), m, axis)
    if relu:
        ref = np.maximum(ref, 0.0)
    ran = []
    for name, fl in ALGOS.items():
        if B.wino_workspace_bytes_1d(N, C, H, W, K, pad, m, r, ax, fl | rf) == BAD:
            continue
        y = h.host(d1.conv(x, U, K, pad, m, r, axis, fl | rf))
        assert np.all(np.isfinite(y)), name
        assert np.all(np.abs(y - ref) <= d1.ELEM * (bound + 1e-30)), name
        ran.append(name)
    print(f"  ran {ran}", flush=True)
    assert "auto" in ran
