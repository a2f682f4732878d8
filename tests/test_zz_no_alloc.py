"""The allocation-free entry point (wino_conv2d_noalloc) against wino_conv2d.

Calls in a row on one GPU, each smaller than the one before, so every call
finds the previous call's contents in the shared static scratch: each output
must equal wino_conv2d's with the same flags (bit for bit: the same kernels
run, and the library is deterministic) and the fp64 oracle within the gate of
its m (16-bit operands: the reduced-precision reference's bound)."""
import numpy as np
import pytest

import gpu_helpers as h
from oracle import direct
from test_gpu_prec16 import PRECS, reference_and_bound
from paper_1903_01521_amd import binding as B

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}

# (N, C, H, W, K, pad, m, flags): split (31.5 MiB of scratch), split (18 MiB),
# AUTO on two channel slices (3 MiB of partial outputs), staged (0.9 MiB),
# staged with fp16 operands (1.4 MiB), split with bf16 operands (3.5 MiB),
# and AUTO on a layer whose split workspace (504 MiB) is past the scratch, so
# the fused kernel runs.
CASES = [
    (4, 256, 56, 56, 256, 1, 4, B.WINO_ALGO_SPLIT),
    (8, 256, 28, 28, 256, 1, 4, B.WINO_ALGO_SPLIT),
    (1, 512, 28, 28, 512, 1, 4, B.WINO_ALGO_AUTO | B.WINO_FLAG_RELU),
    (1, 64, 20, 20, 64, 1, 2, B.WINO_ALGO_STAGED),
    (2, 64, 30, 30, 48, 1, 4, B.WINO_ALGO_STAGED | B.WINO_PREC_F16),
    (4, 64, 56, 56, 64, 1, 4, B.WINO_ALGO_SPLIT | B.WINO_PREC_BF16 | B.WINO_FLAG_RELU),
]
BIG_AUTO = (64, 256, 56, 56, 256, 1, 4, B.WINO_ALGO_AUTO)


def _inputs(N, C, H, W, K, seed):
    rng = np.random.default_rng(seed)
    x = rng.uniform(-1.0, 1.0, (N, C, H, W)).astype(np.float32)
    g = (rng.standard_normal((K, C, 3, 3)) * np.sqrt(2.0 / (9 * C))).astype(np.float32)
    return x, g


def _filters(g, C, K, m, flags):
    prec = flags & B.WINO_PREC_MASK
    U = h.empty_bytes(B.wino_filter_bytes_p(C, K, m, prec))
    B.check(B.wino_filter_transform_p(h.dev(g), U, C, K, m, prec), "wino_filter_transform_p")
    return U


def _both(case, x, g):
    N, C, H, W, K, pad, m, flags = case
    Ho, Wo, *_ = h.geometry(N, H, W, pad, m)
    hx = h.dev(x)
    U = _filters(g, C, K, m, flags)
    y0 = h.empty_bytes(4 * N * K * Ho * Wo).reshape(N, K, Ho, Wo)
    B.check(B.wino_conv2d_noalloc(hx, U, y0, N, C, H, W, K, pad, m, flags), "wino_conv2d_noalloc")
    wsb = B.wino_workspace_bytes(N, C, H, W, K, pad, m, flags)
    ws = h.empty_bytes(wsb) if wsb else None
    y1 = h.empty_bytes(4 * N * K * Ho * Wo).reshape(N, K, Ho, Wo)
    B.check(B.wino_conv2d(hx, U, y1, N, C, H, W, K, pad, m, flags, ws, wsb), "wino_conv2d")
    return h.host(y0), h.host(y1)


def _check_oracle(case, x, g, y, sample):
    N, C, H, W, K, pad, m, flags = case
    xs = x[sample].astype(np.float64)
    if flags & B.WINO_PREC_MASK:
        # the 16-bit path's gate: one 16-bit ulp on either operand of a term
        # plus fp32 accumulation, against the reduced-precision reference
        prec = "fp16" if flags & B.WINO_PREC_MASK == B.WINO_PREC_F16 else "bf16"
        _, u, rnd = PRECS[prec]
        ref, bound = reference_and_bound(xs, g, pad, m, rnd)
        if flags & B.WINO_FLAG_RELU:           # 1-Lipschitz: the bound still holds
            ref = np.maximum(ref, 0.0)
        assert np.all(np.abs(y[sample] - ref) <= (2 * u + 4 * C * 2.0 ** -24 + 2.0 ** -20) * bound + 1e-30)
        return
    ref = direct.conv2d(xs, g, pad)
    if flags & B.WINO_FLAG_RELU:
        ref = np.maximum(ref, 0.0)
    err = h.normwise_err(y[sample], ref)
    print(f"    normwise err {err:.2e}", flush=True)
    assert err <= TOL[m]


def test_noalloc_matches_conv2d_in_a_row():
    for i, case in enumerate(CASES):
        N, C, H, W, K, pad, m, flags = case
        print(f"noalloc call {i}: N={N} C={C} {H}x{W} K={K} m={m} flags={flags:#x}", flush=True)
        x, g = _inputs(N, C, H, W, K, seed=10 + i)
        y0, y1 = _both(case, x, g)
        assert np.array_equal(y0, y1), i
        _check_oracle(case, x, g, y0, [0, N - 1] if N > 1 else [0])


def test_noalloc_auto_past_the_scratch_runs_fused():
    N, C, H, W, K, pad, m, flags = BIG_AUTO
    print(f"noalloc AUTO past the scratch: N={N} C={C} {H}x{W} K={K}", flush=True)
    assert B.wino_workspace_bytes(N, C, H, W, K, pad, m, flags) > B.WINO_NOALLOC_SCRATCH_BYTES
    x, g = _inputs(N, C, H, W, K, seed=20)
    hx = h.dev(x)
    U = _filters(g, C, K, m, flags)
    Ho, Wo, *_ = h.geometry(N, H, W, pad, m)
    y0 = h.empty_bytes(4 * N * K * Ho * Wo).reshape(N, K, Ho, Wo)
    B.check(B.wino_conv2d_noalloc(hx, U, y0, N, C, H, W, K, pad, m, flags), "wino_conv2d_noalloc")
    y1 = h.empty_bytes(4 * N * K * Ho * Wo).reshape(N, K, Ho, Wo)
    B.check(B.wino_conv2d(hx, U, y1, N, C, H, W, K, pad, m, B.WINO_ALGO_FUSED, None, 0), "wino_conv2d")
    y0, y1 = h.host(y0), h.host(y1)
    assert np.array_equal(y0, y1)
    _check_oracle(BIG_AUTO, x, g, y0, [0, N - 1])
    # then a smaller call through the scratch again
    case = CASES[3]
    N, C, H, W, K, pad, m, flags = case
    print(f"noalloc after it: N={N} C={C} {H}x{W} K={K} flags={flags:#x}", flush=True)
    x, g = _inputs(N, C, H, W, K, seed=21)
    y0, y1 = _both(case, x, g)
    assert np.array_equal(y0, y1)
    _check_oracle(case, x, g, y0, [0])
