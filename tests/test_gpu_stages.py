"""Each stage of the staged path, called alone through the C-ABI, against the
oracle's fp64 stage references (GPU)."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import cooktoom as ct
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24          # unit roundoff of fp32


@pytest.mark.parametrize("m", [2, 4])
# small layers take one wave per (filter pair, position group); from 512 filter
# pairs on (the last three shapes) one wave per pair computes every position,
# reading g through LDS when the channel quads come in fours (the last two)
@pytest.mark.parametrize("C,K", [(3, 20), (16, 16), (37, 5), (64, 64), (130, 250), (126, 120), (512, 512)])
def test_filter_transform(m, C, K):
    rng = np.random.default_rng(100 + C + K + m)
    _, g = wl.random_layer(rng, 1, C, 4, 4, K)
    print(f"filter_transform m={m} C={C} K={K}", flush=True)
    U = h.host(h.filter_transform(g, m))
    full = h.unpack_U(U, C, K, m, crop=False)
    got = full[:, :C, :K].astype(np.float64)
    ref = ct.filter_transform(g.astype(np.float64), m)
    # fp64 inside, one rounding to fp32: within one fp32 ulp of the fp64 value.
    assert np.all(np.abs(got - ref) <= 2 * U32 * np.abs(ref) + 1e-45)
    # padding channels / filters are exactly zero
    pad_mask = np.ones(full.shape, bool)
    pad_mask[:, :C, :K] = False
    assert np.all(full[pad_mask] == 0)


@pytest.mark.parametrize("shape", [(2, 5, 9, 11, 1), (1, 3, 6, 6, 0), (1, 8, 57, 57, 1), (3, 4, 1, 1, 1)])
def test_input_transform_m2_is_bit_exact(shape):
    N, C, H, W, pad = shape
    rng = np.random.default_rng(sum(shape))
    x, _ = wl.random_layer(rng, N, C, H, W, 1)
    print(f"input_transform m=2 shape={shape}", flush=True)
    V = h.host(h.input_transform(x, pad, 2))
    Ho, Wo, th, tw, P = h.geometry(N, H, W, pad, 2)
    full = h.unpack_V(V, C, P, 2, crop=False)
    ref = ct.input_transform_m2_paper_order_f32(x, pad)
    assert full.dtype == np.float32
    assert np.array_equal(full[:, :C, :P], ref)
    mask = np.ones(full.shape, bool)
    mask[:, :C, :P] = False
    assert np.all(full[mask] == 0)


@pytest.mark.parametrize("shape", [(2, 5, 9, 11, 1), (1, 8, 57, 57, 1), (1, 3, 7, 6, 0), (2, 4, 12, 12, 2)])
def test_input_transform_m4(shape):
    N, C, H, W, pad = shape
    rng = np.random.default_rng(7 * sum(shape))
    x, _ = wl.random_layer(rng, N, C, H, W, 1)
    print(f"input_transform m=4 shape={shape}", flush=True)
    V = h.host(h.input_transform(x, pad, 4))
    Ho, Wo, th, tw, P = h.geometry(N, H, W, pad, 4)
    full = h.unpack_V(V, C, P, 4, crop=False)
    ref = ct.input_transform(x.astype(np.float64), pad, 4)
    _, _, BT = ct.matrices_f64(4)
    d = ct.extract_regions(np.abs(x.astype(np.float64)), pad, 4)
    bound = np.einsum("au,nctjuv,bv->abcntj", np.abs(BT), d, np.abs(BT)).reshape(36, C, P)
    # two passes of at most 6-term sums with exact small-integer coefficients
    assert np.all(np.abs(full[:, :C, :P] - ref) <= 12 * U32 * bound)
    mask = np.ones(full.shape, bool)
    mask[:, :C, :P] = False
    assert np.all(full[mask] == 0)


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("shape", [(1, 16, 20, 20, 16), (2, 7, 9, 13, 33), (1, 64, 30, 30, 64), (1, 3, 8, 8, 70)])
def test_batched_gemm(m, shape):
    N, C, H, W, K = shape
    pad = 1
    rng = np.random.default_rng(sum(shape) + m)
    x, g = wl.random_layer(rng, N, C, H, W, K)
    print(f"batched_gemm m={m} shape={shape}", flush=True)
    U = h.filter_transform(g, m)
    V = h.input_transform(x, pad, m)
    M = h.host(h.batched_gemm(U, V, N, C, H, W, K, pad, m))
    Ho, Wo, th, tw, P = h.geometry(N, H, W, pad, m)
    Ul = h.unpack_U(h.host(U), C, K, m).astype(np.float64)
    Vl = h.unpack_V(h.host(V), C, P, m).astype(np.float64)
    got = h.unpack_M(M, K, P, m)
    ref = ct.batched_gemm(Ul, Vl)
    bound = ct.batched_gemm(np.abs(Ul), np.abs(Vl))
    # any summation order, FMA or not: |err| <= gamma_C * sum |u||v|
    assert np.all(np.abs(got - ref) <= (C + 2) * U32 * bound + 1e-38)


@pytest.mark.parametrize("m", [2, 4])
@pytest.mark.parametrize("relu", [False, True])
# (N, K, H, W, pad); the kernel takes whole rows of tiles (several rows per
# workgroup up to 64 tiles, a ragged last group) or 64-tile pieces of rows
# wider than that (the last two shapes)
@pytest.mark.parametrize("shape", [(1, 16, 20, 20, 1), (2, 33, 9, 13, 1), (1, 5, 57, 57, 1), (1, 1, 3, 3, 0),
                                   (3, 18, 37, 26, 2), (2, 20, 10, 300, 1), (1, 7, 6, 515, 0)])
def test_output_transform(m, relu, shape):
    N, K, H, W, pad = shape
    Ho, Wo, th, tw, P = h.geometry(N, H, W, pad, m)
    T = (m + 2) ** 2
    rng = np.random.default_rng(sum(shape) + 3 * m + relu)
    Ml = rng.standard_normal((T, K, P)).astype(np.float32)
    print(f"output_transform m={m} relu={relu} shape={shape}", flush=True)
    Md = h.dev(h.pack_M(Ml, K, P, m))
    y = h.host(h.output_transform(Md, N, K, H, W, pad, m, flags=1 if relu else 0))
    ref = ct.output_transform(Ml.astype(np.float64), N, Ho, Wo, m)
    AT, _, _ = ct.matrices_f64(m)
    absAT = np.abs(AT)
    a = m + 2
    Mr = np.abs(Ml.astype(np.float64)).reshape(a, a, K, N, th, tw)
    bound = np.einsum("iu,uvkntw,jv->nktiwj", absAT, Mr, absAT).reshape(N, K, th * m, tw * m)[:, :, :Ho, :Wo]
    if relu:
        ref = np.maximum(ref, 0.0)
    assert y.shape == ref.shape
    assert np.all(np.abs(y - ref) <= 12 * U32 * bound)


def test_maxpool2x2():
    from oracle import nn
    rng = np.random.default_rng(5)
    for (N, C, H, W) in [(2, 3, 8, 8), (1, 5, 7, 9), (1, 1, 2, 2)]:
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        y = torch.empty((N, C, H // 2, W // 2), dtype=torch.float32, device=h.DEV)
        from paper_1903_01521_amd import binding as B
        B.check(B.wino_maxpool2x2(h.dev(x), y, N, C, H, W))
        assert np.array_equal(h.host(y), nn.maxpool2x2(x.astype(np.float64)).astype(np.float32))
