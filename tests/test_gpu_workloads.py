"""The synthetic workloads at their full sizes, on the GPU, against the fp64 oracle.

Single layers small enough are checked whole; large batches are run whole on the
GPU and checked on sampled images (each image's output depends only on that
image).  Stacks are gated per layer -- the oracle recomputes each layer from the
GPU chain's own input to that layer -- and end to end against the oracle's own
fp64 chain."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from oracle import direct
from oracle import nn as onn
from paper_1903_01521_amd import binding as B
from paper_1903_01521_amd import workloads as wl

pytestmark = pytest.mark.gpu

TOL = {2: 1e-4, 4: 1e-3}
E2E_TOL = 1e-3


def _layer(hx: torch.Tensor, g: np.ndarray, L: wl.Layer) -> torch.Tensor:
    U = h.filter_transform(g, L.m)
    return h.conv2d(hx, U, L.K, L.pad, L.m, B.WINO_FLAG_RELU if L.relu else 0)


def _pool(hy: torch.Tensor) -> torch.Tensor:
    N, C, H, W = hy.shape
    out = torch.empty((N, C, H // 2, W // 2), dtype=torch.float32, device=h.DEV)
    B.check(B.wino_maxpool2x2(hy, out, N, C, H, W), "wino_maxpool2x2")
    return out


def _run_stack(w: wl.Workload, sample):
    """Run the whole stack on the GPU; gate every layer on the sampled images;
    return (GPU final output of the samples, the samples' input)."""
    x, gs = wl.generate(w)
    hx = h.dev(x)
    for li, (L, g) in enumerate(zip(w.layers, gs)):
        print(f"{w.name} layer {li}: C={L.C} K={L.K} {L.H}x{L.W} m={L.m}", flush=True)
        xin = h.host(hx)[sample].astype(np.float64)
        hy = _layer(hx, g, L)
        y = h.host(hy)[sample]
        ref = direct.conv2d(xin, g, L.pad)
        if L.relu:
            ref = onn.relu(ref)
        err = h.normwise_err(y, ref)
        print(f"  normwise err {err:.2e}", flush=True)
        assert err <= TOL[L.m], (li, err)
        hx = _pool(hy) if L.pool else hy
    return h.host(hx)[sample], x[sample], gs


def _oracle_chain(w: wl.Workload, x: np.ndarray, gs) -> np.ndarray:
    a = x.astype(np.float64)
    for L, g in zip(w.layers, gs):
        a = direct.conv2d(a, g, L.pad)
        if L.relu:
            a = onn.relu(a)
        if L.pool:
            a = onn.maxpool2x2(a)
    return a


@pytest.mark.parametrize("name", ["f2_n1_c32_k32_56x56", "f4_n1_c64_k64_112x112", "f4_n1_c48_k48_57x57",
                                  "f4_lowc_n1_c3_k64_224x224"])
def test_single_layer_whole(name):
    w = wl.WORKLOADS[name]
    L = w.first
    x, (g,) = wl.generate(w)
    print(f"{name}", flush=True)
    y = h.host(_layer(h.dev(x), g, L))
    ref = direct.conv2d(x, g, L.pad)
    err = h.normwise_err(y, ref)
    print(f"  normwise err {err:.2e}", flush=True)
    assert err <= TOL[L.m]


@pytest.mark.parametrize("name,algo", [("f4_n64_c256_k256_56x56", B.WINO_ALGO_AUTO),
                                       ("f4_n64_c256_k256_56x56", B.WINO_ALGO_STAGED),
                                       ("f4_n64_c256_k256_56x56", B.WINO_ALGO_FUSED),
                                       ("f4_lowc_n64_c3_k64_224x224", B.WINO_ALGO_AUTO)])
def test_large_batch_sampled(name, algo):
    """The whole batch on the GPU (AUTO: the split path for the 256-channel
    layer, low-C for the first layer; the staged and fused paths too), checked
    on sampled images."""
    w = wl.WORKLOADS[name]
    L = w.first
    x, (g,) = wl.generate(w)
    sample = [0, w.N // 2, w.N - 1]
    print(f"{name} algo {algo:#x} sample {sample}", flush=True)
    U = h.filter_transform(g, L.m)
    y = h.host(h.conv2d(h.dev(x), U, L.K, L.pad, L.m, algo | (B.WINO_FLAG_RELU if L.relu else 0)))[sample]
    ref = direct.conv2d(x[sample], g, L.pad)
    err = h.normwise_err(y, ref)
    print(f"  normwise err {err:.2e}", flush=True)
    assert err <= TOL[L.m]


def test_resnet_stage_n8():
    w = wl.WORKLOADS["f4_resnet_stage_n8_c128_28x28"]
    sample = list(range(w.N))
    out, x, gs = _run_stack(w, sample)
    ref = _oracle_chain(w, x, gs)
    err = h.normwise_err(out, ref)
    print(f"  end-to-end normwise err {err:.2e}", flush=True)
    assert err <= E2E_TOL


@pytest.mark.parametrize("name,sample", [("vgg16_stack_n1", [0]), ("vgg16_stack_n32", [0, 31])])
def test_vgg16_stack(name, sample):
    w = wl.WORKLOADS[name]
    out, x, gs = _run_stack(w, sample)
    ref = _oracle_chain(w, x, gs)
    err = h.normwise_err(out, ref)
    print(f"  end-to-end normwise err {err:.2e}", flush=True)
    assert err <= E2E_TOL


def test_large_batch_nhwc_split_sampled():
    """The 256-channel 56x56 layer at N=64 in channel-last layout on the split
    path (the launch the channel-last bench line times): sampled images against
    the fp64 oracle, and the whole batch bit for bit against the NCHW split
    path (the same V, GEMM and output transform; only x's and y's layout
    differ)."""
    from test_gpu_nhwc import conv_nhwc
    w = wl.WORKLOADS["f4_n64_c256_k256_56x56"]
    L = w.first
    x, (g,) = wl.generate(w)
    sample = [0, w.N // 2, w.N - 1]
    print(f"{w.name} channel-last split, sample {sample}", flush=True)
    U = h.filter_transform(g, L.m)
    x_nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    y = h.host(conv_nhwc(x_nhwc, U, L.K, L.pad, L.m, B.WINO_ALGO_SPLIT))
    del x_nhwc
    err = h.normwise_err(y[sample].transpose(0, 3, 1, 2), direct.conv2d(x[sample], g, L.pad))
    print(f"  normwise err {err:.2e}", flush=True)
    assert err <= TOL[L.m]
    y_nchw = h.host(h.conv2d(x, U, L.K, L.pad, L.m, B.WINO_ALGO_SPLIT))
    assert np.array_equal(y.transpose(0, 3, 1, 2), y_nchw)


@pytest.mark.parametrize("prec", ["fp16", "bf16"])
def test_large_batch_16bit_split_sampled(prec):
    """The same layer with 16-bit transform-domain operands on the split path
    (AUTO's choice there, and the launch the 16-bit bench line times): sampled
    images against the reduced-precision reference (U and V rounded once) within
    the rounding bound of the fp32 transforms and accumulation, and against the
    exact result within the error study's bound."""
    from test_gpu_prec16 import PRECS, STUDY, conv16, filter16, reference_and_bound
    flag, u, rnd = PRECS[prec]
    w = wl.WORKLOADS["f4_n64_c256_k256_56x56"]
    L = w.first
    x, (g,) = wl.generate(w)
    st, algo, _ = B.wino_plan_r(w.N, L.C, L.H, L.W, L.K, L.pad, L.m, 3, flag)
    assert st == B.WINO_OK and algo == B.WINO_ALGO_SPLIT
    sample = [0, w.N - 1]
    print(f"{w.name} 16-bit split {prec}, sample {sample}", flush=True)
    U16, _ = filter16(g, L.m, flag)
    y = conv16(x, U16, L.K, L.pad, L.m, flag | B.WINO_ALGO_SPLIT)[sample]
    assert np.all(np.isfinite(y))
    y16, bound = reference_and_bound(x[sample], g, L.pad, L.m, rnd)
    tol = (2 * u + 4 * L.C * 2.0 ** -24 + 2.0 ** -20) * bound
    assert np.all(np.abs(y - y16) <= tol + 1e-30)
    err = h.normwise_err(y, direct.conv2d(x[sample], g, L.pad))
    print(f"  normwise err against the exact result {err:.2e}", flush=True)
    assert err <= STUDY[(prec, L.m)]
