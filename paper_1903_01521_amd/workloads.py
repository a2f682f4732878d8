"""Seeded synthetic workloads: layer shapes and input generators.

This module holds no arithmetic of the method.  It is the one module that both
the HIP path's tests/benchmark and the oracle-side checks draw their inputs
from, so that both see identical fp32 arrays.

Shapes stand in for the 3x3 (and 5x5) layers of the CNNs the paper evaluates
(Sec. 3: VGG-16/19, GoogleNet, Inception-v3, SqueezeNet); no dataset images or
trained weights are used.  Recipe: ``numpy.random.default_rng(seed)`` (PCG64),
the input tensor is drawn first, then each layer's weights in layer order, all
in fp64 and then rounded to fp32.  Weights are He-normal, i.e. N(0, variance
2/(r*r*C_in)) for r x r filters.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Layer:
    C: int
    K: int
    H: int
    W: int
    m: int
    pad: int = 1
    relu: bool = False        # ReLU applied to this layer's output
    pool: bool = False        # 2x2/2 max-pool applied after (the ReLU of) this layer
    r: int = 3                # filter side (3, or 5 with m = 2), or a 1-D filter's length
    axis: str = ""            # "" for r x r filters; "w" for 1 x r, "h" for r x 1 (1-D layers)
    nhwc: bool = False        # channel-last x and y (the generator still returns x as NCHW)


@dataclass(frozen=True)
class Workload:
    name: str
    N: int
    layers: tuple
    x_dist: str = "normal"    # "normal": N(0,1); "uniform": U(-1,1)
    note: str = ""

    @property
    def first(self) -> Layer:
        return self.layers[0]


def _vgg16(N: int) -> Workload:
    spec = [(3, 64, 224), (64, 64, 224), None,
            (64, 128, 112), (128, 128, 112), None,
            (128, 256, 56), (256, 256, 56), (256, 256, 56), None,
            (256, 512, 28), (512, 512, 28), (512, 512, 28), None,
            (512, 512, 14), (512, 512, 14), (512, 512, 14), None]
    layers = []
    for i, s in enumerate(spec):
        if s is None:
            continue
        C, K, HW = s
        pool = i + 1 < len(spec) and spec[i + 1] is None
        layers.append(Layer(C, K, HW, HW, m=2 if HW == 14 else 4, relu=True, pool=pool))
    return Workload(f"vgg16_stack_n{N}", N, tuple(layers),
                    note="13 VGG-16 3x3 layers, ReLU after each, 2x2 max-pool between blocks; "
                         "F(4x4,3x3), F(2x2,3x3) at 14x14")


WORKLOADS = {w.name: w for w in [
    Workload("f2_n1_c32_k32_56x56", 1, (Layer(32, 32, 56, 56, m=2),),
             note="single 3x3 layer, F(2x2,3x3)"),
    Workload("f4_n1_c64_k64_112x112", 1, (Layer(64, 64, 112, 112, m=4),),
             note="single 3x3 layer, F(4x4,3x3)"),
    Workload("f4_n1_c48_k48_57x57", 1, (Layer(48, 48, 57, 57, m=4),),
             note="ragged edge tiles: 15x15 tiles, the last with one valid row/column"),
    Workload("f4_resnet_stage_n8_c128_28x28", 8,
             tuple(Layer(128, 128, 28, 28, m=4, relu=(i < 3)) for i in range(4)),
             note="four 3x3 layers, ReLU between"),
    _vgg16(1),
    _vgg16(32),
    Workload("f4_n64_c256_k256_56x56", 64, (Layer(256, 256, 56, 56, m=4),),
             x_dist="uniform", note="large-batch throughput layer"),
    Workload("f4_lowc_n64_c3_k64_224x224", 64, (Layer(3, 64, 224, 224, m=4),),
             x_dist="uniform", note="low-C first layer"),
    Workload("f4_lowc_n1_c3_k64_224x224", 1, (Layer(3, 64, 224, 224, m=4),),
             x_dist="uniform", note="low-C first layer, batch 1"),
    Workload("f2r5_n32_c48_k64_35x35", 32, (Layer(48, 64, 35, 35, m=2, pad=2, r=5),),
             note="5x5 layer shaped like Inception-v3's 5x5 branch, F(2x2,5x5)"),
    Workload("f4_nhwc_n64_c256_k256_56x56", 64, (Layer(256, 256, 56, 56, m=4, nhwc=True),),
             x_dist="uniform", note="the large-batch layer with channel-last tensors"),
    Workload("f2r7w_n32_c192_k160_17x17", 32, (Layer(192, 160, 17, 17, m=2, pad=3, r=7, axis="w"),),
             note="1x7 layer shaped like Inception-v3's 17x17 blocks, F(1x2,1x7,1x8)"),
    Workload("f2r7h_n32_c192_k160_17x17", 32, (Layer(192, 160, 17, 17, m=2, pad=3, r=7, axis="h"),),
             note="7x1 layer shaped like Inception-v3's 17x17 blocks, F(2x1,7x1,8x1)"),
]}

# The single-layer workload the benchmark times by default: the largest
# single-GPU layer (N=64, C=K=256, 56x56, F(4x4,3x3)).
DEFAULT_BENCH = "f4_n64_c256_k256_56x56"


def generate(w: Workload, seed: int = 0, N: int | None = None):
    """Draw (x, [g_layer, ...]) as fp32 arrays: x [N,C,H,W], g [K,C,R,S]."""
    rng = np.random.default_rng(seed)
    L0 = w.first
    n = w.N if N is None else N
    shape = (n, L0.C, L0.H, L0.W)
    if w.x_dist == "normal":
        x = rng.standard_normal(shape)
    elif w.x_dist == "uniform":
        x = rng.uniform(-1.0, 1.0, shape)
    else:
        raise ValueError(w.x_dist)
    x = x.astype(np.float32)
    gs = []
    for L in w.layers:
        R, S = {"": (L.r, L.r), "w": (1, L.r), "h": (L.r, 1)}[L.axis]
        std = np.sqrt(2.0 / (R * S * L.C))
        gs.append((rng.standard_normal((L.K, L.C, R, S)) * std).astype(np.float32))
    return x, gs


def random_layer(rng: np.random.Generator, N: int, C: int, H: int, W: int, K: int,
                 kind: str = "normal"):
    """Free-form seeded inputs for parity cases: kind 'normal' (x N(0,1), He-normal
    g) or 'int' (small integers, x in [-4, 4], g in [-3, 3])."""
    if kind == "normal":
        x = rng.standard_normal((N, C, H, W)).astype(np.float32)
        g = (rng.standard_normal((K, C, 3, 3)) * np.sqrt(2.0 / (9.0 * C))).astype(np.float32)
    elif kind == "int":
        x = rng.integers(-4, 5, (N, C, H, W)).astype(np.float32)
        g = rng.integers(-3, 4, (K, C, 3, 3)).astype(np.float32)
    else:
        raise ValueError(kind)
    return x, g
