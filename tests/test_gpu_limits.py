"""Layers at the size limits of the 32-bit offsets the input kernels form
(include/wino.h: an image under 1 GiB for the fused and split kernels; the
images of one 16-tile block under 1 GiB for the staged input transform), with
two images so the second image's base lies past 1 GiB.  Outputs are sampled
across both images (corners, edges, the far end of the second image) and each
is checked against its direct fp64 sum."""
import numpy as np
import pytest
import torch

import gpu_helpers as h
from paper_1903_01521_amd import binding as B

pytestmark = pytest.mark.gpu

ELEM = {2: 2e-5, 4: 2e-4}     # elementwise, scaled by the tile's largest |x|*|g| sum


def sampled_check(x, g, y, pad, m, n_samples=384, seed=0):
    N, C, H, W = x.shape
    K = g.shape[0]
    Ho, Wo = y.shape[2], y.shape[3]
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.integers(0, s, n_samples) for s in (N, K, Ho, Wo)], axis=1)
    idx[:6] = [[0, 0, 0, 0], [N - 1, K - 1, Ho - 1, Wo - 1], [0, K - 1, 0, Wo - 1], [N - 1, 0, Ho - 1, 0],
               [N - 1, K // 2, Ho // 2, Wo - 1], [0, 0, Ho - 1, Wo // 2]]
    g64 = g.detach().cpu().double().numpy()
    for n, k, i, j in idx:
        ti, tj = i // m * m, j // m * m
        r0, c0 = ti - pad, tj - pad                      # the tile's input region, m + 2 square
        win = np.zeros((C, m + 2, m + 2))
        a0, a1 = max(r0, 0), min(r0 + m + 2, H)
        b0, b1 = max(c0, 0), min(c0 + m + 2, W)
        win[:, a0 - r0:a1 - r0, b0 - c0:b1 - c0] = x[n, :, a0:a1, b0:b1].cpu().double().numpy()
        di, dj = i - ti, j - tj
        ref = np.sum(win[:, di:di + 3, dj:dj + 3] * g64[k])
        scale = max(np.sum(np.abs(win[:, a:a + 3, b:b + 3]) * np.abs(g64[k]))
                    for a in range(m) for b in range(m))
        got = float(y[n, k, i, j])
        assert abs(got - ref) <= ELEM[m] * (scale + 1e-30), (n, k, i, j, got, ref)


def run(N, C, H, W, K, pad, m, flags):
    gen = torch.Generator(device=h.DEV).manual_seed(1234)
    x = torch.randn((N, C, H, W), generator=gen, device=h.DEV, dtype=torch.float32)
    g = torch.randn((K, C, 3, 3), generator=gen, device=h.DEV, dtype=torch.float32) * (2.0 / (9 * C)) ** 0.5
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    U = h.empty_bytes(B.wino_filter_bytes(C, K, m))
    B.check(B.wino_filter_transform(g, U, C, K, m), "wino_filter_transform")
    y = torch.full((N, K, Ho, Wo), float("nan"), dtype=torch.float32, device=h.DEV)
    wsb = B.wino_workspace_bytes(N, C, H, W, K, pad, m, flags)
    assert wsb != 2**64 - 1
    ws = h.empty_bytes(wsb) if wsb else None
    B.check(B.wino_conv2d(x, U, y, N, C, H, W, K, pad, m, flags, ws, wsb), "wino_conv2d")
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all())
    return x, g, y


@pytest.mark.parametrize("m,algo", [(4, B.WINO_ALGO_FUSED), (2, B.WINO_ALGO_FUSED), (4, B.WINO_ALGO_SPLIT)],
                         ids=["fused-m4", "fused-m2", "split-m4"])
def test_image_just_under_1gib(m, algo):
    # 64 x 2040 x 2040 fp32 = 1 065 369 600 bytes per image, 2 images
    N, C, H, W, K, pad = 2, 64, 2040, 2040, 16, 1
    assert N * C * H * W * 4 > 2 ** 30 > C * H * W * 4
    print(f"limits m={m} algo={algo:#x}", flush=True)
    x, g, y = run(N, C, H, W, K, pad, m, algo)
    sampled_check(x, g, y, pad, m)
    # one image more than the limit is rejected before any launch
    assert B.wino_workspace_bytes(1, 64, 2048, 2048, K, pad, m, algo) == 2**64 - 1


def test_staged_block_images_just_under_1gib():
    # the staged input transform spans 2 images per 16-tile block here:
    # 2 x 64 x 1400 x 1400 fp32 = 1 003 520 000 bytes
    N, C, H, W, K, pad, m = 2, 64, 1400, 1400, 16, 1, 4
    print("limits staged", flush=True)
    x, g, y = run(N, C, H, W, K, pad, m, B.WINO_ALGO_STAGED)
    sampled_check(x, g, y, pad, m)
    assert B.wino_workspace_bytes(N, C, 1450, 1450, K, pad, m, B.WINO_ALGO_STAGED) == 2**64 - 1
