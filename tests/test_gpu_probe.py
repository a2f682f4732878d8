"""The matrix-core peak probe: every wave's check value is exact (the launch did
all its MFMA work), for a short and a longer run."""
import pytest
import torch

import gpu_helpers as h
from paper_1903_01521_amd import binding as B

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("iters", [1, 37, 4096])
def test_mfma_probe_check_values(iters):
    print(f"mfma probe iters={iters}", flush=True)
    out = torch.full((2048,), float("nan"), dtype=torch.float32, device=h.DEV)
    B.check(B.wino_probe_mfma_f32(iters, out), "wino_probe_mfma_f32")
    got = h.host(out)
    assert (got == 32.0 * iters).all()
