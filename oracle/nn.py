"""fp64 glue for layer stacks (test infrastructure only): ReLU and 2x2/2 max-pool.

The paper evaluates the convolution layers of whole CNNs (Sec. 3); between the
3x3 layers of a VGG-style stack sit a ReLU and, between blocks, a 2x2 stride-2
max-pool.  These are the plain definitions, applied to the oracle's own fp64
tensors.
"""
import numpy as np


def relu(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0)


def maxpool2x2(x: np.ndarray) -> np.ndarray:
    """2x2 window, stride 2, floor of odd sizes: y[n,c,i,j] = max over x[n,c,2i+a,2j+b]."""
    N, C, H, W = x.shape
    Ho, Wo = H // 2, W // 2
    y = np.full((N, C, Ho, Wo), -np.inf, dtype=np.float64)
    for a in range(2):
        for b in range(2):
            y = np.maximum(y, x[:, :, a:2 * Ho:2, b:2 * Wo:2])
    return y
