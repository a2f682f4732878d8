"""fp64 direct convolution oracle (test infrastructure only).

Wraps ``liboracle.so`` (compiled from ``direct_conv.c`` with gcc, -O2,
-ffp-contract=off, OpenMP over (n, k)).  The definition it computes is the
multi-channel correlation that Eq. 1 of the paper reaches exactly over the
rationals (Sec. 2, Eq. 1 and Listing 1): see the header of ``direct_conv.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "direct_conv.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()


def build(force: bool = False) -> str:
    """Compile liboracle.so next to its source; returns the library path."""
    if force or not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", "-std=c99", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH) or (
                    os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
                build()
            lib = ctypes.CDLL(_LIB_PATH)
            dp = ctypes.POINTER(ctypes.c_double)
            lib.oracle_conv2d_f64.argtypes = [dp, dp, dp] + [ctypes.c_int] * 7
            lib.oracle_conv2d_f64.restype = ctypes.c_int
            lib.oracle_conv2d_rs_f64.argtypes = [dp, dp, dp] + [ctypes.c_int] * 9
            lib.oracle_conv2d_rs_f64.restype = ctypes.c_int
            lib.oracle_num_threads.argtypes = []
            lib.oracle_num_threads.restype = ctypes.c_int
            _lib = lib
    return _lib


def out_hw(H: int, W: int, pad: int, R: int = 3, S: int = 3) -> tuple[int, int]:
    """Output size of an R x S stride-1 layer with symmetric zero padding."""
    return H + 2 * pad - (R - 1), W + 2 * pad - (S - 1)


def conv2d(x: np.ndarray, g: np.ndarray, pad: int, absval: bool = False) -> np.ndarray:
    """y = x (*) g, stride-1 cross-correlation with zero padding, in fp64.

    x: [N, C, H, W] (any real dtype; widened exactly to fp64)
    g: [K, C, R, S]: 3 x 3 (the method's filters), or any other size (the 5 x 5
       layers of the paper's Table 2)
    Returns y: [N, K, Ho, Wo] fp64.  absval=True evaluates the same sums on |x|
    and |g| (the elementwise magnitude bound used to scale rounding error).
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    g = np.ascontiguousarray(g, dtype=np.float64)
    N, C, H, W = x.shape
    K, C2, R, S = g.shape
    if C2 != C or R < 1 or S < 1:
        raise ValueError("filter must be [K, C, R, S] with C matching x")
    Ho, Wo = out_hw(H, W, pad, R, S)
    if pad < 0 or Ho < 1 or Wo < 1:
        raise ValueError("invalid padding / size")
    y = np.empty((N, K, Ho, Wo), dtype=np.float64)
    dp = ctypes.POINTER(ctypes.c_double)
    if (R, S) == (3, 3):
        rc = _load().oracle_conv2d_f64(x.ctypes.data_as(dp), g.ctypes.data_as(dp),
                                       y.ctypes.data_as(dp), N, C, H, W, K, pad,
                                       1 if absval else 0)
    else:
        rc = _load().oracle_conv2d_rs_f64(x.ctypes.data_as(dp), g.ctypes.data_as(dp),
                                          y.ctypes.data_as(dp), N, C, H, W, K, R, S, pad,
                                          1 if absval else 0)
    if rc != 0:
        raise RuntimeError("oracle direct convolution rejected its arguments")
    return y


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loop uses in this process."""
    return int(_load().oracle_num_threads())
