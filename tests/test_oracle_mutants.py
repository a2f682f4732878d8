"""Plant plausible mistakes in copies of the oracle and check that the pins catch
every one (CPU only).  The oracle source itself is never modified."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import pins_direct

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "direct_conv.c")

# (name, original text, mutated text); every mutant keeps all accesses in bounds.
MUTANTS = [
    ("flipped_rows", "const long u = i + r - pad;", "const long u = i + (2 - r) - pad;"),
    ("flipped_cols", "const long v = j + s - pad;", "const long v = j + (2 - s) - pad;"),
    ("transposed_taps", "gk[r * 3 + s]", "gk[s * 3 + r]"),
    ("pad_offset", "const long u = i + r - pad;", "const long u = i + r - pad + 1;"),
    ("dropped_channel", "for (long c = 0; c < C; ++c)", "for (long c = 0; c < C - 1; ++c)"),
    ("dropped_tap_column", "for (long s = 0; s < 3; ++s)", "for (long s = 0; s < 2; ++s)"),
    ("wrong_sign", "yo[i * Wo + j] += a * w;", "yo[i * Wo + j] -= a * w;"),
    ("filter_k_c_swapped", "g + ((k * C + c) * 3L) * 3L", "g + ((c * K + k) * 3L) * 3L"),
    ("no_zero_init", "yo[p] = 0.0;", "yo[p] = 0.5;"),
    ("abs_of_weights_always", "if (absval) w = fabs(w);", "w = fabs(w);"),
]


def _build_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, (name, old)
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                           "-std=c99", str(path), "-o", str(lib), "-lm"])
    so = ctypes.CDLL(str(lib))
    dp = ctypes.POINTER(ctypes.c_double)
    so.oracle_conv2d_f64.argtypes = [dp, dp, dp] + [ctypes.c_int] * 7
    so.oracle_conv2d_f64.restype = ctypes.c_int

    def conv(x, g, pad):
        x = np.ascontiguousarray(x, dtype=np.float64)
        g = np.ascontiguousarray(g, dtype=np.float64)
        N, C, H, W = x.shape
        K = g.shape[0]
        y = np.empty((N, K, H + 2 * pad - 2, W + 2 * pad - 2))
        rc = so.oracle_conv2d_f64(x.ctypes.data_as(dp), g.ctypes.data_as(dp),
                                  y.ctypes.data_as(dp), N, C, H, W, K, pad, 0)
        assert rc == 0
        return y
    return conv


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_mutant(tmp_path, mutant):
    conv = _build_mutant(tmp_path, *mutant)
    caught = []
    for check in pins_direct.ALL_CHECKS:
        try:
            check(conv)
        except AssertionError:
            caught.append(check.__name__)
    assert caught, f"no pin caught mutant {mutant[0]}"
