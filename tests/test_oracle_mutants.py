"""Plant plausible mistakes in copies of the oracle and check that the pins catch
every one (CPU only).  The oracle source itself is never modified."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import pins_direct
import pins_direct_rs

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "direct_conv.c")

# (name, original text, mutated text); every mutant keeps all accesses in bounds.
# MUTANTS change the 3x3 function, RS_MUTANTS the general R x S one.
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
RS_MUTANTS = [
    ("rs_flipped_rows", "const long u = i + r - pad;", "const long u = i + (R - 1 - r) - pad;"),
    ("rs_flipped_cols", "const long v = j + s - pad;", "const long v = j + (S - 1 - s) - pad;"),
    ("rs_transposed_taps", "gk[r * S + s]", "gk[s * R + r]"),
    ("rs_pad_offset", "const long v = j + s - pad;", "const long v = j + s - pad - 1;"),
    ("rs_dropped_channel", "for (long c = 0; c < C; ++c)", "for (long c = 1; c < C; ++c)"),
    ("rs_dropped_tap_row", "for (long r = 0; r < R; ++r)", "for (long r = 0; r < R - 1; ++r)"),
    ("rs_wrong_sign", "yo[i * Wo + j] += a * w;", "yo[i * Wo + j] += -a * w;"),
    ("rs_filter_k_c_swapped", "g + ((k * C + c) * (long)R) * S", "g + ((c * K + k) * (long)R) * S"),
    ("rs_no_zero_init", "yo[p] = 0.0;", "yo[p] = 1.0;"),
]
RS_SPLIT = "int oracle_conv2d_rs_f64"


def _build_lib(tmp_path, name, old, new, rs):
    src = open(SRC).read()
    head, tail = src.split(RS_SPLIT)
    part = tail if rs else head
    assert part.count(old) == 1, (name, old)
    part = part.replace(old, new)
    src = (head + RS_SPLIT + part) if rs else (part + RS_SPLIT + tail)
    path = tmp_path / f"{name}.c"
    path.write_text(src)
    lib = tmp_path / f"lib{name}.so"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                           "-std=c99", str(path), "-o", str(lib), "-lm"])
    return ctypes.CDLL(str(lib))


def _build_mutant(tmp_path, name, old, new):
    so = _build_lib(tmp_path, name, old, new, rs=False)
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


def _build_rs_mutant(tmp_path, name, old, new):
    so = _build_lib(tmp_path, name, old, new, rs=True)
    dp = ctypes.POINTER(ctypes.c_double)
    so.oracle_conv2d_rs_f64.argtypes = [dp, dp, dp] + [ctypes.c_int] * 9
    so.oracle_conv2d_rs_f64.restype = ctypes.c_int

    def conv(x, g, pad):
        x = np.ascontiguousarray(x, dtype=np.float64)
        g = np.ascontiguousarray(g, dtype=np.float64)
        N, C, H, W = x.shape
        K, _, R, S = g.shape
        y = np.empty((N, K, H + 2 * pad - (R - 1), W + 2 * pad - (S - 1)))
        rc = so.oracle_conv2d_rs_f64(x.ctypes.data_as(dp), g.ctypes.data_as(dp),
                                     y.ctypes.data_as(dp), N, C, H, W, K, R, S, pad, 0)
        assert rc == 0
        return y
    return conv


@pytest.mark.parametrize("mutant", RS_MUTANTS, ids=lambda m: m[0])
def test_rs_pins_catch_mutant(tmp_path, mutant):
    conv = _build_rs_mutant(tmp_path, *mutant)
    caught = []
    for check in pins_direct_rs.ALL_CHECKS:
        try:
            check(conv)
        except AssertionError:
            caught.append(check.__name__)
    assert caught, f"no pin caught mutant {mutant[0]}"


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
