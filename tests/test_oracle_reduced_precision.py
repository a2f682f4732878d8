"""The oracle's 16-bit rounding helpers and the reduced-precision reference
(fp16 / bf16 transform-domain operands), pinned on exactly representable
values, ties, and the full-precision limit (CPU only)."""
import os
import types

import numpy as np
import pytest

from oracle import cooktoom as ct
from oracle import direct


def test_round_bf16_known_values():
    # bf16 keeps 8 significant bits: 1 + 2^-7 is representable, 1 + 2^-8 is a tie
    # (rounds to even: 1), 1 + 3*2^-8 is a tie rounding up to 1 + 2^-6.
    v = np.array([1.0, 1 + 2**-7, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-8 + 2**-20, -3.0, 0.0, 255.0, 257.0])
    want = np.array([1.0, 1 + 2**-7, 1.0, 1 + 2**-6, 1 + 2**-7, -3.0, 0.0, 255.0, 256.0])
    assert np.array_equal(ct.round_bf16(v), want)


def test_round_fp16_known_values():
    v = np.array([1 + 2**-10, 1 + 2**-11, 1 + 3 * 2**-11, 2048.0, 2049.0, 65504.0, 1e-8])
    want = np.array([1 + 2**-10, 1.0, 1 + 2**-9, 2048.0, 2048.0, 65504.0, 0.0])
    assert np.array_equal(ct.round_fp16(v), want)


def test_rounding_error_bounds():
    rng = np.random.default_rng(1)
    a = rng.standard_normal(100000) * 10.0 ** rng.uniform(-3, 3, 100000)
    for fn, u in ((ct.round_bf16, 2.0**-8), (ct.round_fp16, 2.0**-11)):
        r = fn(a)
        big = np.abs(a) > 1e-4                        # clear of fp16's subnormal range
        assert np.all(np.abs(r[big] - a[big]) <= u * np.abs(a[big]))
        assert np.array_equal(fn(r), r)               # idempotent


# Normwise error of the reference against the direct definition on random
# data: about 5e-4 (fp16) and 4e-3 (bf16) for F(2x2,3x3), 7e-3 and 6e-2 for
# F(4x4,3x3), whose transforms amplify the operand rounding.
@pytest.mark.parametrize("prec,tol2,tol4", [("fp16", 2e-3, 2e-2), ("bf16", 2e-2, 1.5e-1)])
def test_reduced_precision_reference_is_close_to_direct(prec, tol2, tol4):
    # Small integers are exact in both formats while |U|, |V| stay small: the
    # reference then equals the direct definition; random data stays within a
    # multiple of the unit roundoff.
    rng = np.random.default_rng(2)
    x = rng.integers(-2, 3, (1, 4, 9, 9)).astype(np.float64)
    g = (rng.integers(-1, 2, (3, 4, 3, 3)) * 4).astype(np.float64)
    assert np.array_equal(ct.reduced_precision_conv_f64(x, g, 1, 2, prec), direct.conv2d(x, g, 1))
    x = rng.standard_normal((1, 16, 12, 12))
    g = rng.standard_normal((8, 16, 3, 3)) * 0.1
    ref = direct.conv2d(x, g, 1)
    for m, tol in ((2, tol2), (4, tol4)):
        y = ct.reduced_precision_conv_f64(x, g, 1, m, prec)
        err = np.abs(y - ref).max() / np.abs(ref).max()
        assert err < tol, (m, err)
        assert err > 1e-6                  # the rounding is really there


# ---------------------------------------------------------------------------
# Where the reference rounds: exactly U and V, nothing after the GEMMs.
#
# F(2x2,3x3), pad 0, a 4x4 image (one tile).  A pixel one-hot at (1,1) scaled by
# sx has V = sx * (B^T e B), whose entries are sx * {0, +-1}; a centre one-hot
# filter scaled by sg has U = sg * (G e G^T), entries sg * {0, +-1/4}.  Scaling
# by a power of two commutes with rounding, so with exact rational transforms
# the only output is y[0,0] = round(sx) * round(sg) when U and V are rounded,
# sx * sg when they are not.  1 + 2^-12 rounds to 1 in both formats; 1 + 2^-9
# is exact in fp16 (11 significant bits) and rounds to 1 in bf16 (8 bits).
# ---------------------------------------------------------------------------

def _one_tile(sx_per_channel, sg):
    C = len(sx_per_channel)
    x = np.zeros((1, C, 4, 4))
    for c, s in enumerate(sx_per_channel):
        x[0, c, 1, 1] = s
    g = np.zeros((1, C, 3, 3))
    g[0, :, 1, 1] = sg
    return x, g


def _expect(y00):
    want = np.zeros((1, 1, 2, 2))
    want[0, 0, 0, 0] = y00
    return want


def check_rounds_v(rp):
    for s, y16, yb16 in ((1 + 2.0**-12, 1.0, 1.0), (1 + 2.0**-9, 1 + 2.0**-9, 1.0)):
        x, g = _one_tile([s], 1.0)
        assert np.array_equal(rp(x, g, 0, 2, "fp16"), _expect(y16)), s
        assert np.array_equal(rp(x, g, 0, 2, "bf16"), _expect(yb16)), s


def check_rounds_u(rp):
    for s, y16, yb16 in ((1 + 2.0**-12, 1.0, 1.0), (1 + 2.0**-9, 1 + 2.0**-9, 1.0)):
        x, g = _one_tile([1.0], s)
        assert np.array_equal(rp(x, g, 0, 2, "fp16"), _expect(y16)), s
        assert np.array_equal(rp(x, g, 0, 2, "bf16"), _expect(yb16)), s


def check_keeps_gemm_sums_and_output_exact(rp):
    # two channels: V entries +-1 and +-2^-12, U entries +-1/4, all exact in
    # both formats; the channel sum 1/4 + 2^-14 (and y = 1 + 2^-12) is not
    # representable in either, so rounding M or y would show.
    x, g = _one_tile([1.0, 2.0**-12], 1.0)
    for prec in ("fp16", "bf16"):
        assert np.array_equal(rp(x, g, 0, 2, prec), _expect(1 + 2.0**-12)), prec


RP_CHECKS = [check_rounds_v, check_rounds_u, check_keeps_gemm_sums_and_output_exact]


@pytest.mark.parametrize("check", RP_CHECKS, ids=lambda c: c.__name__)
def test_reduced_precision_rounding_points(check):
    check(ct.reduced_precision_conv_f64)


_CT_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "cooktoom.py")

RP_MUTANTS = [
    ("v_not_rounded", "V = rnd(input_transform(x, pad, m))", "V = input_transform(x, pad, m)"),
    ("u_not_rounded", "U = rnd(filter_transform(g, m))", "U = filter_transform(g, m)"),
    ("m_rounded_too", "return output_transform(batched_gemm(U, V), N, Ho, Wo, m)",
     "return output_transform(rnd(batched_gemm(U, V)), N, Ho, Wo, m)"),
    ("y_rounded", "return output_transform(batched_gemm(U, V), N, Ho, Wo, m)",
     "return rnd(output_transform(batched_gemm(U, V), N, Ho, Wo, m))"),
    ("formats_swapped", '{"fp16": round_fp16, "bf16": round_bf16}', '{"fp16": round_bf16, "bf16": round_fp16}'),
    ("fp16_as_fp32", ".astype(np.float16).astype(np.float64)", ".astype(np.float32).astype(np.float64)"),
    ("bf16_seven_bits", "scaled = np.ldexp(m, 8)", "scaled = np.ldexp(m, 7)"),
]


@pytest.mark.parametrize("mutant", RP_MUTANTS, ids=lambda m: m[0])
def test_rounding_pins_catch_mutant(mutant):
    name, old, new = mutant
    src = open(_CT_SRC).read()
    assert src.count(old) == 1, name
    mod = types.ModuleType("ct_" + name)
    exec(compile(src.replace(old, new), "ct_" + name, "exec"), mod.__dict__)
    caught = []
    for check in RP_CHECKS:
        try:
            check(mod.reduced_precision_conv_f64)
        except AssertionError:
            caught.append(check.__name__)
    assert caught, f"no pin caught mutant {name}"
