"""The oracle's 16-bit rounding helpers and the reduced-precision reference
(fp16 / bf16 transform-domain operands), pinned on exactly representable
values, ties, and the full-precision limit (CPU only)."""
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
