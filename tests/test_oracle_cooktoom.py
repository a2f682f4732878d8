"""Exact Cook-Toom matrices and the rational Eq. 1 / Listing 1 evaluation, pinned
against what the paper prints and against the direct definition (CPU only)."""
import os
from fractions import Fraction as Q

import numpy as np
import pytest

from oracle import cooktoom as ct
from oracle import direct

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "f2x2_3x3_input_transform.txt")


def _read_golden():
    blocks, cur = {}, None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line in ("XT", "X", "OPS"):
            cur = blocks.setdefault(line, [])
            continue
        cur.append(line)
    XT = [[int(v) for v in r.split()] for r in blocks["XT"]]
    X = [[int(v) for v in r.split()] for r in blocks["X"]]
    ops = []
    for r in blocks["OPS"]:
        out, rhs = r.split("=")
        a, op, b = rhs.split()
        ops.append((int(out), int(a), op, int(b)))
    return XT, X, ops


def test_m2_input_matrix_is_the_printed_one():
    XT, X, _ = _read_golden()
    _, _, BT = ct.cook_toom(2)
    assert [[int(v) for v in r] for r in BT] == XT
    # The paper prints X as well; it must be the transpose of X^T.
    assert [list(r) for r in zip(*XT)] == X


def test_printed_row_sequence_is_bt():
    # The printed add/sub sequence, applied to the unit rows, must give B^T's rows.
    _, _, ops = _read_golden()
    _, _, BT = ct.cook_toom(2)
    unit = [[int(i == j) for j in range(4)] for i in range(4)]
    rows = [None] * 4
    for out, a, op, b in ops:
        sgn = 1 if op == "+" else -1
        rows[out] = [unit[a][j] + sgn * unit[b][j] for j in range(4)]
    assert rows == [[int(v) for v in r] for r in BT]


@pytest.mark.parametrize("m,r", [(2, 3), (4, 3), (2, 5)])
def test_bilinear_identity_1d(m, r):
    # F(m, r) computes y[i] = sum_k g[k] d[i+k] for every g, d: check on all basis pairs.
    AT, G, BT = ct.cook_toom(m, r)
    a = m + r - 1
    for kk in range(r):
        for aa in range(a):
            for i in range(m):
                s = sum((AT[i][j] * G[j][kk] * BT[j][aa] for j in range(a)), Q(0))
                assert s == (1 if aa == i + kk else 0), (m, r, i, kk, aa, s)


@pytest.mark.parametrize("m,r", [(2, 3), (4, 3), (2, 5)])
def test_matrix_shapes_and_points(m, r):
    AT, G, BT = ct.cook_toom(m, r)
    a = m + r - 1
    assert len(AT) == m and all(len(row) == a for row in AT)
    assert len(G) == a and all(len(row) == r for row in G)
    assert len(BT) == a and all(len(row) == a for row in BT)
    # A^T and B^T are integer matrices (the fractions sit in G, applied offline).
    assert all(v.denominator == 1 for row in AT + BT for v in row)


def test_f2x2_5x5_shares_the_input_transform_of_f4x4_3x3():
    # Both have alpha = 6 and the points {0, +-1, +-2, inf}: B^T depends only on
    # the points, so the 5x5 variant reuses the 6x6 input transform.
    assert ct.cook_toom(2, 5)[2] == ct.cook_toom(4, 3)[2]
    # ... while A^T keeps the first two rows of F(4,3)'s except the point at
    # infinity, which picks the leading output coefficient (row m - 1 = 1).
    AT5, AT3 = ct.cook_toom(2, 5)[0], ct.cook_toom(4, 3)[0]
    assert [row[:5] for row in AT5] == [row[:5] for row in AT3[:2]]
    assert [row[5] for row in AT5] == [0, 1]


def test_unsupported_pairs_are_rejected():
    for m, r in [(3, 3), (4, 5), (2, 7)]:
        with pytest.raises(ValueError):
            ct.cook_toom(m, r)


# Fig. 2's example: a 3 x 6 x 6 input, four filters, F(2x2,3x3) -> 2x2 regions of
# 4x4 (valid convolution, so pad 0), plus padded, ragged, batched and m=4 cases.
EXACT_CASES = [
    (1, 3, 6, 6, 4, 0, 2),
    (2, 2, 5, 7, 3, 1, 2),
    (1, 2, 6, 6, 2, 0, 4),
    (1, 2, 7, 9, 3, 1, 4),
    (2, 1, 5, 5, 2, 2, 4),
]


# F(2x2,5x5): valid, padded (pad 2 keeps the size), ragged and one-pixel cases.
EXACT_CASES_5 = [
    (1, 2, 6, 6, 2, 0, 2),
    (1, 2, 7, 9, 3, 2, 2),
    (2, 1, 5, 8, 2, 1, 2),
    (1, 3, 1, 1, 2, 2, 2),
]


@pytest.mark.parametrize("case,r", [(c, 3) for c in EXACT_CASES] + [(c, 5) for c in EXACT_CASES_5])
def test_listing1_over_rationals_equals_direct(case, r):
    N, C, H, W, K, pad, m = case
    rng = np.random.default_rng(sum(case) + r)
    x = rng.integers(-6, 7, (N, C, H, W))
    g = rng.integers(-6, 7, (K, C, r, r))
    yq = ct.winograd_conv_exact(x, g, pad, m)
    yd = direct.conv2d(x.astype(np.float64), g.astype(np.float64), pad)
    assert np.array(yq, dtype=object).shape == yd.shape
    assert all(Q(int(v)) == v for v in np.ravel(np.array(yq, dtype=object)))
    assert np.array_equal(np.array(yq, dtype=np.float64), yd)


@pytest.mark.parametrize("m,r", [(2, 3), (4, 3), (2, 5)])
@pytest.mark.parametrize("shape", [(1, 3, 6, 6, 4, 0), (2, 5, 9, 7, 6, 1), (1, 4, 57, 57, 3, 1),
                                   (3, 2, 1, 1, 2, 1), (1, 1, 5, 5, 1, 0)])
def test_fp64_stages_compose_to_direct(m, r, shape):
    N, C, H, W, K, pad = shape
    if r == 5:
        pad += 1                     # keep Ho, Wo >= 1 for the one-pixel shape
    rng = np.random.default_rng(N * 100 + C + H + r)
    x = rng.standard_normal((N, C, H, W))
    g = rng.standard_normal((K, C, r, r))
    yw = ct.winograd_conv_f64(x, g, pad, m)
    yd = direct.conv2d(x, g, pad)
    bound = direct.conv2d(x, g, pad, absval=True)
    assert yw.shape == yd.shape
    assert np.all(np.abs(yw - yd) <= 1e-12 * (bound + 1e-300))


def test_stage_layouts():
    N, C, H, W, K, pad, m = 2, 3, 10, 9, 5, 1, 4
    rng = np.random.default_rng(11)
    x = rng.standard_normal((N, C, H, W))
    g = rng.standard_normal((K, C, 3, 3))
    Ho, Wo, th, tw, P = ct.geometry(N, H, W, pad, m)
    U = ct.filter_transform(g, m)
    V = ct.input_transform(x, pad, m)
    assert U.shape == (36, C, K) and V.shape == (36, C, P)
    _, G, BT = ct.matrices_f64(m)
    # Spot-check one element of each against its definition.
    k, c, xi, nu = 3, 2, 4, 1
    assert np.isclose(U[xi * 6 + nu, c, k], (G @ g[k, c] @ G.T)[xi, nu], rtol=1e-15, atol=1e-15)
    n, ti, tj = 1, 2, 0
    p = (n * th + ti) * tw + tj
    xe = np.pad(x[n, c], ((pad, 20), (pad, 20)))
    d = xe[ti * m:ti * m + 6, tj * m:tj * m + 6]
    assert np.isclose(V[xi * 6 + nu, c, p], (BT @ d @ BT.T)[xi, nu], rtol=1e-14, atol=1e-14)


def test_paper_order_f32_is_exact_on_integers():
    rng = np.random.default_rng(12)
    x = rng.integers(-1000, 1001, (2, 3, 9, 11)).astype(np.float32)
    V32 = ct.input_transform_m2_paper_order_f32(x, 1)
    V64 = ct.input_transform(x.astype(np.float64), 1, 2)
    assert V32.dtype == np.float32
    assert np.array_equal(V32.astype(np.float64), V64)


def test_paper_order_f32_rounding_is_the_two_pass_order():
    # Non-integer data: each output is ((a -+ b) -+ (c -+ d)) rounded in fp32 at
    # every step, rows first.  Recompute one element that way by hand.
    rng = np.random.default_rng(13)
    x = rng.standard_normal((1, 1, 4, 4)).astype(np.float32)
    V = ct.input_transform_m2_paper_order_f32(x, 0)
    d = x[0, 0]
    f = np.float32
    # t = (0, 0): rows pass row0 - row2, then column pass col0 - col2.
    r0 = [f(d[0, j]) - f(d[2, j]) for j in range(4)]
    assert V[0, 0, 0] == f(r0[0]) - f(r0[2])
    # t = (3, 1): rows pass row1 - row3, columns pass col1 + col2.
    r3 = [f(d[1, j]) - f(d[3, j]) for j in range(4)]
    assert V[3 * 4 + 1, 0, 0] == f(r3[1]) + f(r3[2])


@pytest.mark.parametrize("m,ratio", [(2, 2.25), (4, 4.0)])
def test_multiplication_reduction(m, ratio):
    # Direct: 9 m^2 multiplies per m x m output tile per (c, k); Winograd: (m+2)^2.
    a = m + 2
    assert (9 * m * m) / (a * a) == ratio
    N, C, H, W, K = 1, 3, 4 * m - 2 + 2, 4 * m, 2   # pad 1 -> Ho = H, exactly tiled
    Ho, Wo, th, tw, P = ct.geometry(N, H, W, 1, m)
    assert Ho % m == 0 and Wo % m == 0
    direct_flops = 2 * N * K * C * 9 * Ho * Wo
    gemm_flops = 2 * a * a * P * C * K
    assert direct_flops / gemm_flops == ratio


def test_stage_layouts_5x5():
    N, C, H, W, K, pad, m, r = 2, 3, 10, 9, 5, 2, 2, 5
    rng = np.random.default_rng(21)
    x = rng.standard_normal((N, C, H, W))
    g = rng.standard_normal((K, C, r, r))
    Ho, Wo, th, tw, P = ct.geometry(N, H, W, pad, m, r)
    assert (Ho, Wo) == (H, W)                     # pad 2 keeps the size of a 5x5 layer
    U = ct.filter_transform(g, m)
    V = ct.input_transform(x, pad, m, r)
    assert U.shape == (36, C, K) and V.shape == (36, C, P)
    _, G, BT = ct.matrices_f64(m, r)
    k, c, xi, nu = 4, 1, 3, 5
    assert np.isclose(U[xi * 6 + nu, c, k], (G @ g[k, c] @ G.T)[xi, nu], rtol=1e-15, atol=1e-15)
    n, ti, tj = 1, 3, 2
    p = (n * th + ti) * tw + tj
    xe = np.pad(x[n, c], ((pad, 20), (pad, 20)))
    d = xe[ti * m:ti * m + 6, tj * m:tj * m + 6]
    assert np.isclose(V[xi * 6 + nu, c, p], (BT @ d @ BT.T)[xi, nu], rtol=1e-14, atol=1e-14)
