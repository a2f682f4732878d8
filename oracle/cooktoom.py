"""Cook-Toom / Winograd minimal filtering, exactly and in fp64 (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU baseline may import this
module; the HIP path never does, and its own transform constants are written
independently of anything here.

Contents, each in the paper's notation where it has one (Sec. 2):

* :func:`cook_toom` -- the exact rational matrices of F(m x m, r x r): the output
  (inverse) transform A^T (the paper's Z^T), the filter transform G (its W) and
  the input transform B^T (its X^T), derived from interpolation points.  Only
  the F(2x2,3x3) input matrix is printed in the paper (Sec. 2.1.1); the rest
  follows from the construction below, and the m=2 signs are chosen so that
  B^T equals the printed matrix.  r = 3 is the method's filter size; r = 5 is
  F(2x2,5x5) for the 5x5 layers of the paper's Table 2 (same region size, 6x6,
  as F(4x4,3x3)).
* :func:`winograd_conv_exact` -- Eq. 1 evaluated over the rationals, region by
  region, in the loop order of Listing 1 (per output channel, per output region,
  sum over the input channels in the transform domain, one inverse transform
  per region).  On integer inputs this must equal the direct definition exactly.
* fp64 references of each stage of the three-step decomposition of Sec. 2
  (input transform scattering into the per-position 'A' matrices, the
  per-position GEMMs with the pre-transformed weights 'B', and the output
  transform gathering from 'C'), plus the offline weight transform.
* :func:`input_transform_m2_paper_order_f32` -- the F(2x2,3x3) input transform in
  fp32 with the exact add/sub sequence the paper prints for it (Sec. 2.1.1): a
  pass combining rows, then the same pass combining columns.

Transform-domain index: t = xi * alpha + nu for the (xi, nu) element of an
alpha x alpha region, alpha = m + r - 1 (m + 2 for 3x3 filters), T = alpha^2.
Tile index p = (n*th + ti)*tw + tj with th = ceil(Ho/m), tw = ceil(Wo/m).  Tile (ti, tj) produces output rows
ti*m .. ti*m+m-1 and reads the input region starting at (ti*m - pad, tj*m - pad);
values outside the input (padding and the ragged overhang) are zero, and outputs
beyond Ho x Wo are discarded.
"""
from __future__ import annotations

from fractions import Fraction as Q
from functools import lru_cache
from math import prod

import numpy as np

R_FILTER = 3  # the method's filter size for this path (3x3 layers)
SUPPORTED = ((2, 3), (4, 3), (2, 5))   # (m, r): F(2x2,3x3), F(4x4,3x3), F(2x2,5x5)


# ----------------------------------------------------------------------------
# Exact matrices
# ----------------------------------------------------------------------------

def interpolation_points(m: int, r: int = R_FILTER) -> list[int]:
    """Finite interpolation points of F(m, r); the point at infinity is implied.

    The paper names the Cook-Toom class but not its points.  Reading taken: the
    smallest-magnitude integer points, alpha - 1 = m + r - 2 of them: {0, 1, -1}
    for F(2,3) and {0, 1, -1, 2, -2} for F(4,3) and F(2,5).  Any distinct points
    give an exact algorithm; the choice only changes fp32 rounding.
    """
    if (m, r) not in SUPPORTED:
        raise ValueError("(m, r) must be one of %s" % (SUPPORTED,))
    return [0, 1, -1, 2, -2][:m + r - 2]


def _solve_consistent(rows: list[list[Q]], rhs: list[Q]) -> list[Q]:
    """Exact Gauss-Jordan solve of an over-determined, consistent system with a
    unique solution.  Raises if inconsistent or rank-deficient."""
    n = len(rows[0])
    aug = [list(r) + [b] for r, b in zip(rows, rhs)]
    piv_row = 0
    pivots = []
    for col in range(n):
        sel = next((r for r in range(piv_row, len(aug)) if aug[r][col] != 0), None)
        if sel is None:
            raise ArithmeticError("rank-deficient system")
        aug[piv_row], aug[sel] = aug[sel], aug[piv_row]
        pv = aug[piv_row][col]
        aug[piv_row] = [v / pv for v in aug[piv_row]]
        for r in range(len(aug)):
            if r != piv_row and aug[r][col] != 0:
                f = aug[r][col]
                aug[r] = [a - f * b for a, b in zip(aug[r], aug[piv_row])]
        pivots.append(col)
        piv_row += 1
    for r in range(piv_row, len(aug)):
        if aug[r][n] != 0:
            raise ArithmeticError("inconsistent system")
    return [aug[i][n] for i in range(n)]


@lru_cache(maxsize=None)
def _raw_cook_toom(m: int, r: int = R_FILTER):
    a = m + r - 1
    pts = [Q(p) for p in interpolation_points(m, r)]
    nf = a - 1  # finite points; the last row/column is the point at infinity
    # Output transform: evaluate the length-m output polynomial's basis at each
    # point; the infinity column picks the leading coefficient.
    AT = [[(pts[j] ** i if j < nf else Q(int(i == m - 1))) for j in range(a)]
          for i in range(m)]
    # Filter transform: Lagrange-weighted evaluation of the filter polynomial at
    # each finite point; the infinity row picks the filter's leading tap.
    G = []
    for j in range(nf):
        den = prod((pts[j] - pts[l] for l in range(nf) if l != j), start=Q(1))
        G.append([pts[j] ** k / den for k in range(r)])
    G.append([Q(int(k == r - 1)) for k in range(r)])
    # Input transform: the unique B^T with sum_j AT[i][j] G[j][k] BT[j][a'] equal
    # to [a' == i + k] for all i < m, k < r, a' < alpha, i.e. the 1-D algorithm
    # reproduces y[i] = sum_k g[k] d[i + k] (correlation) for every g and d.
    E = [[AT[i][j] * G[j][k] for j in range(a)] for i in range(m) for k in range(r)]
    cols = []
    for ap in range(a):
        rhs = [Q(int(ap == i + k)) for i in range(m) for k in range(r)]
        cols.append(_solve_consistent(E, rhs))
    BT = [[cols[ap][j] for ap in range(a)] for j in range(a)]
    return AT, G, BT


def cook_toom(m: int, r: int = R_FILTER):
    """Exact (A^T, G, B^T) of F(m x m, r x r) as lists of Fractions.

    Sign normalisation: scaling row j of G by s and row j of B^T by 1/s (or
    column j of A^T by s and row j of B^T by 1/s) leaves the algorithm exact.
    For F(2,3) the paper prints B^T; the raw derivation differs from it by the
    sign of rows 0 and 3, so row 0 is flipped through G and row 3 (the infinity
    row) through A^T.  For F(4,3) and F(2,5) nothing is printed and the raw
    derivation is kept (their B^T coincide: same points).
    """
    AT, G, BT = _raw_cook_toom(m, r)
    AT = [list(row) for row in AT]
    G = [list(row) for row in G]
    BT = [list(row) for row in BT]
    if (m, r) == (2, 3):
        G[0] = [-v for v in G[0]]
        BT[0] = [-v for v in BT[0]]
        for i in range(len(AT)):
            AT[i][3] = -AT[i][3]
        BT[3] = [-v for v in BT[3]]
    return AT, G, BT


def matrices_f64(m: int, r: int = R_FILTER):
    """(A^T, G, B^T) as fp64 numpy arrays (G's thirds are rounded to fp64)."""
    AT, G, BT = cook_toom(m, r)
    f = lambda M: np.array([[float(v) for v in row] for row in M], dtype=np.float64)
    return f(AT), f(G), f(BT)


# ----------------------------------------------------------------------------
# Geometry
# ----------------------------------------------------------------------------

def geometry(N: int, H: int, W: int, pad: int, m: int, r: int = R_FILTER):
    """(Ho, Wo, th, tw, P) of an r x r stride-1 layer tiled into m x m output regions."""
    Ho, Wo = H + 2 * pad - (r - 1), W + 2 * pad - (r - 1)
    th, tw = -(-Ho // m), -(-Wo // m)
    return Ho, Wo, th, tw, N * th * tw


# ----------------------------------------------------------------------------
# Eq. 1 / Listing 1 over the rationals
# ----------------------------------------------------------------------------

def _mm(A, B):
    return [[sum((A[i][l] * B[l][j] for l in range(len(B))), Q(0))
             for j in range(len(B[0]))] for i in range(len(A))]


def _tr(A):
    return [list(r) for r in zip(*A)]


def winograd_conv_exact(x, g, pad: int, m: int):
    """Region-wise multi-channel Winograd convolution over the rationals.

    x: integer/rational array [N][C][H][W]; g: [K][C][r][r] (r = 3, or 5 with
    m = 2).  Returns a nested list [N][K][Ho][Wo] of Fractions.  Pure Python:
    tiny inputs only.
    """
    x = np.asarray(x, dtype=object)
    g = np.asarray(g, dtype=object)
    N, C, H, W = x.shape
    K, r = g.shape[0], g.shape[2]
    AT, G, BT = cook_toom(m, r)
    A, GT, B = _tr(AT), _tr(G), _tr(BT)
    a = m + r - 1
    Ho, Wo, th, tw, _ = geometry(N, H, W, pad, m, r)

    def pix(n, c, u, v):
        if 0 <= u < H and 0 <= v < W:
            return Q(x[n, c, u, v])
        return Q(0)

    # Offline weight transform W w W^T per (output channel, input channel).
    U = [[_mm(_mm(G, [[Q(g[k, c, u, v]) for v in range(r)] for u in range(r)]), GT)
          for c in range(C)] for k in range(K)]
    # Input transform X^T x X of every (image, channel, region).
    V = {}
    for n in range(N):
        for c in range(C):
            for ti in range(th):
                for tj in range(tw):
                    d = [[pix(n, c, ti * m - pad + u, tj * m - pad + v) for v in range(a)]
                         for u in range(a)]
                    V[n, c, ti, tj] = _mm(_mm(BT, d), B)
    y = [[[[Q(0)] * Wo for _ in range(Ho)] for _ in range(K)] for _ in range(N)]
    for k in range(K):                               # each output channel
        for n in range(N):
            for ti in range(th):
                for tj in range(tw):                 # each output region
                    acc = [[Q(0)] * a for _ in range(a)]
                    for c in range(C):               # sum over input channels
                        Uc, Vc = U[k][c], V[n, c, ti, tj]
                        for u in range(a):
                            for v in range(a):
                                acc[u][v] += Uc[u][v] * Vc[u][v]   # Hadamard product
                    out = _mm(_mm(AT, acc), A)       # one inverse transform per region
                    for i in range(m):
                        for j in range(m):
                            oi, oj = ti * m + i, tj * m + j
                            if oi < Ho and oj < Wo:
                                y[n][k][oi][oj] = out[i][j]
    return y


# ----------------------------------------------------------------------------
# fp64 stage references (logical layouts U[T][C][K], V[T][C][P], M[T][K][P])
# ----------------------------------------------------------------------------

def filter_transform(g: np.ndarray, m: int) -> np.ndarray:
    """U[t][c][k] = (G g[k,c] G^T)[xi, nu], t = xi*alpha + nu, in fp64 (r from g)."""
    g = np.asarray(g, dtype=np.float64)
    K, C, r = g.shape[:3]
    _, G, _ = matrices_f64(m, r)
    a = m + r - 1
    U = np.einsum("ar,kcrs,bs->abck", G, g, G)
    return np.ascontiguousarray(U.reshape(a * a, C, K))


def extract_regions(x: np.ndarray, pad: int, m: int, r: int = R_FILTER) -> np.ndarray:
    """d[n, c, ti, tj, u, v] = zero-extended x[n, c, ti*m - pad + u, tj*m - pad + v]."""
    x = np.asarray(x)
    N, C, H, W = x.shape
    a = m + r - 1
    _, _, th, tw, _ = geometry(N, H, W, pad, m, r)
    Hx, Wx = th * m + r - 1, tw * m + r - 1
    xe = np.zeros((N, C, Hx, Wx), dtype=x.dtype)
    h1, w1 = min(H, Hx - pad), min(W, Wx - pad)
    xe[:, :, pad:pad + h1, pad:pad + w1] = x[:, :, :h1, :w1]
    d = np.empty((N, C, th, tw, a, a), dtype=x.dtype)
    for ti in range(th):
        for tj in range(tw):
            d[:, :, ti, tj] = xe[:, :, ti * m:ti * m + a, tj * m:tj * m + a]
    return d


def input_transform(x: np.ndarray, pad: int, m: int, r: int = R_FILTER) -> np.ndarray:
    """V[t][c][p] = (B^T d_{n,c,ti,tj} B)[xi, nu] in fp64, p = (n*th+ti)*tw+tj."""
    _, _, BT = matrices_f64(m, r)
    d = extract_regions(np.asarray(x, dtype=np.float64), pad, m, r)
    N, C, th, tw, a, _ = d.shape
    Vr = np.einsum("au,nctjuv,bv->abcntj", BT, d, BT)
    return np.ascontiguousarray(Vr.reshape(a * a, C, N * th * tw))


def batched_gemm(U: np.ndarray, V: np.ndarray) -> np.ndarray:
    """M[t] = U[t]^T V[t]: for each of the T positions, [K x C] . [C x P]."""
    return np.matmul(np.transpose(U, (0, 2, 1)), V)


def output_transform(M: np.ndarray, N: int, Ho: int, Wo: int, m: int, r: int = R_FILTER) -> np.ndarray:
    """y[n,k,ti*m+i,tj*m+j] = (A^T M_{k,p} A)[i, j], cropped to Ho x Wo, in fp64."""
    AT, _, _ = matrices_f64(m, r)
    T, K, P = M.shape
    a = m + r - 1
    th, tw = -(-Ho // m), -(-Wo // m)
    Mr = np.asarray(M, dtype=np.float64).reshape(a, a, K, N, th, tw)
    # labels: t = ti, w = tj; result axes n, k, ti, i, tj, j -> rows ti*m+i, cols tj*m+j
    Y = np.einsum("iu,uvkntw,jv->nktiwj", AT, Mr, AT)
    y = Y.reshape(N, K, th * m, tw * m)
    return np.ascontiguousarray(y[:, :, :Ho, :Wo])


def winograd_conv_f64(x: np.ndarray, g: np.ndarray, pad: int, m: int) -> np.ndarray:
    """The three stages composed in fp64 (weights transformed first, offline)."""
    N, C, H, W = np.asarray(x).shape
    r = np.asarray(g).shape[2]
    Ho, Wo, _, _, _ = geometry(N, H, W, pad, m, r)
    U = filter_transform(g, m)
    V = input_transform(x, pad, m, r)
    return output_transform(batched_gemm(U, V), N, Ho, Wo, m, r)


def input_transform_m2_paper_order_f32(x: np.ndarray, pad: int) -> np.ndarray:
    """F(2x2,3x3) input transform in fp32 with the paper's printed add/sub order.

    Sec. 2.1.1 gives B^T x as four row operations (row0 - row2, row1 + row2,
    row2 - row1, row1 - row3) and obtains B^T x B by applying the same four
    operations to the columns of that result.  Every coefficient is +-1, so each
    output is two levels of correctly rounded fp32 add/sub in this order.
    Returns V[t][c][p] fp32.
    """
    d = extract_regions(np.asarray(x, dtype=np.float32), pad, 2)
    N, C, th, tw, a, _ = d.shape
    r = [d[..., i, :] for i in range(4)]           # rows of each region
    s = [r[0] - r[2], r[1] + r[2], r[2] - r[1], r[1] - r[3]]
    s = np.stack(s, axis=-2)                       # (B^T d), rows 0..3
    c = [s[..., :, j] for j in range(4)]           # its columns
    v = [c[0] - c[2], c[1] + c[2], c[2] - c[1], c[1] - c[3]]
    V = np.stack(v, axis=-1)                       # (B^T d) B
    assert V.dtype == np.float32
    V = np.transpose(V, (4, 5, 1, 0, 2, 3))        # xi, nu, c, n, ti, tj
    return np.ascontiguousarray(V.reshape(16, C, N * th * tw))


# ----------------------------------------------------------------------------
# 1-D layers (1 x r and r x 1 filters): F(1 x m, 1 x r, 1 x 8)
# ----------------------------------------------------------------------------
# The paper applies variants of the method to 1-D layers as well (1xN and Nx1
# filters, Table 2's 1x7 and 7x1 Inception-v3 layers) and names F(1x6,1x3,1x8),
# F(1x4,1x5,1x8) and F(1x2,1x7,1x8).  A 1-D layer is Eq. 1 with regions of one
# row (or column) of alpha = 8 inputs producing m outputs along that axis.

SUPPORTED_1D = ((6, 3), (4, 5), (2, 7))


def interpolation_points_1d(m: int, r: int) -> list[Q]:
    """The seven finite points of the alpha = 8 variants; infinity is implied.

    The paper gives none.  Reading taken: {0, 1, -1, 2, -2, 1/2, -1/2}, the
    usual choice once the small integers run out (powers of two keep every
    entry of A^T and B^T a dyadic rational, exact in fp32).
    """
    if (m, r) not in SUPPORTED_1D:
        raise ValueError("(m, r) must be one of %s" % (SUPPORTED_1D,))
    return [Q(0), Q(1), Q(-1), Q(2), Q(-2), Q(1, 2), Q(-1, 2)]


@lru_cache(maxsize=None)
def cook_toom_1d(m: int, r: int):
    """Exact (A^T, G, B^T) of F(1 x m, 1 x r, 1 x 8): m x 8, 8 x r, 8 x 8.

    Same construction as the 2-D matrices (A^T from the points, G with the
    Lagrange denominators, B^T the unique exact solution of the bilinear
    identity); no sign normalisation (nothing is printed for these)."""
    pts = interpolation_points_1d(m, r)       # validates (m, r)
    a = m + r - 1
    nf = a - 1
    AT = [[(pts[j] ** i if j < nf else Q(int(i == m - 1))) for j in range(a)] for i in range(m)]
    G = []
    for j in range(nf):
        den = prod((pts[j] - pts[l] for l in range(nf) if l != j), start=Q(1))
        G.append([pts[j] ** k / den for k in range(r)])
    G.append([Q(int(k == r - 1)) for k in range(r)])
    E = [[AT[i][j] * G[j][k] for j in range(a)] for i in range(m) for k in range(r)]
    cols = [_solve_consistent(E, [Q(int(ap == i + k)) for i in range(m) for k in range(r)]) for ap in range(a)]
    BT = [[cols[ap][j] for ap in range(a)] for j in range(a)]
    return AT, G, BT


def matrices_1d_f64(m: int, r: int):
    AT, G, BT = cook_toom_1d(m, r)
    f = lambda M: np.array([[float(v) for v in row] for row in M], dtype=np.float64)
    return f(AT), f(G), f(BT)


def geometry_1d(N: int, H: int, W: int, pad: int, m: int, r: int, axis: str):
    """(Ho, Wo, th, tw, P) of a 1 x r (axis 'w') or r x 1 (axis 'h') layer.  The
    padding applies along the filter's axis only (the other extent is 1);
    tiles are 1 x m (axis 'w') or m x 1 (axis 'h')."""
    if axis == "w":
        Ho, Wo = H, W + 2 * pad - (r - 1)
        th, tw = Ho, -(-Wo // m)
    elif axis == "h":
        Ho, Wo = H + 2 * pad - (r - 1), W
        th, tw = -(-Ho // m), Wo
    else:
        raise ValueError("axis must be 'w' or 'h'")
    return Ho, Wo, th, tw, N * th * tw


def _as_1d(x, g, axis):
    """Move the filtered axis last: x [N, C, L_other, L], g [K, C, r]."""
    x = np.asarray(x)
    g = np.asarray(g)
    if axis == "h":
        x = np.swapaxes(x, 2, 3)
    return x, g.reshape(g.shape[0], g.shape[1], -1)


def conv1d_exact(x, g, pad: int, m: int, axis: str):
    """Eq. 1 / Listing 1 for a 1-D layer over the rationals: each region of 8
    inputs along the axis, per channel, to the transform domain; Hadamard
    products with G g summed over channels; one inverse transform per region.
    g: [K, C, 1, r] (axis 'w') or [K, C, r, 1] (axis 'h').  Tiny inputs only."""
    r = max(np.asarray(g).shape[2:])
    AT, G, BT = cook_toom_1d(m, r)
    xs, gs = _as_1d(np.asarray(x, dtype=object), np.asarray(g, dtype=object), axis)
    N, C, Lo, L = xs.shape
    K = gs.shape[0]
    Lout = L + 2 * pad - (r - 1)
    nt = -(-Lout // m)
    U = [[[sum((G[t][k] * Q(gs[kk, c, k]) for k in range(r)), Q(0)) for t in range(8)]
          for c in range(C)] for kk in range(K)]
    y = np.empty((N, K, Lo, Lout), dtype=object)
    for n in range(N):
        for row in range(Lo):
            for tj in range(nt):
                V = []
                for c in range(C):
                    d = [Q(xs[n, c, row, tj * m - pad + u]) if 0 <= tj * m - pad + u < L else Q(0)
                         for u in range(8)]
                    V.append([sum((BT[t][u] * d[u] for u in range(8)), Q(0)) for t in range(8)])
                for kk in range(K):
                    acc = [sum((U[kk][c][t] * V[c][t] for c in range(C)), Q(0)) for t in range(8)]
                    for i in range(m):
                        j = tj * m + i
                        if j < Lout:
                            y[n, kk, row, j] = sum((AT[i][t] * acc[t] for t in range(8)), Q(0))
    return np.swapaxes(y, 2, 3) if axis == "h" else y


def filter_transform_1d(g: np.ndarray, m: int) -> np.ndarray:
    """U[t][c][k] = (G g[k,c])[t] in fp64; g [K, C, 1, r] or [K, C, r, 1]."""
    g = np.asarray(g, dtype=np.float64)
    K, C = g.shape[:2]
    g = g.reshape(K, C, -1)
    _, G, _ = matrices_1d_f64(m, g.shape[2])
    return np.ascontiguousarray(np.einsum("tr,kcr->tck", G, g))


def input_transform_1d(x: np.ndarray, pad: int, m: int, r: int, axis: str) -> np.ndarray:
    """V[t][c][p] = (B^T d_{n,c,tile})[t] in fp64, p = (n*th + ti)*tw + tj."""
    _, _, BT = matrices_1d_f64(m, r)
    x = np.asarray(x, dtype=np.float64)
    N, C, H, W = x.shape
    Ho, Wo, th, tw, P = geometry_1d(N, H, W, pad, m, r, axis)
    xs = np.swapaxes(x, 2, 3) if axis == "h" else x        # filtered axis last
    Lo, L = xs.shape[2], xs.shape[3]
    nt = tw if axis == "w" else th
    ext = np.zeros((N, C, Lo, nt * m + 7))
    n_in = min(L, nt * m + 7 - pad)
    ext[:, :, :, pad:pad + n_in] = xs[:, :, :, :n_in]
    d = np.stack([ext[:, :, :, j * m:j * m + 8] for j in range(nt)], axis=3)   # n, c, row, tile, u
    v = np.einsum("tu,ncrju->tcnrj", BT, d)              # t, c, n, row(other axis), tile
    if axis == "h":                                      # tiles run along H: p = (n*th + tile)*tw + col
        v = np.swapaxes(v, 3, 4)
    return np.ascontiguousarray(v.reshape(8, C, P))


def output_transform_1d(M: np.ndarray, N: int, Ho: int, Wo: int, m: int, r: int, axis: str) -> np.ndarray:
    """y = A^T M_{k,p} along the axis, cropped to Ho x Wo, in fp64."""
    AT, _, _ = matrices_1d_f64(m, r)
    T, K, P = M.shape
    if axis == "w":
        th, tw = Ho, -(-Wo // m)
        Mr = np.asarray(M, dtype=np.float64).reshape(8, K, N, th, tw)
        Y = np.einsum("it,tknaj->nkaji", AT, Mr).reshape(N, K, th, tw * m)
        return np.ascontiguousarray(Y[:, :, :, :Wo])
    th, tw = -(-Ho // m), Wo
    Mr = np.asarray(M, dtype=np.float64).reshape(8, K, N, th, tw)
    Y = np.einsum("it,tknjb->nkjib", AT, Mr).reshape(N, K, th * m, tw)
    return np.ascontiguousarray(Y[:, :, :Ho, :])


def winograd_conv1d_f64(x: np.ndarray, g: np.ndarray, pad: int, m: int, axis: str) -> np.ndarray:
    N, C, H, W = np.asarray(x).shape
    r = max(np.asarray(g).shape[2:])
    Ho, Wo, _, _, _ = geometry_1d(N, H, W, pad, m, r, axis)
    U = filter_transform_1d(g, m)
    V = input_transform_1d(x, pad, m, r, axis)
    return output_transform_1d(batched_gemm(U, V), N, Ho, Wo, m, r, axis)


# ----------------------------------------------------------------------------
# 16-bit transform-domain operands (fp16 / bf16 GEMM with fp32 accumulation)
# ----------------------------------------------------------------------------
# A reduced-precision variant: U and V are rounded to a 16-bit format before
# the T per-position GEMMs, which accumulate in higher precision; the output
# transform is unchanged.  The reference below rounds the exact (fp64) U and V
# once, to nearest with ties to even, and does everything else in fp64: it is
# the definition the 16-bit GEMM path approximates up to fp32 accumulation and
# the fp32 rounding of its transforms.

def round_fp16(a: np.ndarray) -> np.ndarray:
    """Nearest IEEE binary16 value (ties to even; overflow to inf), as fp64."""
    return np.asarray(a, dtype=np.float64).astype(np.float16).astype(np.float64)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8-bit significand; ties to even), as fp64.

    bfloat16 is the upper half of an IEEE binary32: round the fp64 value to the
    nearest binary32 first only where that cannot change the bf16 result, i.e.
    do the rounding in integer arithmetic on the fp64 bits directly."""
    a = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(a)                      # a = m * 2^e, 0.5 <= |m| < 1
    scaled = np.ldexp(m, 8)                 # 8 significant bits above the point
    r = np.round(scaled)                    # numpy rounds half to even
    out = np.ldexp(r, e - 8)
    return np.where(a == 0, 0.0, out)


def reduced_precision_conv_f64(x: np.ndarray, g: np.ndarray, pad: int, m: int, prec: str) -> np.ndarray:
    """Output of the method when U and V are rounded to ``prec`` ('fp16' or
    'bf16') and everything else is exact (fp64)."""
    rnd = {"fp16": round_fp16, "bf16": round_bf16}[prec]
    N, C, H, W = np.asarray(x).shape
    Ho, Wo, _, _, _ = geometry(N, H, W, pad, m)
    U = rnd(filter_transform(g, m))
    V = rnd(input_transform(x, pad, m))
    return output_transform(batched_gemm(U, V), N, Ho, Wo, m)
