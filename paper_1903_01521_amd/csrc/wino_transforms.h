// Device-side Cook-Toom transforms for F(2x2,3x3), F(4x4,3x3) and F(2x2,5x5).
//
// The matrices (Lavin's names; the paper writes X^T for B^T, W for G and Z^T
// for A^T, Eq. 1):
//
//   m = 2, alpha = 4, points {0, 1, -1, inf}; B^T is the matrix the paper prints
//   for the F(2x2,3x3) input transform (Sec. 2.1.1):
//     B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1]
//     G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1]
//     A^T = [1 1 1 0; 0 1 -1 -1]
//
//   m = 4, alpha = 6, points {0, 1, -1, 2, -2, inf}:
//     B^T = [4 0 -5 0 1 0; 0 -4 -4 1 1 0; 0 4 -4 -1 1 0;
//            0 -2 -1 2 1 0; 0 2 -1 -2 1 0; 0 4 0 -5 0 1]
//     G   = [1/4 0 0; -1/6 -1/6 -1/6; -1/6 1/6 -1/6;
//            1/24 1/12 1/6; 1/24 -1/12 1/6; 0 0 1]
//     A^T = [1 1 1 1 1 0; 0 1 -1 2 -2 0; 0 1 1 4 4 0; 0 1 -1 8 -8 1]
//
//   F(2x2,5x5), alpha = 6, the same points as m = 4 (so the same B^T):
//     G   = [1/4 0 0 0 0; -1/6 -1/6 -1/6 -1/6 -1/6; -1/6 1/6 -1/6 1/6 -1/6;
//            1/24 1/12 1/6 1/3 2/3; 1/24 -1/12 1/6 -1/3 2/3; 0 0 0 0 1]
//     A^T = [1 1 1 1 1 0; 0 1 -1 2 -2 1]
//
// All compute correlation: y[i] = sum_k g[k] d[i+k].  Every 2-D transform is
// the 1-D transform applied along rows (left factor), then along columns
// (right factor): B^T d B = ((B^T d)) then .B, and likewise A^T M A.  For m = 2
// this is the two-pass order the paper prints, so each value is exactly two
// levels of rounded fp32 add/sub in that order.
#pragma once

#include <hip/hip_runtime.h>

namespace wino {

template <int MT> struct Tile {
    static constexpr int A = MT + 2;   // region side, alpha
    static constexpr int T = A * A;    // transform-domain elements per region
};

// ---------------------------------------------------------------- 1-D B^T
__device__ __forceinline__ void bt_1d(const float (&a)[4], float (&r)[4]) {
    r[0] = a[0] - a[2];
    r[1] = a[1] + a[2];
    r[2] = a[2] - a[1];
    r[3] = a[1] - a[3];
}

__device__ __forceinline__ void bt_1d(const float (&a)[6], float (&r)[6]) {
    // rows of B^T for m = 4, grouped so that shared differences are formed once
    const float d31 = a[3] - a[1];
    const float d42 = a[4] - a[2];
    r[0] = __builtin_fmaf(4.0f, a[0] - a[2], a[4] - a[2]);     //  4a0 - 5a2 + a4
    r[1] = __builtin_fmaf(-4.0f, a[1] + a[2], a[3] + a[4]);    // -4a1 - 4a2 + a3 + a4
    r[2] = __builtin_fmaf(4.0f, a[1] - a[2], a[4] - a[3]);     //  4a1 - 4a2 - a3 + a4
    r[3] = __builtin_fmaf(2.0f, d31, d42);                     // -2a1 - a2 + 2a3 + a4
    r[4] = __builtin_fmaf(-2.0f, d31, d42);                    //  2a1 - a2 - 2a3 + a4
    r[5] = __builtin_fmaf(4.0f, a[1] - a[3], a[5] - a[3]);     //  4a1 - 5a3 + a5
}

// ---------------------------------------------------------------- 1-D A^T
__device__ __forceinline__ void at_1d(const float (&a)[4], float (&r)[2]) {
    r[0] = a[0] + a[1] + a[2];
    r[1] = a[1] - a[2] - a[3];
}

__device__ __forceinline__ void at_1d(const float (&a)[6], float (&r)[2]) {      // F(2,5)
    r[0] = (a[0] + (a[1] + a[2])) + (a[3] + a[4]);            // a0 + a1 + a2 + a3 + a4
    r[1] = __builtin_fmaf(2.0f, a[3] - a[4], a[1] - a[2]) + a[5];   // a1 - a2 + 2a3 - 2a4 + a5
}

__device__ __forceinline__ void at_1d(const float (&a)[6], float (&r)[4]) {
    const float s12 = a[1] + a[2], d12 = a[1] - a[2];
    const float s34 = a[3] + a[4], d34 = a[3] - a[4];
    r[0] = a[0] + s12 + s34;                                   // a0 + a1 + a2 + a3 + a4
    r[1] = __builtin_fmaf(2.0f, d34, d12);                     // a1 - a2 + 2a3 - 2a4
    r[2] = __builtin_fmaf(4.0f, s34, s12);                     // a1 + a2 + 4a3 + 4a4
    r[3] = __builtin_fmaf(8.0f, d34, d12) + a[5];              // a1 - a2 + 8a3 - 8a4 + a5
}

// ---------------------------------------------------------------- 2-D
// v[xi*A + nu] = (B^T d B)[xi][nu]
template <int MT>
__device__ __forceinline__ void input_tf(const float (&d)[MT + 2][MT + 2], float (&v)[(MT + 2) * (MT + 2)]) {
    constexpr int A = MT + 2;
    float s[A][A];
#pragma unroll
    for (int j = 0; j < A; ++j) {          // along rows: column j of B^T d
        float col[A], r[A];
#pragma unroll
        for (int i = 0; i < A; ++i) col[i] = d[i][j];
        bt_1d(col, r);
#pragma unroll
        for (int i = 0; i < A; ++i) s[i][j] = r[i];
    }
#pragma unroll
    for (int i = 0; i < A; ++i) {          // along columns: row i of (B^T d) B
        float r[A];
        bt_1d(s[i], r);
#pragma unroll
        for (int j = 0; j < A; ++j) v[i * A + j] = r[j];
    }
}

// o[i][j] = (A^T M A)[i][j], M[xi][nu] = mv[xi*A + nu]; A = MT + R - 1
template <int MT, int R = 3>
__device__ __forceinline__ void output_tf(const float (&mv)[(MT + R - 1) * (MT + R - 1)], float (&o)[MT][MT]) {
    constexpr int A = MT + R - 1;
    float s[MT][A];
#pragma unroll
    for (int j = 0; j < A; ++j) {          // along rows: column j of A^T M
        float col[A], r[MT];
#pragma unroll
        for (int i = 0; i < A; ++i) col[i] = mv[i * A + j];
        at_1d(col, r);
#pragma unroll
        for (int i = 0; i < MT; ++i) s[i][j] = r[i];
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {         // along columns: row i of (A^T M) A
        float r[MT];
        at_1d(s[i], r);
#pragma unroll
        for (int j = 0; j < MT; ++j) o[i][j] = r[j];
    }
}

// ---------------------------------------------------------------- row subsets
// A wave that owns only transform-domain rows X0 .. X0+RN-1 needs only those
// rows of B^T d B, and its share of A^T M A (the output transform is linear in
// M, so the shares of all row groups add up to the full result).

// v[(xi - X0)*A + nu] = (B^T d B)[xi][nu] for xi in [X0, X0+RN).  The first pass
// evaluates the full 1-D transform per column; unused rows are dead code.
template <int MT, int X0, int RN>
__device__ __forceinline__ void input_tf_rows(const float (&d)[MT + 2][MT + 2], float (&v)[RN * (MT + 2)]) {
    constexpr int A = MT + 2;
    float s[RN][A];
#pragma unroll
    for (int j = 0; j < A; ++j) {
        float col[A], r[A];
#pragma unroll
        for (int i = 0; i < A; ++i) col[i] = d[i][j];
        bt_1d(col, r);
#pragma unroll
        for (int i = 0; i < RN; ++i) s[i][j] = r[X0 + i];
    }
#pragma unroll
    for (int i = 0; i < RN; ++i) {
        float r[A];
        bt_1d(s[i], r);
#pragma unroll
        for (int j = 0; j < A; ++j) v[i * A + j] = r[j];
    }
}

// r[i] = sum over xi in [X0, X0+RN) of A^T[i][xi] * a[xi - X0]
template <int MT, int X0, int RN> struct AtRows;
template <> struct AtRows<2, 0, 4> {
    __device__ static void f(const float (&a)[4], float (&r)[2]) { at_1d(a, r); }
};
template <> struct AtRows<4, 0, 6> {
    __device__ static void f(const float (&a)[6], float (&r)[4]) { at_1d(a, r); }
};
template <> struct AtRows<2, 0, 2> {            // rows 0, 1 of A^T = [1 1 1 0; 0 1 -1 -1]
    __device__ static void f(const float (&a)[2], float (&r)[2]) {
        r[0] = a[0] + a[1];
        r[1] = a[1];
    }
};
template <> struct AtRows<2, 2, 2> {            // rows 2, 3
    __device__ static void f(const float (&a)[2], float (&r)[2]) {
        r[0] = a[0];
        r[1] = -a[0] - a[1];
    }
};
template <> struct AtRows<4, 0, 3> {            // rows 0, 1, 2 of the m = 4 A^T
    __device__ static void f(const float (&a)[3], float (&r)[4]) {
        const float s12 = a[1] + a[2], d12 = a[1] - a[2];
        r[0] = a[0] + s12;
        r[1] = d12;
        r[2] = s12;
        r[3] = d12;
    }
};
template <> struct AtRows<2, 0, 3> {            // rows 0, 1, 2 of the F(2,5) A^T (2 x 6)
    __device__ static void f(const float (&a)[3], float (&r)[2]) {
        r[0] = a[0] + (a[1] + a[2]);
        r[1] = a[1] - a[2];
    }
};
template <> struct AtRows<2, 3, 3> {            // rows 3, 4, 5 of the F(2,5) A^T
    __device__ static void f(const float (&a)[3], float (&r)[2]) {
        r[0] = a[0] + a[1];
        r[1] = __builtin_fmaf(2.0f, a[0] - a[1], a[2]);
    }
};
template <> struct AtRows<4, 3, 3> {            // rows 3, 4, 5
    __device__ static void f(const float (&a)[3], float (&r)[4]) {
        const float s34 = a[0] + a[1], d34 = a[0] - a[1];
        r[0] = s34;
        r[1] = 2.0f * d34;
        r[2] = 4.0f * s34;
        r[3] = __builtin_fmaf(8.0f, d34, a[2]);
    }
};

// o = A^T M' A where M' keeps rows [X0, X0+RN) of M (mv holds just those
// rows); A^T is m x (m + R - 1) (R = 5 only with m = 2).
template <int MT, int X0, int RN, int R = 3>
__device__ __forceinline__ void output_tf_rows(const float (&mv)[RN * (MT + R - 1)], float (&o)[MT][MT]) {
    constexpr int A = MT + R - 1;
    float s[MT][A];
#pragma unroll
    for (int j = 0; j < A; ++j) {
        float col[RN], r[MT];
#pragma unroll
        for (int i = 0; i < RN; ++i) col[i] = mv[i * A + j];
        AtRows<MT, X0, RN>::f(col, r);
#pragma unroll
        for (int i = 0; i < MT; ++i) s[i][j] = r[i];
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        float r[MT];
        at_1d(s[i], r);
#pragma unroll
        for (int j = 0; j < MT; ++j) o[i][j] = r[j];
    }
}

// ---------------------------------------------------------------- filter, fp64
// U = G g G^T evaluated in fp64 with an integer-scaled G (S*G has integer
// entries: S = 2 for F(2,3), S = 24 for F(4,3) and F(2,5)): the two
// small-integer products are exact or nearly so in fp64, the scale 1/S^2 is
// applied once as a multiplication (relative error <= 2^-52), and the result
// is rounded to fp32.  Integer-valued results (g a multiple of S^2) come out
// exact.
template <int MT, int R = 3> struct GScaled;
template <> struct GScaled<2> {
    static constexpr double INV_S2 = 1.0 / 4.0;
    __device__ static void rows(const double (&a)[3], double (&r)[4]) {
        r[0] = 2.0 * a[0];
        r[1] = a[0] + a[1] + a[2];
        r[2] = a[0] - a[1] + a[2];
        r[3] = 2.0 * a[2];
    }
};
template <> struct GScaled<4> {
    static constexpr double INV_S2 = 1.0 / 576.0;
    __device__ static void rows(const double (&a)[3], double (&r)[6]) {
        r[0] = 6.0 * a[0];
        r[1] = -4.0 * (a[0] + a[1] + a[2]);
        r[2] = -4.0 * (a[0] - a[1] + a[2]);
        r[3] = a[0] + 2.0 * a[1] + 4.0 * a[2];
        r[4] = a[0] - 2.0 * a[1] + 4.0 * a[2];
        r[5] = 24.0 * a[2];
    }
};
template <> struct GScaled<2, 5> {
    static constexpr double INV_S2 = 1.0 / 576.0;
    __device__ static void rows(const double (&a)[5], double (&r)[6]) {
        const double se = a[0] + a[2] + a[4], so = a[1] + a[3];
        r[0] = 6.0 * a[0];
        r[1] = -4.0 * (se + so);
        r[2] = -4.0 * (se - so);
        const double ev = a[0] + 4.0 * a[2] + 16.0 * a[4], od = 2.0 * a[1] + 8.0 * a[3];
        r[3] = ev + od;
        r[4] = ev - od;
        r[5] = 24.0 * a[4];
    }
};

// Positions T0 .. T0+3 of U = G g G^T (t = xi*A + nu), fp64 inside, each
// rounded once to fp32.  Only the rows of (S G) g that these positions need are
// live after unrolling; the rest is dead code.
template <int MT, int T0, int R = 3>
__device__ __forceinline__ float4 filter_tf4(const float (&g)[R][R]) {
    constexpr int A = MT + R - 1;
    double cs[R][A];                       // (S G) g, column c, every row
#pragma unroll
    for (int c = 0; c < R; ++c) {
        double col[R];
#pragma unroll
        for (int k = 0; k < R; ++k) col[k] = (double)g[k][c];
        GScaled<MT, R>::rows(col, cs[c]);
    }
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {          // ((S G) g) (S G)^T at row xi, column nu
        const int t = T0 + e, xi = t / A, nu = t % A;
        double row[R];
#pragma unroll
        for (int c = 0; c < R; ++c) row[c] = cs[c][xi];
        double r[A];
        GScaled<MT, R>::rows(row, r);
        o[e] = (float)(r[nu] * GScaled<MT, R>::INV_S2);
    }
    return make_float4(o[0], o[1], o[2], o[3]);
}

}  // namespace wino

namespace wino {

// ---------------------------------------------------------------- 1-D, alpha = 8
// F(1xm, 1xr, 1x8) for 1xr / rx1 filters, (m, r) = (6, 3), (4, 5), (2, 7), with
// the points {0, 1, -1, 2, -2, 1/2, -1/2, inf}.  B^T is the same for the three
// (it depends only on the points); every entry of B^T and A^T is a dyadic
// rational, exact in fp32:
//   B^T = [-1   0  21/4    0  -21/4    0   1  0;
//           0   1     1 -17/4 -17/4    1   1  0;
//           0  -1     1  17/4 -17/4   -1   1  0;
//           0 1/2   1/4  -5/2  -5/4    2   1  0;
//           0 -1/2  1/4   5/2  -5/4   -2   1  0;
//           0   2     4  -5/2    -5  1/2   1  0;
//           0  -2     4   5/2    -5 -1/2   1  0;
//           0  -1     0  21/4     0 -21/4  0  1]
//   A^T[i] = [i == 0, 1, (-1)^i, 2^i, (-2)^i, 2^-i, (-2)^-i, i == m-1]
//   G[j][k] = p_j^k / prod_{l != j} (p_j - p_l) (finite points), G[7] = e_{r-1};
//   90 G is an integer matrix: rows -90 e_0, -20 (1)^k, -20 (-1)^k, 2^k,
//   (-2)^k, 2^(6-k), (-1)^k 2^(6-k), 90 e_{r-1}.
__device__ __forceinline__ void bt8(const float (&d)[8], float (&v)[8]) {
    const float d24 = d[2] - d[4], d35 = d[3] - d[5];
    v[0] = __builtin_fmaf(5.25f, d24, d[6] - d[0]);
    v[7] = __builtin_fmaf(5.25f, d35, d[7] - d[1]);
    const float s15 = d[1] + d[5], s26 = d[2] + d[6];
    v[1] = __builtin_fmaf(-4.25f, d[3] + d[4], s15 + s26);
    v[2] = __builtin_fmaf(4.25f, d[3] - d[4], s26 - s15);
    const float o3 = __builtin_fmaf(0.5f, d[1], __builtin_fmaf(-2.5f, d[3], 2.0f * d[5]));
    const float e3 = __builtin_fmaf(0.25f, d[2], __builtin_fmaf(-1.25f, d[4], d[6]));
    v[3] = e3 + o3;
    v[4] = e3 - o3;
    const float o5 = __builtin_fmaf(2.0f, d[1], __builtin_fmaf(-2.5f, d[3], 0.5f * d[5]));
    const float e5 = __builtin_fmaf(4.0f, d[2], __builtin_fmaf(-5.0f, d[4], d[6]));
    v[5] = e5 + o5;
    v[6] = e5 - o5;
}

template <int M>
__device__ __forceinline__ void at8(const float (&a)[8], float (&o)[M]) {
    const float s1 = a[1] + a[2], d1 = a[1] - a[2];
    const float s2 = a[3] + a[4], d2 = a[3] - a[4];
    const float s3 = a[5] + a[6], d3 = a[5] - a[6];
#pragma unroll
    for (int i = 0; i < M; ++i) {
        const float p = (float)(1 << i), q = 1.0f / (float)(1 << i);     // 2^i, 2^-i (exact)
        float v = (i & 1) ? __builtin_fmaf(p, d2, __builtin_fmaf(q, d3, d1))
                          : __builtin_fmaf(p, s2, __builtin_fmaf(q, s3, s1));
        if (i == 0) v += a[0];
        if (i == M - 1) v += a[7];
        o[i] = v;
    }
}

// U = G g in fp64 with the integer matrix 90 G, scaled once by 1/90, rounded
// once to fp32.
template <int R>
__device__ __forceinline__ void filter_tf8(const float (&g)[R], float (&u)[8]) {
    double s = 0, a = 0, p2 = 0, m2 = 0, h = 0, mh = 0;
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const double v = (double)g[k], sg = (k & 1) ? -1.0 : 1.0;
        s += v;
        a += sg * v;
        p2 += (double)(1 << k) * v;
        m2 += sg * (double)(1 << k) * v;
        h += (double)(1 << (6 - k)) * v;
        mh += sg * (double)(1 << (6 - k)) * v;
    }
    const double r[8] = {-90.0 * g[0], -20.0 * s, -20.0 * a, p2, m2, h, mh, 90.0 * g[R - 1]};
#pragma unroll
    for (int t = 0; t < 8; ++t) u[t] = (float)(r[t] * (1.0 / 90.0));
}

}  // namespace wino
