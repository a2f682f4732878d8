/*
 * Oracle (test infrastructure only): plain fp64 direct 3x3 stride-1 convolution.
 *
 * Only tests, the smoke check and the CPU-baseline leg of the benchmark may load
 * this library.  The product path never calls it, and it shares no code, header,
 * table or constant with the HIP kernels.
 *
 * What it computes.  Eq. 1 of the paper writes one layer as a sum over the C input
 * channels of per-channel filter/region products, taken region by region over the
 * output (Sec. 2, the text around Eq. 1 and Listing 1).  Over the rationals that
 * sum is exactly the direct multi-channel correlation, so the oracle is that
 * definition written out:
 *
 *   y[n,k,i,j] = sum_{c<C} sum_{r<3} sum_{s<3} xt[n,c,i+r-pad,j+s-pad] * g[k,c,r,s]
 *
 * with xt = x inside [0,H)x[0,W) and 0 outside (symmetric zero padding), for
 * 0 <= i < Ho = H+2pad-2, 0 <= j < Wo = W+2pad-2.  The channel sum runs over
 * c = 0..C-1 (the garbled upper bound of Eq. 1 is read as Listing 1's c < C).
 * No kernel flip: correlation, the convention of CNN frameworks.
 *
 * Seven plain loops (n, k, c, r, s, i, j); OpenMP over (n, k) only; no blocking,
 * no intrinsics, no BLAS.  Build with -O2 -ffp-contract=off, no fast-math, so every
 * product and sum is one correctly rounded fp64 operation in loop order.
 *
 * absval != 0 evaluates the same loops on |x| and |g|, giving the elementwise
 * magnitude bound (|x| * |g|)[n,k,i,j] used to scale rounding errors.
 */
#include <stddef.h>
#include <math.h>

int oracle_conv2d_f64(const double* x, const double* g, double* y,
                      int N, int C, int H, int W, int K, int pad, int absval)
{
    if (!x || !g || !y || N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || pad < 0)
        return -1;
    const long Ho = (long)H + 2L * pad - 2;
    const long Wo = (long)W + 2L * pad - 2;
    if (Ho < 1 || Wo < 1)
        return -1;

    long nk;
#pragma omp parallel for schedule(dynamic, 1)
    for (nk = 0; nk < (long)N * K; ++nk) {
        const long n = nk / K;
        const long k = nk % K;
        double* yo = y + ((n * K + k) * Ho) * Wo;
        for (long p = 0; p < Ho * Wo; ++p)
            yo[p] = 0.0;
        for (long c = 0; c < C; ++c) {
            const double* xi = x + ((n * C + c) * (long)H) * W;
            const double* gk = g + ((k * C + c) * 3L) * 3L;
            for (long r = 0; r < 3; ++r) {
                for (long s = 0; s < 3; ++s) {
                    double w = gk[r * 3 + s];
                    if (absval) w = fabs(w);
                    for (long i = 0; i < Ho; ++i) {
                        const long u = i + r - pad;
                        if (u < 0 || u >= H) continue;       /* zero padding: row outside */
                        for (long j = 0; j < Wo; ++j) {
                            const long v = j + s - pad;
                            if (v < 0 || v >= W) continue;   /* zero padding: column outside */
                            double a = xi[u * W + v];
                            if (absval) a = fabs(a);
                            yo[i * Wo + j] += a * w;
                        }
                    }
                }
            }
        }
    }
    return 0;
}

/*
 * The same definition for an R x S filter (the paper's layers also have 5x5
 * filters, Table 2): g is [K][C][R][S],
 *
 *   y[n,k,i,j] = sum_{c<C} sum_{r<R} sum_{s<S} xt[n,c,i+r-pad,j+s-pad] * g[k,c,r,s]
 *
 * for 0 <= i < Ho = H+2pad-(R-1), 0 <= j < Wo = W+2pad-(S-1).  Same loops, same
 * rules; kept apart from the 3x3 function above so that function stays exactly
 * as pinned.
 */
int oracle_conv2d_rs_f64(const double* x, const double* g, double* y,
                         int N, int C, int H, int W, int K, int R, int S, int pad, int absval)
{
    if (!x || !g || !y || N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || R <= 0 || S <= 0 || pad < 0)
        return -1;
    const long Ho = (long)H + 2L * pad - (R - 1);
    const long Wo = (long)W + 2L * pad - (S - 1);
    if (Ho < 1 || Wo < 1)
        return -1;

    long nk;
#pragma omp parallel for schedule(dynamic, 1)
    for (nk = 0; nk < (long)N * K; ++nk) {
        const long n = nk / K;
        const long k = nk % K;
        double* yo = y + ((n * K + k) * Ho) * Wo;
        for (long p = 0; p < Ho * Wo; ++p)
            yo[p] = 0.0;
        for (long c = 0; c < C; ++c) {
            const double* xi = x + ((n * C + c) * (long)H) * W;
            const double* gk = g + ((k * C + c) * (long)R) * S;
            for (long r = 0; r < R; ++r) {
                for (long s = 0; s < S; ++s) {
                    double w = gk[r * S + s];
                    if (absval) w = fabs(w);
                    for (long i = 0; i < Ho; ++i) {
                        const long u = i + r - pad;
                        if (u < 0 || u >= H) continue;       /* zero padding: row outside */
                        for (long j = 0; j < Wo; ++j) {
                            const long v = j + s - pad;
                            if (v < 0 || v >= W) continue;   /* zero padding: column outside */
                            double a = xi[u * W + v];
                            if (absval) a = fabs(a);
                            yo[i * Wo + j] += a * w;
                        }
                    }
                }
            }
        }
    }
    return 0;
}

/* Number of OpenMP threads the oracle's parallel loop will use. */
int oracle_num_threads(void)
{
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
