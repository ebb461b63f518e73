/*
 * CPU oracle for block-sparse convolution with temporal feature copying.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path links, loads or calls
 * this file; only the tests, the package's smoke check and the benchmark's CPU
 * baseline leg do. It shares no code with the HIP path.
 *
 * What it computes is the plain definition of a 2-D convolution layer evaluated
 * at every output position (a dense layer, the operation that BlockCopy executes
 * block-sparsely, Section 3.1): a cross-correlation with zero padding, bias, an
 * optional residual term and an optional ReLU, accumulated in fp64 in the fixed
 * order ci -> i -> j. The block selection (which outputs are kept from the
 * previous execution) is applied afterwards, in oracle/__init__.py.
 *
 * Layout is the mathematical NCHW form with weights OIHW; all values are fp64.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

static double conv_point(const double *x, int cin, int h, int w,
                         const double *wt, int kh, int kw, int stride, int pad,
                         int nn, int co, int y, int xo)
{
    double acc = 0.0;
    for (int ci = 0; ci < cin; ++ci) {
        const double *xc = x + ((size_t)nn * cin + ci) * (size_t)h * w;
        const double *wc = wt + ((size_t)co * cin + ci) * (size_t)kh * kw;
        for (int i = 0; i < kh; ++i) {
            int iy = y * stride - pad + i;
            if (iy < 0 || iy >= h) continue;          /* zero padding */
            for (int j = 0; j < kw; ++j) {
                int ix = xo * stride - pad + j;
                if (ix < 0 || ix >= w) continue;      /* zero padding */
                acc += wc[i * kw + j] * xc[(size_t)iy * w + ix];
            }
        }
    }
    return acc;
}

static double finish(double acc, const double *bias, const double *res, size_t ridx,
                     int co, int relu)
{
    double z = acc;
    if (bias) z += bias[co];
    if (res) z += res[ridx];
    if (relu && !(z > 0.0)) z = (z != z) ? z : 0.0;   /* ReLU, NaN passes through */
    return z;
}

/* Dense layer: out[n][co][y][x] for every position. ho/wo are the PyTorch conv
 * output sizes floor((h + 2 pad - kh) / stride) + 1. */
void oracle_conv2d_dense(const double *x, int n, int cin, int h, int w,
                         const double *wt, int cout, int kh, int kw,
                         int stride, int pad, const double *bias,
                         const double *residual, int relu,
                         double *out, int ho, int wo)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int nn = 0; nn < n; ++nn)
        for (int co = 0; co < cout; ++co)
            for (int y = 0; y < ho; ++y)
                for (int xo = 0; xo < wo; ++xo) {
                    size_t o = (((size_t)nn * cout + co) * ho + y) * (size_t)wo + xo;
                    double acc = conv_point(x, cin, h, w, wt, kh, kw, stride, pad, nn, co, y, xo);
                    out[o] = finish(acc, bias, residual, o, co, relu);
                }
}

/* The same definition at listed output points pts[k] = (n, co, y, x); residual,
 * when given, is indexed like the full output [n][cout][ho][wo]. */
void oracle_conv2d_points(const double *x, int n, int cin, int h, int w,
                          const double *wt, int cout, int kh, int kw,
                          int stride, int pad, const double *bias,
                          const double *residual, int relu, int ho, int wo,
                          const int32_t *pts, int64_t npts, double *out)
{
    (void)n;
    #pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < npts; ++k) {
        int nn = pts[4 * k], co = pts[4 * k + 1], y = pts[4 * k + 2], xo = pts[4 * k + 3];
        size_t o = (((size_t)nn * cout + co) * ho + y) * (size_t)wo + xo;
        double acc = conv_point(x, cin, h, w, wt, kh, kw, stride, pad, nn, co, y, xo);
        out[k] = finish(acc, bias, residual, o, co, relu);
    }
}

/* The same definition at every output point of the listed output blocks only (the
 * oracle's "only active" mode: identical arithmetic per point, inactive blocks
 * skipped). Block id b = (img * gh + gy) * gw + gx covers output rows gy*bh ..
 * gy*bh + bh - 1 and columns gx*bw .. gx*bw + bw - 1 of image img; out is the full
 * [n][cout][ho][wo] array, written at those points only. */
void oracle_conv2d_blocks(const double *x, int n, int cin, int h, int w,
                          const double *wt, int cout, int kh, int kw,
                          int stride, int pad, const double *bias,
                          const double *residual, int relu, double *out, int ho, int wo,
                          const int32_t *blocks, int nblocks, int gh, int gw)
{
    (void)n;
    const int bh = ho / gh, bw = wo / gw;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int k = 0; k < nblocks; ++k)
        for (int co = 0; co < cout; ++co) {
            const int b = blocks[k];
            const int nn = b / (gh * gw), gy = (b % (gh * gw)) / gw, gx = b % gw;
            for (int y = gy * bh; y < (gy + 1) * bh; ++y)
                for (int xo = gx * bw; xo < (gx + 1) * bw; ++xo) {
                    size_t o = (((size_t)nn * cout + co) * ho + y) * (size_t)wo + xo;
                    double acc = conv_point(x, cin, h, w, wt, kh, kw, stride, pad, nn, co, y, xo);
                    out[o] = finish(acc, bias, residual, o, co, relu);
                }
        }
}

/* Dense max pooling with -inf padding (the padded positions never win). */
void oracle_maxpool2d_dense(const double *x, int n, int c, int h, int w,
                            int k, int stride, int pad, double *out, int ho, int wo)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int nn = 0; nn < n; ++nn)
        for (int cc = 0; cc < c; ++cc)
            for (int y = 0; y < ho; ++y)
                for (int xo = 0; xo < wo; ++xo) {
                    const double *xc = x + ((size_t)nn * c + cc) * (size_t)h * w;
                    double m = -INFINITY;
                    for (int i = 0; i < k; ++i) {
                        int iy = y * stride - pad + i;
                        if (iy < 0 || iy >= h) continue;
                        for (int j = 0; j < k; ++j) {
                            int ix = xo * stride - pad + j;
                            if (ix < 0 || ix >= w) continue;
                            double v = xc[(size_t)iy * w + ix];
                            if (v != v || v > m) m = (m != m) ? m : v;  /* NaN propagates */
                        }
                    }
                    out[(((size_t)nn * c + cc) * ho + y) * (size_t)wo + xo] = m;
                }
}

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
