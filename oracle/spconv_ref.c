/*
 * CPU oracle for the sparse 1x1 convolution (test infrastructure only).
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use
 * this file.  It shares no code with the GPU library: it is the plain
 * definition of the operation, evaluated slowly in double precision.
 *
 * Definition (paper Sec. 1 and Sec. 3.2 with Fig. 2: a 1x1 convolution over a
 * CHW tensor is the product of the Cout x Cin weight matrix with the
 * Cin x (H*W) activation matrix; Sec. 3.2: with 1xk output-channel blocks, k
 * consecutive output channels share one nonzero pattern; Sec. 3.3: weights are
 * stored in a block-compressed-sparse-row format).  The fused bias and
 * activation come from the layer specification, not from the paper:
 *
 *     Y[n, r, p] = act( b[r] + sum_{stored (r, c)} W[r, c] * X[n, c, p] )
 *
 * for every image n, output channel r and spatial position p.
 *
 * Arguments
 *   cout, cin, k      output channels, input channels, output-block height (1 = CSR)
 *   row_ptr[cout/k+1] block-row offsets into col_idx
 *   col_idx[nnzb]     input channel of each stored block
 *   values[nnzb*k]    block-major values: values[t*k + i] = W[rb*k + i, col_idx[t]]
 *   bias[cout]        may be NULL (zeros)
 *   act               0 none, 1 max(v, 0), 2 min(max(v, 0), 6)
 *   x_f16             0: x is float[n][cin][hw]; 1: x holds IEEE binary16 bit patterns
 *   y[n][cout][hw]    act(b + sum), before rounding to the storage type (double)
 *   scale[n][cout][hw] sum over the stored terms of |W[r, c] * X[n, c, p]|
 *                      (the scale of the floating-point error bound); may be NULL
 *
 * Each output element is accumulated in double, starting from zero, over the
 * stored blocks of its row in the order given (ascending channel for a valid
 * CSR), and the bias is added last.  Compiled with -ffp-contract=off so every
 * product and sum is rounded on its own.
 *
 * Returns 0, -1 if a column index is out of range, -2 if scratch allocation fails.
 *
 * Below it: the same stage over a double input (spconv_ref_run_f64), a
 * depthwise 3x3 stage (spconv_ref_dw3x3, and spconv_ref_dw3x3_f64 over a
 * double input) for the fused depthwise -> 1x1 path, and the other CHW
 * operators of a whole network (paper Sec. 3.1 and Sec. 3.3): the dense 3x3
 * convolution from an HWC image to CHW (spconv_ref_conv3x3_hwc) and global
 * average pooling (spconv_ref_gap).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

/* Decode one IEEE 754 binary16 value (1 sign, 5 exponent, 10 fraction bits). */
double spconv_ref_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0)
        v = ldexp((double)frac, -24);                 /* zero and subnormals: frac * 2^-24 */
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(frac | 0x400), expo - 25); /* (1024 + frac) * 2^(e-15-10) */
    return sign ? -v : v;
}

static double apply_act(double v, int act)
{
    if (act == 1)
        return v > 0.0 ? v : 0.0;
    if (act == 2) {
        if (!(v > 0.0))
            return 0.0;
        return v < 6.0 ? v : 6.0;
    }
    return v;
}

/* The 1x1 stage.  x_kind: 0 float, 1 binary16 bits, 2 double.  xs (may be
 * NULL): a per-input-element error scale of x itself, added to the output
 * scale as |W[r, c]| * xs[n, c, p] (used when x is the exact output of an
 * earlier stage that the GPU evaluates in fp32). */
static int ref_spmm(int32_t cout, int32_t cin, int32_t k, int32_t kc,
                    const int32_t *row_ptr, const int32_t *col_idx,
                    const float *values, const float *bias, int32_t act,
                    const void *x, int32_t x_kind, const double *xs, int64_t n, int64_t hw,
                    double *y, double *scale)
{
    const int32_t rows = cout / k;
    int bad = 0;
    for (int32_t t = 0; t < row_ptr[rows]; ++t)
        if (col_idx[t] < 0 || (int64_t)col_idx[t] + kc > cin)
            bad = 1;
    if (bad)
        return -1;

    int nomem = 0;
#pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(hw > 0 ? hw : 1));
        double *s = (double *)malloc(sizeof(double) * (size_t)(hw > 0 ? hw : 1));
        if (!acc || !s) {
#pragma omp atomic write
            nomem = 1;
        }
#pragma omp for collapse(2) schedule(dynamic, 1)
        for (int64_t img = 0; img < n; ++img) {
            for (int32_t rb = 0; rb < rows; ++rb) {
                if (!acc || !s)
                    continue;
                for (int32_t i = 0; i < k; ++i) {
                    const int32_t r = rb * k + i;
                    for (int64_t p = 0; p < hw; ++p) {
                        acc[p] = 0.0;
                        s[p] = 0.0;
                    }
                    /* stored order: ascending input channel for a valid CSR
                     * (blocks in order, the kc channels of a block ascending) */
                    for (int32_t t = row_ptr[rb]; t < row_ptr[rb + 1]; ++t) {
                        for (int32_t j = 0; j < kc; ++j) {
                            const int64_t c = (int64_t)col_idx[t] + j;
                            const double wv = (double)values[((int64_t)t * k + i) * kc + j];
                            const int64_t xrow = (img * cin + c) * hw;
                            for (int64_t p = 0; p < hw; ++p) {
                                const double xv = x_kind == 2 ? ((const double *)x)[xrow + p]
                                    : x_kind == 1 ? spconv_ref_half_to_double(((const uint16_t *)x)[xrow + p])
                                    : (double)((const float *)x)[xrow + p];
                                const double prod = wv * xv;
                                acc[p] += prod;
                                s[p] += fabs(prod);
                                if (xs)
                                    s[p] += fabs(wv) * xs[xrow + p];
                            }
                        }
                    }
                    const double b = bias ? (double)bias[r] : 0.0;
                    double *yr = y + (img * cout + r) * hw;
                    for (int64_t p = 0; p < hw; ++p)
                        yr[p] = apply_act(acc[p] + b, act);
                    if (scale) {
                        double *sr = scale + (img * cout + r) * hw;
                        for (int64_t p = 0; p < hw; ++p)
                            sr[p] = s[p];
                    }
                }
            }
        }
        free(acc);
        free(s);
    }
    if (nomem)
        return -2;
    return 0;
}

int spconv_ref_run(int32_t cout, int32_t cin, int32_t k,
                   const int32_t *row_ptr, const int32_t *col_idx,
                   const float *values, const float *bias, int32_t act,
                   const void *x, int32_t x_f16, int64_t n, int64_t hw,
                   double *y, double *scale)
{
    return ref_spmm(cout, cin, k, 1, row_ptr, col_idx, values, bias, act, x, x_f16 ? 1 : 0, NULL, n, hw, y,
                    scale);
}

/* The same with blocks of k output channels x kc input channels (Sec. 3.2
 * names the block shapes, Fig. 5 compares 1x4, 4x1 and 2x2 blocks):
 * col_idx[t] is the first input channel of block t and
 * values[(t * k + i) * kc + j] = W[rb * k + i, col_idx[t] + j]; a block
 * must lie inside [0, cin).  kc = 1 is spconv_ref_run. */
int spconv_ref_run_blocked(int32_t cout, int32_t cin, int32_t k, int32_t kc,
                           const int32_t *row_ptr, const int32_t *col_idx,
                           const float *values, const float *bias, int32_t act,
                           const void *x, int32_t x_f16, int64_t n, int64_t hw,
                           double *y, double *scale)
{
    if (kc < 1)
        return -1;
    return ref_spmm(cout, cin, k, kc, row_ptr, col_idx, values, bias, act, x, x_f16 ? 1 : 0, NULL, n, hw, y,
                    scale);
}

/* The 1x1 stage over a double-precision input x with its own error scale xs
 * (both [n][cin][hw]); the output scale is sum |W * x| + |W| * xs. */
int spconv_ref_run_f64(int32_t cout, int32_t cin, int32_t k,
                       const int32_t *row_ptr, const int32_t *col_idx,
                       const float *values, const float *bias, int32_t act,
                       const double *x, const double *xs, int64_t n, int64_t hw,
                       double *y, double *scale)
{
    return ref_spmm(cout, cin, k, 1, row_ptr, col_idx, values, bias, act, x, 2, xs, n, hw, y, scale);
}

/*
 * Depthwise 3x3 convolution with zero padding 1 and stride s over CHW images
 * (the MobileNet block: a depthwise convolution per channel, then the 1x1;
 * paper Sec. 2 and Sec. 3.3), evaluated in double:
 *
 *   D[n, c, oy, ox] = act( b[c] + sum_{dy, dx in 0..2} K[c, dy, dx] * X[n, c, s*oy + dy - 1, s*ox + dx - 1] )
 *
 * with X taken as zero outside the image; output size ho = (h - 1) / s + 1,
 * wo = (w - 1) / s + 1.  x: float [n][c][h][w]; k: float [c][3][3];
 * bias: [c] or NULL.  d: [n][c][ho][wo]; sd (may be NULL): the scale
 * |b[c]| + sum |K * X| of each output.  Returns 0, or -1 for a bad stride.
 */
int spconv_ref_dw3x3(int64_t n, int32_t c, int32_t h, int32_t w, int32_t stride,
                     const float *x, const float *k, const float *bias, int32_t act,
                     double *d, double *sd)
{
    if (stride < 1)
        return -1;
    const int64_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t img = 0; img < n; ++img) {
        for (int32_t ch = 0; ch < c; ++ch) {
            const float *xc = x + (img * c + ch) * (int64_t)h * w;
            const float *kc = k + (int64_t)ch * 9;
            const double b = bias ? (double)bias[ch] : 0.0;
            for (int64_t oy = 0; oy < ho; ++oy) {
                for (int64_t ox = 0; ox < wo; ++ox) {
                    double acc = 0.0, s = 0.0;
                    for (int dy = 0; dy < 3; ++dy) {
                        const int64_t iy = oy * stride + dy - 1;
                        if (iy < 0 || iy >= h)
                            continue;
                        for (int dx = 0; dx < 3; ++dx) {
                            const int64_t ix = ox * stride + dx - 1;
                            if (ix < 0 || ix >= w)
                                continue;
                            const double prod = (double)kc[dy * 3 + dx] * (double)xc[iy * w + ix];
                            acc += prod;
                            s += fabs(prod);
                        }
                    }
                    const int64_t o = ((img * c + ch) * ho + oy) * wo + ox;
                    d[o] = apply_act(acc + b, act);
                    if (sd)
                        sd[o] = s + fabs(b);
                }
            }
        }
    }
    return 0;
}

/*
 * The depthwise 3x3 stage over a double input x [n][c][h][w] with its own
 * error scale xs (same shape, may be NULL): as spconv_ref_dw3x3, and the
 * output scale also carries sum |K| * xs over the taps inside the image.
 */
int spconv_ref_dw3x3_f64(int64_t n, int32_t c, int32_t h, int32_t w, int32_t stride,
                         const double *x, const double *xs, const float *k, const float *bias, int32_t act,
                         double *d, double *sd)
{
    if (stride < 1)
        return -1;
    const int64_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t img = 0; img < n; ++img) {
        for (int32_t ch = 0; ch < c; ++ch) {
            const int64_t plane = (img * c + ch) * (int64_t)h * w;
            const float *kc = k + (int64_t)ch * 9;
            const double b = bias ? (double)bias[ch] : 0.0;
            for (int64_t oy = 0; oy < ho; ++oy) {
                for (int64_t ox = 0; ox < wo; ++ox) {
                    double acc = 0.0, s = 0.0;
                    for (int dy = 0; dy < 3; ++dy) {
                        const int64_t iy = oy * stride + dy - 1;
                        if (iy < 0 || iy >= h)
                            continue;
                        for (int dx = 0; dx < 3; ++dx) {
                            const int64_t ix = ox * stride + dx - 1;
                            if (ix < 0 || ix >= w)
                                continue;
                            const double kv = (double)kc[dy * 3 + dx];
                            const double prod = kv * x[plane + iy * w + ix];
                            acc += prod;
                            s += fabs(prod);
                            if (xs)
                                s += fabs(kv) * xs[plane + iy * w + ix];
                        }
                    }
                    const int64_t o = ((img * c + ch) * ho + oy) * wo + ox;
                    d[o] = apply_act(acc + b, act);
                    if (sd)
                        sd[o] = s + fabs(b);
                }
            }
        }
    }
    return 0;
}

/*
 * Dense 3x3 convolution from an HWC image to CHW (the network's first layer,
 * which the paper keeps dense and runs on the image in HWC order, writing the
 * CHW layout the sparse layers read; Sec. 3.1, Sec. 3.3):
 *
 *     Y[n, o, oy, ox] = act( b[o] + sum_{dy, dx in 0..2} sum_{i < cin}
 *                                     Wt[o][dy][dx][i] * X[n, s*oy + dy - 1, s*ox + dx - 1, i] )
 *
 * with X zero outside the image (padding 1) and stride s: ho = (h - 1) / s + 1,
 * wo = (w - 1) / s + 1.  x: float [n][h][w][cin]; wt: float
 * [cout][3][3][cin]; bias [cout] or NULL.  y: double [n][cout][ho][wo]; ys
 * (may be NULL): |b| + sum |Wt * X|.  Returns 0, or -1 for a bad stride.
 */
int spconv_ref_conv3x3_hwc(int64_t n, int32_t h, int32_t w, int32_t cin, int32_t cout, int32_t stride,
                           const float *x, const float *wt, const float *bias, int32_t act,
                           double *y, double *ys)
{
    if (stride < 1)
        return -1;
    const int64_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t img = 0; img < n; ++img) {
        for (int32_t o = 0; o < cout; ++o) {
            const double b = bias ? (double)bias[o] : 0.0;
            for (int64_t oy = 0; oy < ho; ++oy) {
                for (int64_t ox = 0; ox < wo; ++ox) {
                    double acc = 0.0, s = 0.0;
                    for (int dy = 0; dy < 3; ++dy) {
                        const int64_t iy = oy * stride + dy - 1;
                        if (iy < 0 || iy >= h)
                            continue;
                        for (int dx = 0; dx < 3; ++dx) {
                            const int64_t ix = ox * stride + dx - 1;
                            if (ix < 0 || ix >= w)
                                continue;
                            for (int32_t i = 0; i < cin; ++i) {
                                const double prod = (double)wt[((int64_t)o * 9 + dy * 3 + dx) * cin + i] *
                                                    (double)x[((img * h + iy) * w + ix) * cin + i];
                                acc += prod;
                                s += fabs(prod);
                            }
                        }
                    }
                    const int64_t q = ((img * cout + o) * ho + oy) * wo + ox;
                    y[q] = apply_act(acc + b, act);
                    if (ys)
                        ys[q] = s + fabs(b);
                }
            }
        }
    }
    return 0;
}

/*
 * Global average pooling over CHW planes (Sec. 3.3): y[n][c] = (1 / hw) *
 * sum_p x[n][c][p], the sum in ascending p from zero.  x: double
 * [n][c][hw]; xs (may be NULL): its error scale, pooled the same way into ys
 * together with sum |x| / hw.  Returns 0, or -1 for hw < 1.
 */
int spconv_ref_gap(int64_t n, int32_t c, int64_t hw, const double *x, const double *xs, double *y, double *ys)
{
    if (hw < 1)
        return -1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t img = 0; img < n; ++img) {
        for (int32_t ch = 0; ch < c; ++ch) {
            const double *xp = x + (img * c + ch) * hw;
            double acc = 0.0, s = 0.0;
            for (int64_t p = 0; p < hw; ++p) {
                acc += xp[p];
                s += fabs(xp[p]);
                if (xs)
                    s += xs[(img * c + ch) * hw + p];
            }
            y[img * c + ch] = acc / (double)hw;
            if (ys)
                ys[img * c + ch] = s / (double)hw;
        }
    }
    return 0;
}

/* Number of OpenMP threads the oracle runs with (1 when built without OpenMP). */
int spconv_ref_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
