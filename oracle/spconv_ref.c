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

int spconv_ref_run(int32_t cout, int32_t cin, int32_t k,
                   const int32_t *row_ptr, const int32_t *col_idx,
                   const float *values, const float *bias, int32_t act,
                   const void *x, int32_t x_f16, int64_t n, int64_t hw,
                   double *y, double *scale)
{
    const int32_t rows = cout / k;
    int bad = 0;
    for (int32_t t = 0; t < row_ptr[rows]; ++t)
        if (col_idx[t] < 0 || col_idx[t] >= cin)
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
                    /* stored order: ascending input channel for a valid CSR */
                    for (int32_t t = row_ptr[rb]; t < row_ptr[rb + 1]; ++t) {
                        const int64_t c = col_idx[t];
                        const double wv = (double)values[(int64_t)t * k + i];
                        const int64_t xrow = (img * cin + c) * hw;
                        for (int64_t p = 0; p < hw; ++p) {
                            const double xv = x_f16
                                ? spconv_ref_half_to_double(((const uint16_t *)x)[xrow + p])
                                : (double)((const float *)x)[xrow + p];
                            const double prod = wv * xv;
                            acc[p] += prod;
                            s[p] += fabs(prod);
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
