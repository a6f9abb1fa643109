// Internal interface between the C ABI and the network-operator kernels
// (net_kernels.hip).  Arguments are validated by the caller.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace spconv {

// Dense 3x3 convolution, padding 1: x [n][h][w][cin] -> y [n][cout][ho][wo];
// wt [cout][3][3][cin]; bias [cout] or null; 1 <= cin <= 8.
hipError_t launch_conv3x3_hwc(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t h,
                              int32_t w, int32_t cin, int32_t cout, int32_t stride, int32_t act, hipStream_t stream);

// Depthwise 3x3, padding 1: x [n][c][h][w] -> y [n][c][ho][wo]; k [c][3][3]; bias [c] or null.
hipError_t launch_dw3x3(const float *x, const float *k, const float *bias, float *y, int32_t n, int32_t c,
                        int32_t h, int32_t w, int32_t stride, int32_t act, hipStream_t stream);

// Dense fully connected layer: x [n][cin], wt [cout][cin], bias [cout] or null -> y [n][cout].
hipError_t launch_linear(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t cin,
                         int32_t cout, int32_t act, hipStream_t stream);

// Global average pooling: x [n][c][hw] -> y [n][c].
hipError_t launch_gap(const float *x, float *y, int32_t n, int32_t c, int64_t hw, hipStream_t stream);

}  // namespace spconv
