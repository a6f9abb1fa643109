// gfx950 kernels for the CHW operators around the sparse 1x1 in a MobileNet
// (Fast Sparse ConvNets, Sec. 3.1 and Sec. 3.3): the dense 3x3 convolution
// that reads the HWC image and writes CHW, a standalone depthwise 3x3 (for
// layers whose strip does not fit the fused strip kernel), global average
// pooling and the dense classifier.  All three are memory-bound elementwise-style kernels:
// one thread per output element (per output pixel for the convolution), fp32
// arithmetic, zero padding 1.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "net_kernels.hpp"

namespace spconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float clamp_act(float v, int32_t act) {
    const float lo = act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = act == 2 ? 6.0f : __builtin_huge_valf();
    return fminf(fmaxf(v, lo), hi);
}

// Dense 3x3 convolution, HWC in, CHW out:
//   Y[n, o, oy, ox] = act(b[o] + sum_{dy, dx, i} Wt[o][dy][dx][i] * X[n, s*oy + dy - 1, s*ox + dx - 1, i])
// Thread = one output pixel: it gathers the 9 * CIN inputs of its receptive
// field once (zeros outside the image) and produces all cout channels, the
// weights read from LDS (every lane reads the same word: a broadcast).
// Consecutive threads are consecutive ox, so each channel's stores coalesce.
template <int CIN>
__global__ void __launch_bounds__(256)
conv3x3_hwc_kernel(const float *__restrict__ x, const float *__restrict__ wt, const float *__restrict__ bias,
                   float *__restrict__ y, int64_t pixels, int32_t h, int32_t w, int32_t ho, int32_t wo,
                   int32_t cout, int32_t stride, int32_t act) {
    extern __shared__ float sw[];  // cout * 9 * CIN weights, then cout biases
    const int32_t nw = cout * 9 * CIN;
    for (int32_t i = threadIdx.x; i < nw; i += blockDim.x)
        sw[i] = wt[i];
    for (int32_t i = threadIdx.x; i < cout; i += blockDim.x)
        sw[nw + i] = bias ? bias[i] : 0.0f;
    __syncthreads();
    const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= pixels)
        return;
    const int64_t img = q / (static_cast<int64_t>(ho) * wo);
    const int32_t pp = static_cast<int32_t>(q - img * ho * wo);
    const int32_t oy = pp / wo, ox = pp - oy * wo;
    float v[9][CIN];
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
        const int32_t iy = oy * stride + dy - 1;
#pragma unroll
        for (int dx = 0; dx < 3; ++dx) {
            const int32_t ix = ox * stride + dx - 1;
            const bool in = iy >= 0 && iy < h && ix >= 0 && ix < w;
            const float *px = x + ((img * h + (in ? iy : 0)) * w + (in ? ix : 0)) * CIN;
#pragma unroll
            for (int i = 0; i < CIN; ++i)
                v[dy * 3 + dx][i] = in ? px[i] : 0.0f;
        }
    }
    const int64_t plane = static_cast<int64_t>(ho) * wo;
    float *yo = y + img * cout * plane + pp;
    for (int32_t o = 0; o < cout; ++o) {
        const float *wo9 = sw + o * 9 * CIN;
        float acc = 0.0f;
#pragma unroll
        for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int i = 0; i < CIN; ++i)
                acc = __builtin_fmaf(wo9[t * CIN + i], v[t][i], acc);
        yo[o * plane] = clamp_act(acc + sw[nw + o], act);
    }
}

// Depthwise 3x3: thread = one output element (n, c, oy, ox), taps in dy, dx
// order from zero, then the bias, then the activation.
__global__ void __launch_bounds__(256)
dw3x3_kernel(const float *__restrict__ x, const float *__restrict__ k, const float *__restrict__ bias,
             float *__restrict__ y, int64_t total, int32_t c, int32_t h, int32_t w, int32_t ho, int32_t wo,
             int32_t stride, int32_t act) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= total)
        return;
    const int64_t plane_o = static_cast<int64_t>(ho) * wo;
    const int64_t nc = q / plane_o;  // n * c + channel
    const int32_t ch = static_cast<int32_t>(nc % c);
    const int32_t pp = static_cast<int32_t>(q - nc * plane_o);
    const int32_t oy = pp / wo, ox = pp - oy * wo;
    const float *xc = x + nc * h * static_cast<int64_t>(w);
    const float *kc = k + ch * 9;
    float acc = 0.0f;
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
        const int32_t iy = oy * stride + dy - 1;
        if (iy < 0 || iy >= h)
            continue;
#pragma unroll
        for (int dx = 0; dx < 3; ++dx) {
            const int32_t ix = ox * stride + dx - 1;
            if (ix >= 0 && ix < w)
                acc = __builtin_fmaf(kc[dy * 3 + dx], xc[static_cast<int64_t>(iy) * w + ix], acc);
        }
    }
    y[q] = clamp_act(acc + (bias ? bias[ch] : 0.0f), act);
}

// Global average pooling: thread = one (n, c) plane, summed in ascending
// position from zero in fp32, then multiplied by 1 / hw.
__global__ void __launch_bounds__(256)
gap_kernel(const float *__restrict__ x, float *__restrict__ y, int64_t planes, int64_t hw, float inv) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= planes)
        return;
    const float *xp = x + q * hw;
    float acc = 0.0f;
    for (int64_t p = 0; p < hw; ++p)
        acc += xp[p];
    y[q] = acc * inv;
}

// Dense fully connected layer (the classifier the paper keeps dense, Sec. 3.1):
//   y[n, r] = act(b[r] + sum_c W[r, c] * x[n, c]),  W row-major [cout][cin].
// A wavefront owns 64 consecutive rows (lane = row) and kImg images: each W
// load feeds kImg FMAs, the x loads are the same address in every lane (one
// line per instruction), and the stores are consecutive rows.  VEC: 16-byte
// loads (cin a multiple of 4, pointers 16-byte aligned).  fp32 FMA in
// ascending c from zero, then the bias, then the activation.
constexpr int kImg = 4;

template <bool VEC>
__global__ void __launch_bounds__(64)
linear_kernel(const float *__restrict__ x, const float *__restrict__ wt, const float *__restrict__ bias,
              float *__restrict__ y, int32_t n, int32_t cin, int32_t cout, int32_t act) {
    const int32_t r = blockIdx.x * 64 + threadIdx.x;
    const int32_t n0 = blockIdx.y * kImg;
    const int32_t rr = r < cout ? r : cout - 1;  // past the last row: compute row cout - 1, store nothing
    const float *wr = wt + static_cast<int64_t>(rr) * cin;
    const float *xi[kImg];
#pragma unroll
    for (int i = 0; i < kImg; ++i)
        xi[i] = x + static_cast<int64_t>(n0 + i < n ? n0 + i : n - 1) * cin;
    float acc[kImg] = {};
    if constexpr (VEC) {
        for (int32_t c = 0; c < cin; c += 4) {
            const f4 wv = *reinterpret_cast<const f4 *>(wr + c);
#pragma unroll
            for (int i = 0; i < kImg; ++i) {
                const f4 xv = *reinterpret_cast<const f4 *>(xi[i] + c);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[i] = __builtin_fmaf(wv[e], xv[e], acc[i]);
            }
        }
    } else {
        for (int32_t c = 0; c < cin; ++c) {
            const float wv = wr[c];
#pragma unroll
            for (int i = 0; i < kImg; ++i)
                acc[i] = __builtin_fmaf(wv, xi[i][c], acc[i]);
        }
    }
    if (r >= cout)
        return;
    const float b = bias ? bias[r] : 0.0f;
#pragma unroll
    for (int i = 0; i < kImg; ++i)
        if (n0 + i < n)
            y[static_cast<int64_t>(n0 + i) * cout + r] = clamp_act(acc[i] + b, act);
}

using ConvFn = void (*)(const float *, const float *, const float *, float *, int64_t, int32_t, int32_t, int32_t,
                        int32_t, int32_t, int32_t, int32_t);

ConvFn pick_conv(int32_t cin) {
    switch (cin) {
    case 1: return conv3x3_hwc_kernel<1>;
    case 2: return conv3x3_hwc_kernel<2>;
    case 3: return conv3x3_hwc_kernel<3>;
    case 4: return conv3x3_hwc_kernel<4>;
    case 5: return conv3x3_hwc_kernel<5>;
    case 6: return conv3x3_hwc_kernel<6>;
    case 7: return conv3x3_hwc_kernel<7>;
    case 8: return conv3x3_hwc_kernel<8>;
    default: return nullptr;
    }
}

constexpr int kThreads = 256;

}  // namespace

hipError_t launch_conv3x3_hwc(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t h,
                              int32_t w, int32_t cin, int32_t cout, int32_t stride, int32_t act,
                              hipStream_t stream) {
    ConvFn kern = pick_conv(cin);
    if (!kern)
        return hipErrorInvalidValue;
    const int32_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t pixels = static_cast<int64_t>(n) * ho * wo;
    const int64_t blocks = (pixels + kThreads - 1) / kThreads;
    const size_t lds = static_cast<size_t>(cout) * (9 * cin + 1) * sizeof(float);
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, stream, x, wt, bias, y,
                       pixels, h, w, ho, wo, cout, stride, act);
    return hipGetLastError();
}

hipError_t launch_dw3x3(const float *x, const float *k, const float *bias, float *y, int32_t n, int32_t c,
                        int32_t h, int32_t w, int32_t stride, int32_t act, hipStream_t stream) {
    const int32_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t total = static_cast<int64_t>(n) * c * ho * wo;
    const int64_t blocks = (total + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(dw3x3_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, x, k, bias,
                       y, total, c, h, w, ho, wo, stride, act);
    return hipGetLastError();
}

hipError_t launch_linear(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t cin,
                         int32_t cout, int32_t act, hipStream_t stream) {
    const bool vec = cin % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(wt) % 16 == 0;
    const dim3 grid(static_cast<unsigned>((cout + 63) / 64), static_cast<unsigned>((n + kImg - 1) / kImg));
    if (vec)
        hipLaunchKernelGGL(linear_kernel<true>, grid, dim3(64), 0, stream, x, wt, bias, y, n, cin, cout, act);
    else
        hipLaunchKernelGGL(linear_kernel<false>, grid, dim3(64), 0, stream, x, wt, bias, y, n, cin, cout, act);
    return hipGetLastError();
}

hipError_t launch_gap(const float *x, float *y, int32_t n, int32_t c, int64_t hw, hipStream_t stream) {
    const int64_t planes = static_cast<int64_t>(n) * c;
    const int64_t blocks = (planes + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(gap_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, x, y, planes,
                       hw, 1.0f / static_cast<float>(hw));
    return hipGetLastError();
}

}  // namespace spconv
