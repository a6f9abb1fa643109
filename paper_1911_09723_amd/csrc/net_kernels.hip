// gfx950 kernels for the CHW operators around the sparse 1x1 in a MobileNet
// (Fast Sparse ConvNets, Sec. 3.1 and Sec. 3.3): the dense 3x3 convolution
// that reads the HWC image and writes CHW, a standalone depthwise 3x3 (for
// layers whose strip does not fit the fused strip kernel), global average
// pooling and the dense classifier.  All three are memory-bound elementwise-style kernels:
// one thread per output element (per output pixel for the convolution), fp32
// arithmetic, zero padding 1.
#include <hip/hip_runtime.h>

#include <algorithm>
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
// field once (zeros outside the image) and produces all cout channels.  A
// weight is the same for every lane, so the weights are read through the
// constant address space: scalar loads into SGPRs that each FMA takes as an
// operand (an LDS copy costs one LDS read per four FMAs and bounds the
// kernel).  Workgroup = 256 consecutive pixels of one image (block b covers
// image b / bpi), so no thread divides 64-bit indices; consecutive threads
// are consecutive pixels and each channel's stores coalesce.
using ConstF = const __attribute__((address_space(4))) float;

template <int CIN>
__global__ void __launch_bounds__(256)
conv3x3_hwc_kernel(const float *__restrict__ x, const float *__restrict__ wt, const float *__restrict__ bias,
                   float *__restrict__ y, int32_t bpi, int32_t h, int32_t w, int32_t ho, int32_t wo,
                   int32_t cout, int32_t stride, int32_t act) {
    const int32_t img = blockIdx.x / bpi;
    const int32_t plane = ho * wo;
    const int32_t pp = (blockIdx.x - img * bpi) * 256 + threadIdx.x;
    if (pp >= plane)
        return;
    const int32_t oy = pp / wo, ox = pp - oy * wo;
    const float *xi = x + static_cast<int64_t>(img) * h * w * CIN;
    float v[9][CIN];
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
        const int32_t iy = oy * stride + dy - 1;
#pragma unroll
        for (int dx = 0; dx < 3; ++dx) {
            const int32_t ix = ox * stride + dx - 1;
            const bool in = iy >= 0 && iy < h && ix >= 0 && ix < w;
            const float *px = xi + ((in ? iy : 0) * w + (in ? ix : 0)) * CIN;
#pragma unroll
            for (int i = 0; i < CIN; ++i)
                v[dy * 3 + dx][i] = in ? px[i] : 0.0f;
        }
    }
    float *yo = y + static_cast<int64_t>(img) * cout * plane + pp;
    ConstF *cw = (ConstF *)wt;
    ConstF *cb = (ConstF *)bias;
#pragma unroll 2
    for (int32_t o = 0; o < cout; ++o) {
        ConstF *wo9 = cw + o * 9 * CIN;
        float acc = 0.0f;
#pragma unroll
        for (int t = 0; t < 9; ++t)
#pragma unroll
            for (int i = 0; i < CIN; ++i)
                acc = __builtin_fmaf(wo9[t * CIN + i], v[t][i], acc);
        yo[static_cast<int64_t>(o) * plane] = clamp_act(acc + (cb ? cb[o] : 0.0f), act);
    }
}

// Depthwise 3x3 by columns: lane = one output column ox of one (n, c)
// plane and a group of D consecutive output rows oy0 .. oy0 + D - 1.  The
// lane loads the S*D + 3 - S input rows the group needs (3 values each, its
// columns S*ox - 1 .. S*ox + 1) all at once, so a wavefront waits for
// memory once, then forms its D outputs in registers.  A wavefront holds
// 64 / wo whole planes side by side when wo <= 64 (lane l: plane l / wo,
// column l % wo), else one 64-column part of a plane; its lanes share the
// row group, so a row in the top or bottom padding is the same for all of
// them.  Taps in dy, dx order from zero, then the bias, then the activation;
// a tap in the padding multiplies a zero (+0 added to a sum that started at
// +0 changes nothing).
template <int S, int D>
__global__ void __launch_bounds__(256)
dw3x3_cols_kernel(const float *__restrict__ x, const float *__restrict__ k, const float *__restrict__ bias,
                  float *__restrict__ y, int64_t planes, int32_t c, int32_t h, int32_t w, int32_t ho, int32_t wo,
                  int32_t act, int32_t ppw, int32_t wpp, int32_t segs) {
    const int32_t lane = threadIdx.x & 63;
    const int32_t gw = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // grid wavefront
    const int32_t unit = gw / segs;  // plane group (or plane part) of this wavefront
    const int32_t seg = gw - unit * segs;
    int64_t plane0;  // first plane of the wavefront
    int32_t sub, ox;
    if (wpp == 0) {
        plane0 = static_cast<int64_t>(unit) * ppw;
        sub = lane / wo;
        ox = lane - sub * wo;
        if (sub >= ppw)
            return;
    } else {
        const int32_t pl = unit / wpp;
        plane0 = pl;
        sub = 0;
        ox = (unit - pl * wpp) * 64 + lane;
        if (ox >= wo)
            return;
    }
    const int64_t plane = plane0 + sub;
    if (plane >= planes)
        return;
    const int32_t ch = (static_cast<int32_t>(plane0 % c) + sub) % c;
    float kk[9];
#pragma unroll
    for (int t = 0; t < 9; ++t)
        kk[t] = k[ch * 9 + t];
    const float b = bias ? bias[ch] : 0.0f;
    const float lo = act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = act == 2 ? 6.0f : __builtin_huge_valf();
    const float *xp = x + plane * h * w;
    float *yp = y + plane * ho * wo + ox;
    // this lane's three input columns; one outside the image reads column
    // ix1 (always inside) and is replaced by zero, as is a row outside it
    // (read as row 0).  The rows are loaded raw and masked after they land.
    const int32_t ix1 = ox * S;
    const bool lok = ix1 >= 1, rok = ix1 + 1 < w;
    const int32_t ix0 = lok ? ix1 - 1 : ix1, ix2 = rok ? ix1 + 1 : ix1;
    const int32_t oy0 = seg * D;
    constexpr int R = S * D + 3 - S;  // input rows S*oy0 - 1 .. S*(oy0 + D - 1) + 1
    float win[R][3];
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int32_t iy = S * oy0 - 1 + i;
        const float *r = xp + (iy >= 0 && iy < h ? iy : 0) * w;
        win[i][0] = r[ix0];
        win[i][1] = r[ix1];
        win[i][2] = r[ix2];
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int32_t iy = S * oy0 - 1 + i;
        const bool in = iy >= 0 && iy < h;  // the same for the whole wavefront
        win[i][0] = in && lok ? win[i][0] : 0.0f;
        win[i][1] = in ? win[i][1] : 0.0f;
        win[i][2] = in && rok ? win[i][2] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < D; ++j) {
        if (oy0 + j < ho) {
            float acc = 0.0f;
#pragma unroll
            for (int dy = 0; dy < 3; ++dy)
#pragma unroll
                for (int dx = 0; dx < 3; ++dx)
                    acc = __builtin_fmaf(kk[dy * 3 + dx], win[S * j + dy][dx], acc);
            yp[(oy0 + j) * wo] = fminf(fmaxf(acc + b, lo), hi);
        }
    }
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

// Global average pooling for small planes (hw <= kGapMaxHw): a wavefront
// owns 64 consecutive planes, whose 64 hw values are contiguous; it copies
// them into LDS with coalesced loads (16 bytes per lane when aligned), then
// each lane sums one plane in ascending p in fp32, as gap_kernel does.
constexpr int32_t kGapMaxHw = 256;

template <bool VEC>
__global__ void __launch_bounds__(64)
gap_staged_kernel(const float *__restrict__ x, float *__restrict__ y, int64_t planes, int32_t hw, float inv) {
    extern __shared__ __align__(16) float buf[];
    const int lane = threadIdx.x;
    const int64_t q0 = static_cast<int64_t>(blockIdx.x) * 64;
    const int32_t nq = static_cast<int32_t>(planes - q0 < 64 ? planes - q0 : 64);
    const int32_t total = nq * hw;
    const float *src = x + q0 * hw;
    if constexpr (VEC) {
        const int32_t nvec = total / 4;  // whole 16-byte groups, then the last few values
#pragma unroll 8
        for (int32_t v = lane; v < nvec; v += 64)
            *reinterpret_cast<f4 *>(buf + 4 * v) = *reinterpret_cast<const f4 *>(src + 4 * v);
        for (int32_t t = 4 * nvec + lane; t < total; t += 64)
            buf[t] = src[t];
    } else {
        for (int32_t t = lane; t < total; t += 64)
            buf[t] = src[t];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane >= nq)
        return;
    const float *pl = buf + lane * hw;
    float acc = 0.0f;
    for (int32_t p = 0; p < hw; ++p)
        acc += pl[p];
    y[q0 + lane] = acc * inv;
}

// Dense fully connected layer (the classifier the paper keeps dense, Sec. 3.1):
//   y[n, r] = act(b[r] + sum_c W[r, c] * x[n, c]),  W row-major [cout][cin].
// Lane = image (64 per wavefront), kLinRows rows per workgroup: every
// wavefront reads its lanes' images with 16-byte loads (each line serves 8 of
// them through L1) and the rows' weights, the same for all lanes, with
// scalar loads.  The kLinSplit wavefronts of a workgroup take consecutive
// ranges of the input channels; each lane sums its range in ascending c by
// fp32 FMA from zero, the range sums are added in ascending order through
// LDS, then the bias, then the activation.  VEC: 16-byte loads (cin a
// multiple of 4, x and W 16-byte aligned).
constexpr int kLinRows = 4;
constexpr int kLinSplit = 16;

template <bool VEC>
__global__ void __launch_bounds__(64 * kLinSplit)
linear_kernel(const float *__restrict__ x, const float *__restrict__ wt, const float *__restrict__ bias,
              float *__restrict__ y, int32_t n, int32_t cin, int32_t cout, int32_t act) {
    __shared__ float part[kLinSplit][kLinRows][64];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int32_t r0 = blockIdx.x * kLinRows;
    const int32_t img = blockIdx.y * 64 + lane;
    const float *xr = x + static_cast<int64_t>(img < n ? img : n - 1) * cin;
    int32_t chunk = (cin + kLinSplit - 1) / kLinSplit;
    if constexpr (VEC)
        chunk = (chunk + 3) & ~3;
    const int32_t c0 = wave * chunk < cin ? wave * chunk : cin;
    const int32_t c1 = c0 + chunk < cin ? c0 + chunk : cin;
    typedef const __attribute__((address_space(4))) float cfloat;
    typedef const __attribute__((address_space(4))) f4 cf4;
    cfloat *wr[kLinRows];
#pragma unroll
    for (int i = 0; i < kLinRows; ++i)
        wr[i] = (cfloat *)(wt + static_cast<int64_t>(r0 + i < cout ? r0 + i : cout - 1) * cin);
    float acc[kLinRows] = {};
    if constexpr (VEC) {
#pragma unroll 4
        for (int32_t c = c0; c < c1; c += 4) {
            const f4 xv = *reinterpret_cast<const f4 *>(xr + c);
#pragma unroll
            for (int i = 0; i < kLinRows; ++i) {
                const f4 wv = *(cf4 *)(wr[i] + c);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[i] = __builtin_fmaf(wv[e], xv[e], acc[i]);
            }
        }
    } else {
        for (int32_t c = c0; c < c1; ++c) {
            const float xv = xr[c];
#pragma unroll
            for (int i = 0; i < kLinRows; ++i)
                acc[i] = __builtin_fmaf(wr[i][c], xv, acc[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < kLinRows; ++i)
        part[wave][i][lane] = acc[i];
    __syncthreads();
    if (threadIdx.x >= 64 * kLinRows)
        return;
    const int i = threadIdx.x >> 6;
    const int32_t r = r0 + i;
    if (r >= cout || img >= n)
        return;
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < kLinSplit; ++w)
        sum += part[w][i][lane];
    y[static_cast<int64_t>(img) * cout + r] = clamp_act(sum + (bias ? bias[r] : 0.0f), act);
}

using ConvFn = void (*)(const float *, const float *, const float *, float *, int32_t, int32_t, int32_t, int32_t,
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
// output rows per wavefront of the depthwise kernel, stride 1 and 2
constexpr int kDwRows1 = 8;
constexpr int kDwRows2 = 4;

}  // namespace

hipError_t launch_conv3x3_hwc(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t h,
                              int32_t w, int32_t cin, int32_t cout, int32_t stride, int32_t act,
                              hipStream_t stream) {
    ConvFn kern = pick_conv(cin);
    if (!kern)
        return hipErrorInvalidValue;
    const int32_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t bpi = (static_cast<int64_t>(ho) * wo + kThreads - 1) / kThreads;
    // per-image offsets are 32-bit, the grid one dimension
    if (static_cast<int64_t>(h) * w * cin >= INT32_MAX || bpi * n >= INT32_MAX)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(bpi * n)), dim3(kThreads), 0, stream, x, wt, bias, y,
                       static_cast<int32_t>(bpi), h, w, ho, wo, cout, stride, act);
    return hipGetLastError();
}

hipError_t launch_dw3x3(const float *x, const float *k, const float *bias, float *y, int32_t n, int32_t c,
                        int32_t h, int32_t w, int32_t stride, int32_t act, hipStream_t stream) {
    const int32_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t planes = static_cast<int64_t>(n) * c;
    // wavefront layout: whole planes side by side, or 64-column parts; one
    // group of output rows each
    const int32_t ppw = wo <= 64 ? 64 / wo : 0;
    const int32_t wpp = wo <= 64 ? 0 : (wo + 63) / 64;
    const int64_t units = wo <= 64 ? (planes + ppw - 1) / ppw : planes * wpp;
    const int32_t rows = stride == 1 ? kDwRows1 : kDwRows2;
    const int32_t segs = (ho + rows - 1) / rows;
    const int64_t waves = units * segs;
    if (waves >= INT32_MAX - 3 || static_cast<int64_t>(h) * w >= INT32_MAX)
        return hipErrorInvalidValue;
    auto kern = stride == 1 ? dw3x3_cols_kernel<1, kDwRows1> : dw3x3_cols_kernel<2, kDwRows2>;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>((waves + 3) / 4)), dim3(kThreads), 0, stream, x, k, bias, y,
                       planes, c, h, w, ho, wo, act, ppw, wpp, segs);
    return hipGetLastError();
}

hipError_t launch_linear(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t cin,
                         int32_t cout, int32_t act, hipStream_t stream) {
    const bool vec = cin % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(wt) % 16 == 0;
    const dim3 grid(static_cast<unsigned>((cout + kLinRows - 1) / kLinRows), static_cast<unsigned>((n + 63) / 64));
    if (vec)
        hipLaunchKernelGGL(linear_kernel<true>, grid, dim3(64 * kLinSplit), 0, stream, x, wt, bias, y, n, cin, cout,
                           act);
    else
        hipLaunchKernelGGL(linear_kernel<false>, grid, dim3(64 * kLinSplit), 0, stream, x, wt, bias, y, n, cin,
                           cout, act);
    return hipGetLastError();
}

hipError_t launch_gap(const float *x, float *y, int32_t n, int32_t c, int64_t hw, hipStream_t stream) {
    const int64_t planes = static_cast<int64_t>(n) * c;
    if (hw <= kGapMaxHw) {
        const bool vec = reinterpret_cast<uintptr_t>(x) % 16 == 0;  // every group starts 256 hw bytes in
        const unsigned gblocks = static_cast<unsigned>((planes + 63) / 64);
        const size_t lds = static_cast<size_t>(64) * hw * sizeof(float);
        if (vec)
            hipLaunchKernelGGL(gap_staged_kernel<true>, dim3(gblocks), dim3(64), lds, stream, x, y, planes,
                               static_cast<int32_t>(hw), 1.0f / static_cast<float>(hw));
        else
            hipLaunchKernelGGL(gap_staged_kernel<false>, dim3(gblocks), dim3(64), lds, stream, x, y, planes,
                               static_cast<int32_t>(hw), 1.0f / static_cast<float>(hw));
        return hipGetLastError();
    }
    const int64_t blocks = (planes + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(gap_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, x, y, planes,
                       hw, 1.0f / static_cast<float>(hw));
    return hipGetLastError();
}

}  // namespace spconv
