// gfx950 kernels for the CHW operators around the sparse 1x1 in a MobileNet
// (Fast Sparse ConvNets, Sec. 3.1 and Sec. 3.3): the dense 3x3 convolution
// that reads the HWC image and writes CHW, a standalone depthwise 3x3, global
// average pooling and the dense classifier, all fp32 with zero padding 1.
// They are memory-bound: each keeps its loads and stores coalesced and its
// per-element instruction count small (weights that are the same for a whole
// wavefront come through scalar loads).
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

// Depthwise 3x3 by columns, for planes too wide for whole planes per
// wavefront: lane = one output column ox of one 64-column part of an
// (n, c) plane, walking down a segment of its output rows in groups of D.
// The lane holds the input rows of the current group in registers (its
// columns S*ox - 1 .. S*ox + 1, three loads per row), and the rows of the
// next group are loaded while the current one is computed; the lanes of a
// wavefront walk the same rows.  Taps in dy, dx order from zero, then the
// bias, then the activation; a tap in the padding multiplies a zero (+0
// added to a sum that started at +0 changes nothing).
//
// Addressing is 32-bit through buffer resources over the wavefront's
// planes: a tap in the padding (a column outside the image, or any row
// outside it) gets an offset past the resource's size, and the hardware
// returns zero for it without touching memory.
using Rsrc = __amdgpu_buffer_rsrc_t;
__device__ __forceinline__ Rsrc buffer_of(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0), static_cast<int>(bytes),
                                             0x00020000);
}
// Offset of a tap outside the image: at least 2^30 bytes, beyond every
// resource of this kernel (the host keeps a wavefront's planes below 2^30
// bytes), and two of them added stay below 2^32.
constexpr uint32_t kDwOut = 0x40000000u;

template <int S, int D>
__global__ void __launch_bounds__(256)
dw3x3_cols_kernel(const float *__restrict__ x, const float *__restrict__ k, const float *__restrict__ bias,
                  float *__restrict__ y, int64_t planes, int32_t c, int32_t h, int32_t w, int32_t ho, int32_t wo,
                  int32_t act, int32_t wpp, int32_t segs, int32_t seg_rows) {
    const int32_t lane = threadIdx.x & 63;
    const int32_t gw = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // grid wavefront
    const int32_t unit = gw / segs;  // plane part of this wavefront
    const int32_t seg = gw - unit * segs;
    const int64_t plane0 = unit / wpp;
    constexpr int32_t nwp = 1, sub = 0;
    const int32_t ox = static_cast<int32_t>(unit - plane0 * wpp) * 64 + lane;
    if (ox >= wo)
        return;
    const int32_t ch = (static_cast<int32_t>(plane0 % c) + sub) % c;
    float kk[9];
#pragma unroll
    for (int t = 0; t < 9; ++t)
        kk[t] = k[ch * 9 + t];
    const float b = bias ? bias[ch] : 0.0f;
    const float lo = act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t ihw = h * w, ohw = ho * wo;
    const Rsrc rx = buffer_of(x + plane0 * ihw, static_cast<uint32_t>(nwp * ihw * 4));
    const Rsrc ry = buffer_of(y + plane0 * ohw, static_cast<uint32_t>(nwp * ohw * 4));
    // byte offsets of this lane's three input columns in its plane (past
    // the resource when outside the image) and of its output column
    const int32_t ix1 = ox * S;
    const bool lok = ix1 >= 1, rok = ix1 + 1 < w;  // columns inside the image
    const uint32_t cbase = static_cast<uint32_t>(sub * ihw + ix1) * 4;
    const uint32_t c0 = lok ? cbase - 4 : kDwOut, c1 = cbase, c2 = rok ? cbase + 4 : kDwOut;
    const uint32_t yo = static_cast<uint32_t>(sub * ohw + ox) * 4;
    auto load_row = [&](int32_t iy, float *a) __attribute__((always_inline)) {
        const uint32_t ro = iy >= 0 && iy < h ? static_cast<uint32_t>(iy * w) * 4 : kDwOut;  // uniform
        a[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rx, c0 + ro, 0, 0));
        a[1] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rx, c1 + ro, 0, 0));
        a[2] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rx, c2 + ro, 0, 0));
    };
    // The window holds input rows S*oy - 1 .. S*(oy + D - 1) + 1 of group
    // oy: C rows carried from the last group and NR new ones, loaded while
    // the last group was computed.
    constexpr int C = 3 - S;
    constexpr int NR = S * D;
    const int32_t oy0 = seg * seg_rows;
    const int32_t oy1 = oy0 + seg_rows < ho ? oy0 + seg_rows : ho;
    float win[C + NR][3], nxt[NR][3];
#pragma unroll
    for (int i = 0; i < C; ++i)
        load_row(S * oy0 - 1 + i, win[i]);
#pragma unroll
    for (int i = 0; i < NR; ++i)
        load_row(S * oy0 - 1 + C + i, nxt[i]);
    for (int32_t oy = oy0; oy < oy1; oy += D) {
#pragma unroll
        for (int i = 0; i < NR; ++i)
#pragma unroll
            for (int e = 0; e < 3; ++e)
                win[C + i][e] = nxt[i][e];
        if (oy + D < oy1) {
#pragma unroll
            for (int i = 0; i < NR; ++i)
                load_row(S * (oy + D) - 1 + C + i, nxt[i]);
        }
#pragma unroll
        for (int j = 0; j < D; ++j) {
            if (oy + j < oy1) {
                float acc = 0.0f;
#pragma unroll
                for (int dy = 0; dy < 3; ++dy)
#pragma unroll
                    for (int dx = 0; dx < 3; ++dx)
                        acc = __builtin_fmaf(kk[dy * 3 + dx], win[S * j + dy][dx], acc);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fminf(fmaxf(acc + b, lo), hi)), ry, yo,
                                                      static_cast<int32_t>((oy + j) * wo * 4), 0);
            }
        }
#pragma unroll
        for (int i = 0; i < C; ++i)
#pragma unroll
            for (int e = 0; e < 3; ++e)
                win[i][e] = win[NR + i][e];
    }
}

// The same depthwise 3x3 with V adjacent output columns per lane and whole
// planes in every wavefront: lane = lane-column lc of one plane (outputs
// V*lc .. V*lc + V - 1), which loads its S*V input columns of a row with one
// or two V-wide loads (the address unit handles a lane per cycle, whatever
// the width, so wide loads move several times the bytes per cycle) and takes
// the column left of them (and, for stride 1, the one right of them) from the
// neighbouring lanes.  Needs w a multiple of S*V and x, y aligned to 4*V
// bytes; wo / V lane-columns per plane row at most 64.
template <int S, int V>
struct DwVec {
    static constexpr int D = S == 2 && V == 4 ? 2 : 4;  // output rows per group
    static constexpr int C = 3 - S;                      // rows carried between groups
    static constexpr int NR = S * D;                     // new rows per group
    static constexpr int RW = S * V + 3 - S;             // register row: left, S*V loaded, right (stride 1)
};

template <int V>
__device__ __forceinline__ void load_vec(Rsrc r, uint32_t off, float *dst) {
    if constexpr (V == 4) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            dst[e] = __uint_as_float(v[e]);
    } else if constexpr (V == 2) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
        dst[0] = __uint_as_float(v[0]);
        dst[1] = __uint_as_float(v[1]);
    } else {
        dst[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
    }
}

template <int V>
__device__ __forceinline__ void store_vec(Rsrc r, uint32_t off, int32_t soff, const float *src) {
    if constexpr (V == 4) {
        typedef uint32_t u4v __attribute__((ext_vector_type(4)));
        const u4v v = {__float_as_uint(src[0]), __float_as_uint(src[1]), __float_as_uint(src[2]),
                       __float_as_uint(src[3])};
        __builtin_amdgcn_raw_buffer_store_b128(v, r, off, soff, 0);
    } else if constexpr (V == 2) {
        typedef uint32_t u2v __attribute__((ext_vector_type(2)));
        const u2v v = {__float_as_uint(src[0]), __float_as_uint(src[1])};
        __builtin_amdgcn_raw_buffer_store_b64(v, r, off, soff, 0);
    } else {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(src[0]), r, off, soff, 0);
    }
}

template <int S, int V>
__global__ void __launch_bounds__(256)
dw3x3_vec_kernel(const float *__restrict__ x, const float *__restrict__ k, const float *__restrict__ bias,
                 float *__restrict__ y, int64_t planes, int32_t c, int32_t h, int32_t w, int32_t ho, int32_t wo,
                 int32_t act, int32_t ppw, int32_t segs, int32_t seg_rows) {
    using G = DwVec<S, V>;
    constexpr int D = G::D, C = G::C, NR = G::NR, RW = G::RW;
    const int32_t lane = threadIdx.x & 63;
    const int32_t gw = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // grid wavefront
    const int32_t unit = gw / segs;  // plane group of this wavefront
    const int32_t seg = gw - unit * segs;
    const int32_t lcols = wo / V;    // lane-columns per plane row
    const int64_t plane0 = static_cast<int64_t>(unit) * ppw;
    const int32_t nwp = static_cast<int32_t>(planes - plane0 < ppw ? planes - plane0 : ppw);
    const int32_t sub = lane / lcols;
    const int32_t lc = lane - sub * lcols;
    if (sub >= nwp)
        return;
    const int32_t ch = (static_cast<int32_t>(plane0 % c) + sub) % c;
    // the plane's 9 taps as three 12-byte loads (one address-unit cycle per
    // lane each, against nine for single words)
    float kk[9];
    {
        const Rsrc rk = buffer_of(k, static_cast<uint32_t>(c * 36));
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            const auto t = __builtin_amdgcn_raw_buffer_load_b96(rk, ch * 36 + q * 12, 0, 0);
#pragma unroll
            for (int e = 0; e < 3; ++e)
                kk[q * 3 + e] = __uint_as_float(t[e]);
        }
    }
    const float b = bias ? bias[ch] : 0.0f;
    const float lo = act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t ihw = h * w, ohw = ho * wo;
    const Rsrc rx = buffer_of(x + plane0 * ihw, static_cast<uint32_t>(nwp * ihw * 4));
    const Rsrc ry = buffer_of(y + plane0 * ohw, static_cast<uint32_t>(nwp * ohw * 4));
    const bool lok = lc > 0, rok = lc + 1 < lcols;  // neighbour lane of the same plane
    const uint32_t xo = static_cast<uint32_t>(sub * ihw + lc * S * V) * 4;
    // the second load of stride 2 (columns past the first V): past the row's
    // end only when V = 1 and w is odd, and then a padding tap
    const uint32_t xo1 = lc * S * V + V < w ? xo + V * 4 : kDwOut;
    const uint32_t yo = static_cast<uint32_t>(sub * ohw + lc * V) * 4;
    const int left = ((lane + 63) & 63) << 2, right = ((lane + 1) & 63) << 2;  // lane byte addresses
    // a row: S*V loaded values at [1 .. S*V]; [0] and (stride 1) [V + 1]
    // filled in from the neighbours once the loads have landed
    auto load_row = [&](int32_t iy, float *a) __attribute__((always_inline)) {
        const uint32_t ro = iy >= 0 && iy < h ? static_cast<uint32_t>(iy * w) * 4 : kDwOut;  // uniform row
        load_vec<V>(rx, xo + ro, a + 1);
        if constexpr (S == 2)
            load_vec<V>(rx, xo1 + ro, a + 1 + V);
    };
    auto finish_row = [&](float *a) __attribute__((always_inline)) {
        const float l = __int_as_float(__builtin_amdgcn_ds_bpermute(left, __float_as_int(a[S * V])));
        a[0] = lok ? l : 0.0f;
        if constexpr (S == 1) {
            const float r = __int_as_float(__builtin_amdgcn_ds_bpermute(right, __float_as_int(a[1])));
            a[V + 1] = rok ? r : 0.0f;
        }
    };
    const int32_t oy0 = seg * seg_rows;
    const int32_t oy1 = oy0 + seg_rows < ho ? oy0 + seg_rows : ho;
    float win[C + NR][RW], nxt[NR][RW];
#pragma unroll
    for (int i = 0; i < C; ++i)
        load_row(S * oy0 - 1 + i, win[i]);
#pragma unroll
    for (int i = 0; i < NR; ++i)
        load_row(S * oy0 - 1 + C + i, nxt[i]);
#pragma unroll
    for (int i = 0; i < C; ++i)
        finish_row(win[i]);
    for (int32_t oy = oy0; oy < oy1; oy += D) {
#pragma unroll
        for (int i = 0; i < NR; ++i) {
#pragma unroll
            for (int e = 0; e < RW; ++e)
                win[C + i][e] = nxt[i][e];
            finish_row(win[C + i]);
        }
        if (oy + D < oy1) {
#pragma unroll
            for (int i = 0; i < NR; ++i)
                load_row(S * (oy + D) - 1 + C + i, nxt[i]);
        }
#pragma unroll
        for (int j = 0; j < D; ++j) {
            if (oy + j < oy1) {
                float out[V];
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    // output column V*lc + v reads register columns S*v .. S*v + 2
                    float acc = 0.0f;
#pragma unroll
                    for (int dy = 0; dy < 3; ++dy)
#pragma unroll
                        for (int dx = 0; dx < 3; ++dx)
                            acc = __builtin_fmaf(kk[dy * 3 + dx], win[S * j + dy][S * v + dx], acc);
                    out[v] = fminf(fmaxf(acc + b, lo), hi);
                }
                store_vec<V>(ry, yo, static_cast<int32_t>((oy + j) * wo * 4), out);
            }
        }
#pragma unroll
        for (int i = 0; i < C; ++i)
#pragma unroll
            for (int e = 0; e < RW; ++e)
                win[i][e] = win[NR + i][e];
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
// owns kGapPlanes consecutive planes, whose values are contiguous; it copies
// them into its own LDS area with coalesced loads (16 bytes per lane when
// aligned, all of a lane's loads in flight at once), then each of the first
// kGapPlanes lanes sums one plane in ascending p in fp32, as gap_kernel
// does.  Four wavefronts per workgroup, 64 planes.
constexpr int32_t kGapMaxHw = 256;
constexpr int32_t kGapPlanes = 16;

template <bool VEC>
__global__ void __launch_bounds__(256)
gap_staged_kernel(const float *__restrict__ x, float *__restrict__ y, int64_t planes, int32_t hw, float inv) {
    extern __shared__ __align__(16) float buf[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    float *wb = buf + wave * kGapPlanes * hw;  // 64 hw bytes per wavefront: 16-byte aligned
    const int64_t q0 = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * kGapPlanes;
    if (q0 >= planes)
        return;
    const int32_t nq = static_cast<int32_t>(planes - q0 < kGapPlanes ? planes - q0 : kGapPlanes);
    const int32_t total = nq * hw;
    const float *src = x + q0 * hw;  // 64 hw bytes per group of planes: 16-byte aligned when x is
    if constexpr (VEC) {
        const int32_t nvec = total / 4;  // whole 16-byte groups, then the last few values
#pragma unroll 4
        for (int32_t v = lane; v < nvec; v += 64)
            *reinterpret_cast<f4 *>(wb + 4 * v) = *reinterpret_cast<const f4 *>(src + 4 * v);
        for (int32_t t = 4 * nvec + lane; t < total; t += 64)
            wb[t] = src[t];
    } else {
#pragma unroll 4
        for (int32_t t = lane; t < total; t += 64)
            wb[t] = src[t];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane >= nq)
        return;
    const float *pl = wb + lane * hw;
    float acc = 0.0f;
    for (int32_t p = 0; p < hw; ++p)
        acc += pl[p];
    y[q0 + lane] = acc * inv;
}

// Dense fully connected layer (the classifier the paper keeps dense, Sec. 3.1):
//   y[n, r] = act(b[r] + sum_c W[r, c] * x[n, c]),  W row-major [cout][cin].
// A dense product, so it runs on the matrix cores: a workgroup owns a tile of
// 16 images x 16 output rows (enough tiles to spread the classifier of a
// batch of 64 over the whole GPU), and its kLinWaves wavefronts split the
// input channels into equal chunks (a multiple of 16 each).  A wavefront
// accumulates its chunk with fp32 16x16x4 matrix instructions (lane l
// supplies image or row l % 16 and the k quarter l / 16); within each block
// of 16 channels, step s takes channels s, 4 + s, 8 + s and 12 + s, so a
// lane's four steps read 4 consecutive channels of its image and of its row:
// one 16-byte load each (VEC: cin a multiple of 4, x and W 16-byte aligned;
// else element loads), all of a batch of blocks issued before its first
// matrix instruction.  The chunk sums are added in ascending chunk order
// through LDS, then the bias, then the activation.  Images and rows past the
// end read the last one and are not stored.
constexpr int kLinWaves = 8;
constexpr int kLinBatch = 4;  // blocks of 16 channels loaded together

template <bool VEC>
__global__ void __launch_bounds__(64 * kLinWaves)
linear_kernel(const float *__restrict__ x, const float *__restrict__ wt, const float *__restrict__ bias,
              float *__restrict__ y, int32_t n, int32_t cin, int32_t cout, int32_t act) {
    __shared__ float part[kLinWaves * 4 * 64];  // each wavefront's 16 x 16 accumulator tile
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int i = lane & 15, kq = lane >> 4;
    const int32_t img = min(static_cast<int32_t>(blockIdx.y) * 16 + i, n - 1);
    const int32_t row = min(static_cast<int32_t>(blockIdx.x) * 16 + i, cout - 1);
    const float *xr = x + static_cast<int64_t>(img) * cin;
    const float *wr = wt + static_cast<int64_t>(row) * cin;
    // this thread's output after the reduction (threads 0 .. 255): register
    // r = t / 64 of lane l = t % 64 holds image 4 (l / 16) + r and row l % 16
    // of the tile; its bias is loaded now, off the critical path
    const int t = threadIdx.x;
    const int r_out = (t >> 6) & 3, l_out = t & 63;
    const int32_t oi = static_cast<int32_t>(blockIdx.y) * 16 + 4 * (l_out >> 4) + r_out;
    const int32_t oj = static_cast<int32_t>(blockIdx.x) * 16 + (l_out & 15);
    const float bo = bias && t < 256 ? bias[min(oj, cout - 1)] : 0.0f;
    const int32_t chunk = ((cin + kLinWaves - 1) / kLinWaves + 15) & ~15;
    const int32_t k_begin = wave * chunk;
    const int32_t k_end = min(cin, k_begin + chunk);
    f4 c = {0.f, 0.f, 0.f, 0.f};
    for (int32_t kbat = k_begin; kbat < k_end; kbat += 16 * kLinBatch) {
        float av[kLinBatch][4], bv[kLinBatch][4];
#pragma unroll
        for (int q = 0; q < kLinBatch; ++q) {
            const int32_t kb = kbat + 16 * q + 4 * kq;  // this lane's 4 channels of block q
            if constexpr (VEC) {
                // cin and the chunk bounds are multiples of 4: the 4 channels are all in or all out
                const bool in = kb < k_end;
                const f4 xa = in ? *reinterpret_cast<const f4 *>(xr + kb) : f4{0.f, 0.f, 0.f, 0.f};
                const f4 wb = in ? *reinterpret_cast<const f4 *>(wr + kb) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    av[q][e] = xa[e];
                    bv[q][e] = wb[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool in = kb + e < k_end;
                    av[q][e] = in ? xr[kb + e] : 0.0f;
                    bv[q][e] = in ? wr[kb + e] : 0.0f;
                }
            }
        }
#pragma unroll
        for (int q = 0; q < kLinBatch; ++q)
#pragma unroll
            for (int sstep = 0; sstep < 4; ++sstep)
                c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[q][sstep], bv[q][sstep], c, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
        part[(wave * 4 + r) * 64 + lane] = c[r];
    __syncthreads();
    if (t >= 256)
        return;
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < kLinWaves; ++w)
        sum += part[(w * 4 + r_out) * 64 + l_out];
    if (oi < n && oj < cout)
        y[static_cast<int64_t>(oi) * cout + oj] = clamp_act(sum + bo, act);
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
// depthwise kernel: output rows per group, wavefronts wanted per launch
constexpr int kDwRows = 4;
constexpr int64_t kDwWaves = 8192;

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
    // (a wavefront's planes stay below 2^30 bytes)
    const int64_t pbytes = static_cast<int64_t>(h) * w * 4;
    if (pbytes >= (int64_t{1} << 30))
        return hipErrorInvalidValue;
    // widest lane vector the shape and pointers allow, with whole planes in
    // a wavefront
    const uintptr_t align = reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y);
    int32_t vw = 1;
    for (int32_t v : {4, 2}) {
        if (w % (stride * v) == 0 && align % (4 * v) == 0 && wo / v <= 64) {
            vw = v;
            break;
        }
    }
    const int32_t lcols = wo / vw;
    const bool vec = lcols <= 64;
    const int32_t ppw =
        vec ? static_cast<int32_t>(std::min<int64_t>(64 / lcols, ((int64_t{1} << 30) - 1) / pbytes)) : 0;
    const int32_t wpp = vec ? 0 : (wo + 63) / 64;
    const int64_t units = vec ? (planes + ppw - 1) / ppw : planes * wpp;
    // row segments: about two wavefronts per SIMD slot (8 per SIMD of 256
    // compute units), a whole number of row groups each
    const int32_t rows = vec && stride == 2 && vw == 4 ? 2 : kDwRows;
    const int32_t groups = (ho + rows - 1) / rows;
    const int32_t want = static_cast<int32_t>(std::min<int64_t>(groups, (kDwWaves + units - 1) / units));
    const int32_t seg_rows = (groups + want - 1) / want * rows;
    const int32_t segs = (ho + seg_rows - 1) / seg_rows;
    const int64_t waves = units * segs;
    if (waves >= INT32_MAX - 3)
        return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>((waves + 3) / 4));
    if (vec) {
        using Fn = void (*)(const float *, const float *, const float *, float *, int64_t, int32_t, int32_t, int32_t,
                            int32_t, int32_t, int32_t, int32_t, int32_t, int32_t);
        Fn kern = stride == 1 ? (vw == 4 ? dw3x3_vec_kernel<1, 4> : vw == 2 ? dw3x3_vec_kernel<1, 2> : dw3x3_vec_kernel<1, 1>)
                              : (vw == 4 ? dw3x3_vec_kernel<2, 4> : vw == 2 ? dw3x3_vec_kernel<2, 2> : dw3x3_vec_kernel<2, 1>);
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, x, k, bias, y, planes, c, h, w, ho, wo, act, ppw,
                           segs, seg_rows);
    } else {
        auto kern = stride == 1 ? dw3x3_cols_kernel<1, kDwRows> : dw3x3_cols_kernel<2, kDwRows>;
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, x, k, bias, y, planes, c, h, w, ho, wo, act, wpp,
                           segs, seg_rows);
    }
    return hipGetLastError();
}

hipError_t launch_linear(const float *x, const float *wt, const float *bias, float *y, int32_t n, int32_t cin,
                         int32_t cout, int32_t act, hipStream_t stream) {
    const bool vec = cin % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(wt) % 16 == 0;
    const dim3 grid(static_cast<unsigned>((cout + 15) / 16), static_cast<unsigned>((n + 15) / 16));
    if (vec)
        hipLaunchKernelGGL(linear_kernel<true>, grid, dim3(64 * kLinWaves), 0, stream, x, wt, bias, y, n, cin, cout,
                           act);
    else
        hipLaunchKernelGGL(linear_kernel<false>, grid, dim3(64 * kLinWaves), 0, stream, x, wt, bias, y, n, cin,
                           cout, act);
    return hipGetLastError();
}

hipError_t launch_gap(const float *x, float *y, int32_t n, int32_t c, int64_t hw, hipStream_t stream) {
    const int64_t planes = static_cast<int64_t>(n) * c;
    if (hw <= kGapMaxHw) {
        const bool vec = reinterpret_cast<uintptr_t>(x) % 16 == 0;  // every group starts 64 hw bytes in
        const unsigned gblocks = static_cast<unsigned>((planes + 4 * kGapPlanes - 1) / (4 * kGapPlanes));
        const size_t lds = static_cast<size_t>(4 * kGapPlanes) * hw * sizeof(float);
        if (vec)
            hipLaunchKernelGGL(gap_staged_kernel<true>, dim3(gblocks), dim3(256), lds, stream, x, y, planes,
                               static_cast<int32_t>(hw), 1.0f / static_cast<float>(hw));
        else
            hipLaunchKernelGGL(gap_staged_kernel<false>, dim3(gblocks), dim3(256), lds, stream, x, y, planes,
                               static_cast<int32_t>(hw), 1.0f / static_cast<float>(hw));
        return hipGetLastError();
    }
    const int64_t blocks = (planes + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(gap_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream, x, y, planes,
                       hw, 1.0f / static_cast<float>(hw));
    return hipGetLastError();
}

}  // namespace spconv
