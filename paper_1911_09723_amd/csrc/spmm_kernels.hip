// gfx950 (CDNA4) kernels for the sparse 1x1 convolution
//     Y[n, r, p] = act(b[r] + sum_c W[r, c] * X[n, c, p])
// (Fast Sparse ConvNets, Sec. 3.2 / Fig. 2), over NCHW tensors.
//
// Columns.  The product's dense operand has Cin rows and N*H*W columns; column
// j is (image j / HW, position j % HW).  A workgroup owns one tile of
// `TC` consecutive columns.  Within a wavefront, lanes are split into
// `RPW = 64 / G` groups of G lanes; a group works on one (block) row and each
// lane accumulates Q = 16 / sizeof(element) consecutive columns, so a group
// covers the whole tile and every X access of a lane is one 16-byte vector.
// This is the paper's first insight (Sec. 3.2: the activations are dense, so
// load them as vectors along H*W) mapped onto wave64 lanes.
//
// Strip kernel.  The paper's second and third insights (Sec. 3.2, Fig. 3:
// walk output rows in the inner loop while one strip of spatial columns stays
// in the near cache) become: the workgroup copies the strip X[:, tile]
// (Cin x TC elements, <= 160 KiB) from HBM into LDS once, coalesced, and then
// every wavefront walks its rows reading X only from LDS.  Each nonzero costs
// one address computation, one 16-byte LDS read and Q * K FMAs per lane; with
// 1xK output blocks (Sec. 3.2: K rows share the pattern) the same X vector
// feeds K rows from registers.
//
// Direct kernel.  When Cin * TC does not fit in LDS, the same loop reads X
// straight from global memory (L1/L2).
//
// Weights.  Rows are packed by the host planner (planner.hpp) into bundles of
// RPW rows with a common padded length; a lane group loads the next four
// channel indices of its row with one 16-byte load and the weights with one
// (K = 1) or four (K = 4) 16-byte loads.  Accumulation is fp32 with FMA, in
// ascending input-channel order, starting from zero; the bias is added after
// the sum, then the activation, then one round-to-nearest-even conversion to
// the storage type.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "launch.hpp"

namespace spconv {
namespace {

template <bool F16>
struct Elem;
template <>
struct Elem<false> {
    using T = float;
    static __device__ __forceinline__ float to_f32(float v) { return v; }
    static __device__ __forceinline__ float from_f32(float v) { return v; }
};
template <>
struct Elem<true> {
    using T = _Float16;
    static __device__ __forceinline__ float to_f32(_Float16 v) { return static_cast<float>(v); }
    static __device__ __forceinline__ _Float16 from_f32(float v) { return static_cast<_Float16>(v); }
};

// Columns of one lane: Q consecutive flattened columns starting at j.
template <int Q>
struct LaneCols {
    int64_t j;       // first column
    int64_t img;     // image of the first column (vector path)
    int32_t pos;     // spatial position of the first column (vector path)
    bool full;       // all Q columns exist
};

template <int Q>
__device__ __forceinline__ LaneCols<Q> lane_cols(int64_t j, int64_t m, int32_t hw) {
    LaneCols<Q> lc;
    lc.j = j;
    lc.img = j / hw;
    lc.pos = static_cast<int32_t>(j - lc.img * hw);
    lc.full = j + Q <= m;
    return lc;
}

// Element offset of column e of a lane into an NCHW tensor with `ch` channels
// (channel 0); -1 if the column is past the end.
template <int Q>
__device__ __forceinline__ int64_t col_offset(const LaneCols<Q> &lc, int e, int64_t m, int32_t hw,
                                              int32_t ch) {
    const int64_t j = lc.j + e;
    if (j >= m)
        return -1;
    const int64_t img = j / hw;
    const int64_t p = j - img * hw;
    return img * ch * hw + p;
}

template <int G, int K, bool F16, bool STRIP>
__global__ void __launch_bounds__(1024)
spmm_kernel(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
            const float *__restrict__ val, const int4 *__restrict__ hdr, const int32_t *__restrict__ rows,
            const int32_t *__restrict__ wave_ptr, const float *__restrict__ bias, int32_t cin,
            int32_t cout, int32_t hw, int64_t m, int32_t act, int32_t vec) {
    using T = typename Elem<F16>::T;
    constexpr int E = sizeof(T);
    constexpr int Q = 16 / E;       // columns per lane
    constexpr int TC = G * Q;       // columns per tile
    constexpr int RPW = 64 / G;     // rows (lane groups) per wavefront
    constexpr int ROWB = G * 16;    // bytes of one strip row in LDS

    extern __shared__ __align__(16) unsigned char lds[];
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);

    const int tid = threadIdx.x;
    const int64_t j0 = static_cast<int64_t>(blockIdx.x) * TC;
    const int lane = tid & 63;
    const int g = lane / G;
    const int li = lane % G;

    if constexpr (STRIP) {
        // Stage X[:, j0 : j0 + TC] into LDS as [cin][TC]: thread (c, i) copies
        // the 16 bytes of columns j0 + i*Q .. + Q-1 of channel c.
        const int si = tid % G;
        const int cstep = static_cast<int>(blockDim.x) / G;
        const LaneCols<Q> lc = lane_cols<Q>(j0 + static_cast<int64_t>(si) * Q, m, hw);
        if (vec && lc.full) {
            const T *src = x + (lc.img * cin) * hw + lc.pos;
            for (int c = tid / G; c < cin; c += cstep)
                *reinterpret_cast<uint4 *>(lds + c * ROWB + si * 16) =
                    *reinterpret_cast<const uint4 *>(src + static_cast<int64_t>(c) * hw);
        } else {
            int64_t off[Q];
#pragma unroll
            for (int e = 0; e < Q; ++e)
                off[e] = col_offset<Q>(lc, e, m, hw, cin);
            for (int c = tid / G; c < cin; c += cstep) {
                T v[Q];
#pragma unroll
                for (int e = 0; e < Q; ++e)
                    v[e] = off[e] >= 0 ? x[off[e] + static_cast<int64_t>(c) * hw] : T(0);
                *reinterpret_cast<uint4 *>(lds + c * ROWB + si * 16) = *reinterpret_cast<const uint4 *>(v);
            }
        }
        __syncthreads();
    }

    const LaneCols<Q> lc = lane_cols<Q>(j0 + static_cast<int64_t>(li) * Q, m, hw);
    const bool lane_vec = vec && lc.full;
    int64_t xoff[Q];
    if constexpr (!STRIP) {
#pragma unroll
        for (int e = 0; e < Q; ++e)
            xoff[e] = col_offset<Q>(lc, e, m, hw, cin);
    }

    // X values (as fp32) of channel c for this lane's Q columns.
    auto load_x = [&](int32_t c, float (&xf)[Q]) {
        if constexpr (STRIP) {
            const uint4 raw = *reinterpret_cast<const uint4 *>(lds + c * ROWB + li * 16);
            const T *v = reinterpret_cast<const T *>(&raw);
#pragma unroll
            for (int e = 0; e < Q; ++e)
                xf[e] = Elem<F16>::to_f32(v[e]);
        } else {
            if (lane_vec) {
                const uint4 raw = *reinterpret_cast<const uint4 *>(
                    x + (lc.img * cin + c) * static_cast<int64_t>(hw) + lc.pos);
                const T *v = reinterpret_cast<const T *>(&raw);
#pragma unroll
                for (int e = 0; e < Q; ++e)
                    xf[e] = Elem<F16>::to_f32(v[e]);
            } else {
#pragma unroll
                for (int e = 0; e < Q; ++e)
                    xf[e] = xoff[e] >= 0 ? Elem<F16>::to_f32(x[xoff[e] + static_cast<int64_t>(c) * hw]) : 0.0f;
            }
        }
    };

    // wavefront index, uniform across the wave: bundle headers and loop
    // bounds then live in scalar registers
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int bbeg = wave_ptr[wave];
    const int bend = wave_ptr[wave + 1];
    for (int b = bbeg; b < bend; ++b) {
        const int4 h = hdr[b];
        float acc[K][Q];
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int e = 0; e < Q; ++e)
                acc[kk][e] = 0.0f;

        // main part: four slots per step
        const int32_t *ip = idx + h.x + g * 4;
        const float *vp = val + static_cast<int64_t>(h.x + g * 4) * K;
        for (int t = 0; t < h.y; t += 4) {
            const int4 c4 = *reinterpret_cast<const int4 *>(ip);
            float w[4][K];
            if constexpr (K == 1) {
                const float4 w4 = *reinterpret_cast<const float4 *>(vp);
                w[0][0] = w4.x;
                w[1][0] = w4.y;
                w[2][0] = w4.z;
                w[3][0] = w4.w;
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float4 w4 = *reinterpret_cast<const float4 *>(vp + u * K);
                    w[u][0] = w4.x;
                    w[u][1] = w4.y;
                    w[u][2] = w4.z;
                    w[u][3] = w4.w;
                }
            }
            const int32_t cs[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float xf[Q];
                load_x(cs[u], xf);
#pragma unroll
                for (int kk = 0; kk < K; ++kk)
#pragma unroll
                    for (int e = 0; e < Q; ++e)
                        acc[kk][e] = __builtin_fmaf(w[u][kk], xf[e], acc[kk][e]);
            }
            ip += RPW * 4;
            vp += RPW * 4 * K;
        }
        // tail: one slot per step
        ip = idx + h.x + h.y * RPW + g;
        vp = val + static_cast<int64_t>(h.x + h.y * RPW + g) * K;
        for (int t = 0; t < h.z; ++t) {
            const int32_t c = *ip;
            float w[K];
            if constexpr (K == 1) {
                w[0] = *vp;
            } else {
                const float4 w4 = *reinterpret_cast<const float4 *>(vp);
                w[0] = w4.x;
                w[1] = w4.y;
                w[2] = w4.z;
                w[3] = w4.w;
            }
            float xf[Q];
            load_x(c, xf);
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
#pragma unroll
                for (int e = 0; e < Q; ++e)
                    acc[kk][e] = __builtin_fmaf(w[kk], xf[e], acc[kk][e]);
            ip += RPW;
            vp += RPW * K;
        }

        // epilogue: bias, activation, one rounding, store
        const int rb = rows[b * RPW + g];
        if (rb < 0 || lc.j >= m)
            continue;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) {
            const int r = rb * K + kk;
            const float bv = bias[r];
            T out[Q];
#pragma unroll
            for (int e = 0; e < Q; ++e) {
                float v = acc[kk][e] + bv;
                if (act == 1)
                    v = fmaxf(v, 0.0f);
                else if (act == 2)
                    v = fminf(fmaxf(v, 0.0f), 6.0f);
                out[e] = Elem<F16>::from_f32(v);
            }
            if (lane_vec) {
                *reinterpret_cast<uint4 *>(y + (lc.img * cout + r) * static_cast<int64_t>(hw) + lc.pos) =
                    *reinterpret_cast<const uint4 *>(out);
            } else {
#pragma unroll
                for (int e = 0; e < Q; ++e) {
                    const int64_t o = col_offset<Q>(lc, e, m, hw, cout);
                    if (o >= 0)
                        y[o + static_cast<int64_t>(r) * hw] = out[e];
                }
            }
        }
    }
}

template <int G, int K, bool F16, bool STRIP>
hipError_t launch_one(const DevicePlan &p, const void *x, void *y, int64_t m, int32_t hw, int32_t vec,
                      hipStream_t stream) {
    constexpr int Q = 16 / (F16 ? 2 : 4);
    constexpr int TC = G * Q;
    auto kern = spmm_kernel<G, K, F16, STRIP>;
    const int lds = STRIP ? p.lds_bytes : 0;
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        if (e != hipSuccess)
            return e;
    }
    const int64_t tiles = (m + TC - 1) / TC;
    dim3 grid(static_cast<unsigned>(tiles));
    dim3 block(static_cast<unsigned>(p.waves * 64));
    hipLaunchKernelGGL(kern, grid, block, lds, stream, x, y, p.idx, p.val,
                       reinterpret_cast<const int4 *>(p.hdr), p.rows, p.wave_ptr, p.bias, p.cin, p.cout, hw, m,
                       p.act, vec);
    return hipGetLastError();
}

template <int K, bool F16, bool STRIP>
hipError_t dispatch_g(const DevicePlan &p, const void *x, void *y, int64_t m, int32_t hw, int32_t vec,
                      hipStream_t s) {
    switch (p.lanes_per_row) {
    case 8:
        return launch_one<8, K, F16, STRIP>(p, x, y, m, hw, vec, s);
    case 16:
        return launch_one<16, K, F16, STRIP>(p, x, y, m, hw, vec, s);
    case 32:
        return launch_one<32, K, F16, STRIP>(p, x, y, m, hw, vec, s);
    case 64:
        return launch_one<64, K, F16, STRIP>(p, x, y, m, hw, vec, s);
    default:
        return hipErrorInvalidValue;
    }
}

template <bool F16, bool STRIP>
hipError_t dispatch_k(const DevicePlan &p, const void *x, void *y, int64_t m, int32_t hw, int32_t vec,
                      hipStream_t s) {
    return p.k == 4 ? dispatch_g<4, F16, STRIP>(p, x, y, m, hw, vec, s)
                    : dispatch_g<1, F16, STRIP>(p, x, y, m, hw, vec, s);
}

}  // namespace

hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int64_t m, int32_t hw, int32_t vec,
                       hipStream_t stream) {
    const bool strip = p.kernel == KERNEL_STRIP;
    if (p.storage == 1)
        return strip ? dispatch_k<true, true>(p, x, y, m, hw, vec, stream)
                     : dispatch_k<true, false>(p, x, y, m, hw, vec, stream);
    return strip ? dispatch_k<false, true>(p, x, y, m, hw, vec, stream)
                 : dispatch_k<false, false>(p, x, y, m, hw, vec, stream);
}

}  // namespace spconv
