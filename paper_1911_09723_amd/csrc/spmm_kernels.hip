// gfx950 (CDNA4) kernels for the sparse 1x1 convolution
//     Y[n, r, p] = act(b[r] + sum_c W[r, c] * X[n, c, p])
// (Fast Sparse ConvNets, Sec. 3.2 / Fig. 2), over NCHW tensors.
//
// Columns.  The product's dense operand has Cin rows and N*H*W columns; column
// j is (image j / HW, position j % HW).  A workgroup owns one tile of TC
// consecutive columns at a time.  Within a wavefront, lanes are split into
// RPW = 64 / G groups of G lanes; a group works on one (block) row, and each
// lane accumulates Q columns, read as NV 16-byte vectors per nonzero.  This
// is the paper's first insight (Sec. 3.2: the activations are dense, so load
// them as vectors along H*W) mapped onto wave64 lanes.
//
// Strip kernel.  The second and third insights (Sec. 3.2, Fig. 3: walk the
// output rows in the inner loop while one strip of spatial columns stays in
// the near cache, and prefetch the next strip) become:
//   * the strip X[:, tile] (Cin x TC elements) sits in LDS and compute
//     wavefronts walk their rows reading X only from there -- each nonzero
//     costs one address computation, NV 16-byte LDS reads and
//     NV * (16 / element size) * K FMAs per lane; with 1xK output blocks
//     (Sec. 3.2) one X vector feeds K rows from registers;
//   * loader wavefronts fetch the NEXT tile's strip from HBM into their
//     registers while the compute wavefronts work, and copy it into LDS
//     between two workgroup barriers (vector-memory operations of one
//     wavefront complete in order, so a compute wavefront that issued the
//     strip loads would stall its own weight loads behind them);
//   * workgroups are persistent: each walks tiles blockIdx.x, + gridDim.x, ...
//
// Weight streams.  The host planner (planner.hpp) packs each wavefront's rows
// into bundles of RPW rows stored back to back, so a wavefront reads one
// continuous stream of steps (4 slots per row).  The main loop is a software
// pipeline over that stream that does not stop at bundle boundaries: channel
// indices are fetched DI steps ahead, weights DW steps ahead, X vectors read
// from LDS DX steps ahead, and when the step just multiplied in is the last of
// its bundle (a flag bit in its first channel index) the bundle's results get
// bias, activation and one round-to-nearest-even conversion and are stored.
// Per-bundle rows and biases sit in LDS, copied there once per launch.  The
// weight loads are buffer loads whose scalar offset walks the stream, so no
// vector ALU goes to weight addressing.  Accumulation is fp32 FMA in ascending
// input-channel order from zero; the bias is added after the sum.
//
// Direct kernel.  When Cin * TC does not fit in LDS, a simpler loop reads X
// straight from global memory (L1/L2), one tile and one bundle at a time.
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

// ---------------------------------------------------------------------------
// Buffer loads: 128-bit buffer resource (base, byte size) in scalar registers,
// a per-lane offset and a wavefront-uniform offset.  Reads past `bytes` return
// zero.  Word 3 is the gfx9-family raw-buffer configuration.
// ---------------------------------------------------------------------------
using Rsrc = __amdgpu_buffer_rsrc_t;

__device__ __forceinline__ Rsrc make_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}

__device__ __forceinline__ uint4 bload16(Rsrc r, int32_t voff, int32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ uint32_t bload4(Rsrc r, int32_t voff, int32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}

// X is read once and Y written once: stream them past the caches with
// non-temporal 16-byte accesses, so the weight stream that every workgroup
// re-reads keeps its place in L2.
typedef unsigned int V4U __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load16_stream(const void *p) {
    const V4U v = __builtin_nontemporal_load(static_cast<const V4U *>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ void store16_stream(void *p, const uint4 &u) {
    V4U v = {u.x, u.y, u.z, u.w};
    __builtin_nontemporal_store(v, static_cast<V4U *>(p));
}

// ---------------------------------------------------------------------------
// Column addressing in NCHW tensors
// ---------------------------------------------------------------------------

// Where QV consecutive flattened columns j .. j+QV-1 live: image and spatial
// position of column j, and whether all QV columns exist and sit in the same
// image (then they are contiguous in every channel).
struct ColPos {
    int32_t j;
    uint32_t img;
    int32_t p;
    bool whole;
};

template <int QV>
__device__ __forceinline__ ColPos col_pos(int32_t j, int32_t m, int32_t hw) {
    ColPos cp;
    cp.j = j;
    cp.img = static_cast<uint32_t>(j) / static_cast<uint32_t>(hw);
    cp.p = j - static_cast<int32_t>(cp.img) * hw;
    cp.whole = j + QV <= m && cp.p + QV <= hw;
    return cp;
}

// Read the QV columns of `cp` in channel c (of `ch`) into a 16-byte vector.
// `vec` promises 16-byte alignment of every whole run (HW a multiple of QV and
// a 16-byte aligned tensor); other whole runs are read element by element from
// one base address; runs that cross an image or the end are gathered with
// bounds checks (zeros past the end).
template <typename T, int QV>
__device__ __forceinline__ uint4 gather16(const T *__restrict__ x, const ColPos &cp, int32_t m, int32_t hw,
                                          int32_t ch, int32_t c, bool vec) {
    if (cp.whole) {
        const T *src = x + (static_cast<int64_t>(cp.img) * ch + c) * hw + cp.p;
        if (vec)
            return load16_stream(src);
        T v[QV];
#pragma unroll
        for (int e = 0; e < QV; ++e)
            v[e] = src[e];
        return *reinterpret_cast<const uint4 *>(v);
    }
    T v[QV];
#pragma unroll
    for (int e = 0; e < QV; ++e) {
        const int32_t jj = cp.j + e;
        v[e] = T(0);
        if (jj < m) {
            const uint32_t img = static_cast<uint32_t>(jj) / static_cast<uint32_t>(hw);
            const int32_t p = jj - static_cast<int32_t>(img) * hw;
            v[e] = x[(static_cast<int64_t>(img) * ch + c) * hw + p];
        }
    }
    return *reinterpret_cast<const uint4 *>(v);
}

// Store QV columns of `cp` in output channel r (of `ch`); same cases as gather16.
template <typename T, int QV>
__device__ __forceinline__ void scatter16(T *__restrict__ y, const ColPos &cp, int32_t m, int32_t hw, int32_t ch,
                                          int32_t r, bool vec, const T (&out)[QV]) {
    if (cp.whole) {
        T *dst = y + (static_cast<int64_t>(cp.img) * ch + r) * hw + cp.p;
        if (vec) {
            store16_stream(dst, *reinterpret_cast<const uint4 *>(out));
        } else {
#pragma unroll
            for (int e = 0; e < QV; ++e)
                dst[e] = out[e];
        }
        return;
    }
#pragma unroll
    for (int e = 0; e < QV; ++e) {
        const int32_t jj = cp.j + e;
        if (jj < m) {
            const uint32_t img = static_cast<uint32_t>(jj) / static_cast<uint32_t>(hw);
            const int32_t p = jj - static_cast<int32_t>(img) * hw;
            y[(static_cast<int64_t>(img) * ch + r) * hw + p] = out[e];
        }
    }
}

__device__ __forceinline__ float activate(float v, int act) {
    if (act == 1)
        return fmaxf(v, 0.0f);
    if (act == 2)
        return fminf(fmaxf(v, 0.0f), 6.0f);
    return v;
}

// ---------------------------------------------------------------------------
// Weight stream
// ---------------------------------------------------------------------------

// Channel indices of one step (for one lane group), and its weights.
struct Idx4 {
    int32_t c[4];
};
template <int K>
struct W4 {
    float w[4][K];
};

// Load the step whose first slot is `slot0` (a multiple of 4; lane group g
// reads slots slot0 + 4g .. + 3).  `lo` is this lane's byte offset 16 * g.
__device__ __forceinline__ Idx4 load_idx(Rsrc ri, int32_t lo, int32_t slot0) {
    const uint4 c4 = bload16(ri, lo, slot0 * 4);
    return Idx4{{static_cast<int32_t>(c4.x), static_cast<int32_t>(c4.y), static_cast<int32_t>(c4.z),
                 static_cast<int32_t>(c4.w)}};
}

template <int K>
__device__ __forceinline__ W4<K> load_w(Rsrc rv, int32_t lo, int32_t slot0) {
    W4<K> s;
    if constexpr (K == 1) {
        const uint4 w4 = bload16(rv, lo, slot0 * 4);
        s.w[0][0] = __uint_as_float(w4.x);
        s.w[1][0] = __uint_as_float(w4.y);
        s.w[2][0] = __uint_as_float(w4.z);
        s.w[3][0] = __uint_as_float(w4.w);
    } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint4 w4 = bload16(rv, lo * K + u * 16, slot0 * 4 * K);
            s.w[u][0] = __uint_as_float(w4.x);
            s.w[u][1] = __uint_as_float(w4.y);
            s.w[u][2] = __uint_as_float(w4.z);
            s.w[u][3] = __uint_as_float(w4.w);
        }
    }
    return s;
}

constexpr int gcd_i(int a, int b) { return b ? gcd_i(b, a % b) : a; }
constexpr int lcm_i(int a, int b) { return a / gcd_i(a, b) * b; }

// Pipeline depths (in steps) of the main loop: channel indices DI ahead of
// their multiply, weights DW ahead, LDS reads DX ahead.  Deeper rings hide
// more latency but cost registers.
template <int K, bool F16, int NV>
struct PipeDepth {
    // Unstructured fp32 rows need an LDS read per FMA, so their X vectors are
    // read a step ahead; 1x4 blocks and fp16 rows read them in the step that
    // uses them and spend the registers on wider accumulators instead.
    static constexpr bool kAheadX = K == 1 && !F16;
    static constexpr int DI = 3;
    static constexpr int DW = (kAheadX && NV == 1) ? 3 : 1;
    static constexpr int DX = kAheadX ? 1 : 0;
    static constexpr int P = lcm_i(lcm_i(DI + 1, DW + 1), DX + 1);
    static_assert(DI <= kLookaheadSteps && DW <= kLookaheadSteps, "planner padding too small");
};

// ---------------------------------------------------------------------------
// Strip kernel
// ---------------------------------------------------------------------------

constexpr int kLoaderVecs = 16;  // 16-byte strip vectors one loader lane holds

template <int G, int NV, int K, bool F16>
__global__ void __launch_bounds__(1024)
spmm_strip(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
           const float *__restrict__ val, const int4 *__restrict__ hdr, const int32_t *__restrict__ meta,
           const int32_t *__restrict__ wave_ptr, int32_t cin, int32_t cout, int32_t hw, int32_t m, int32_t act,
           int32_t vec, int32_t cwaves, int32_t idx_bytes, int32_t val_bytes, int32_t strip_bytes,
           int32_t meta_words, int32_t nbundles) {
    using T = typename Elem<F16>::T;
    constexpr int E = sizeof(T);
    constexpr int QV = 16 / E;        // columns per 16-byte vector
    constexpr int Q = NV * QV;        // columns per lane
    constexpr int TC = G * Q;         // columns per tile
    constexpr int RPW = 64 / G;       // rows (lane groups) per wavefront
    constexpr int ROWB = G * NV * 16; // bytes of one strip row in LDS
    constexpr int CPR = G * NV;       // 16-byte vectors per strip row
    static_assert(64 % CPR == 0, "a loader lane must keep one column vector");

    extern __shared__ __align__(16) unsigned char lds[];
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tiles = (m + TC - 1) / TC;
    int tile = blockIdx.x;
    if (tile >= tiles)
        return;  // the whole workgroup leaves: no barrier is skipped by part of it

    if (wave >= cwaves) {
        // ----- loader wavefront -----
        const int nl = static_cast<int>(blockDim.x >> 6) - cwaves;
        const int ll = (wave - cwaves) * 64 + lane;
        const int cc = ll % CPR;            // which 16-byte vector of a strip row
        const int c0 = ll / CPR;            // first channel
        const int cstep = nl * 64 / CPR;    // channel stride between this lane's vectors
        uint4 pf[kLoaderVecs];
        auto fetch = [&](int t) {
            const ColPos cp = col_pos<QV>(t * TC + cc * QV, m, hw);
#pragma unroll
            for (int i = 0; i < kLoaderVecs; ++i) {
                const int c = c0 + i * cstep;
                if (c < cin)
                    pf[i] = gather16<T, QV>(x, cp, m, hw, cin, c, vec != 0);
            }
        };
        auto deposit = [&]() {
#pragma unroll
            for (int i = 0; i < kLoaderVecs; ++i) {
                const int c = c0 + i * cstep;
                if (c < cin)
                    *reinterpret_cast<uint4 *>(lds + c * ROWB + cc * 16) = pf[i];
            }
        };
        fetch(tile);
        deposit();
        __syncthreads();  // strip(tile) ready
        for (;;) {
            const int next = tile + gridDim.x;
            if (next < tiles)
                fetch(next);
            __syncthreads();  // compute wavefronts done with strip(tile)
            if (next >= tiles)
                break;
            deposit();
            __syncthreads();  // strip(next) ready
            tile = next;
        }
        return;
    }

    // ----- compute wavefront -----
    const int g = lane / G;
    const int li = lane % G;
    const int32_t lo = g * 16;  // byte offset of this lane group's 4-slot chunk in a step
    int32_t *meta_lds = reinterpret_cast<int32_t *>(lds + strip_bytes);
    const float *bias_lds = reinterpret_cast<const float *>(meta_lds + nbundles * RPW);

    // Without loader wavefronts, every wavefront copies strips between tiles.
    const bool self_load = static_cast<int>(blockDim.x >> 6) == cwaves;
    auto copy_strip = [&](int t) {
        const int cc = tid % CPR;
        const int cstep = static_cast<int>(blockDim.x) / CPR;
        const ColPos cp = col_pos<QV>(t * TC + cc * QV, m, hw);
        int c = tid / CPR;
        for (; c + 3 * cstep < cin; c += 4 * cstep) {
            uint4 v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] = gather16<T, QV>(x, cp, m, hw, cin, c + i * cstep, vec != 0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *reinterpret_cast<uint4 *>(lds + (c + i * cstep) * ROWB + cc * 16) = v[i];
        }
        for (; c < cin; c += cstep)
            *reinterpret_cast<uint4 *>(lds + c * ROWB + cc * 16) = gather16<T, QV>(x, cp, m, hw, cin, c, vec != 0);
    };

    // LDS byte offset of each of the lane's vectors within a strip row, and
    // the first column of each vector within the tile.
    int32_t voff[NV], vcol[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        voff[v] = v * (ROWB / NV) + li * 16;
        vcol[v] = v * (TC / NV) + li * QV;
    }
    const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(idx_bytes));
    const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(val_bytes));
    const int bbeg = wave_ptr[wave];
    const int bend = wave_ptr[wave + 1];
    // this wavefront's continuous stream: first slot and number of steps
    constexpr int SS = RPW * 4;  // slots per step
    int32_t sbase = 0, nsteps = 0;
    if (bend > bbeg) {
        const int4 h0 = hdr[bbeg];
        const int4 h1 = hdr[bend - 1];
        sbase = h0.x;
        nsteps = (h1.x + h1.y * SS - h0.x) / SS;
    }

    // per-bundle rows and biases into LDS (once per launch)
    for (int i = tid; i < meta_words; i += cwaves * 64)
        meta_lds[i] = meta[i];
    if (self_load)
        copy_strip(tile);
    __syncthreads();  // strip(tile) and the bundle table ready

    using PC = PipeDepth<K, F16, NV>;
    constexpr int DI = PC::DI, DW = PC::DW, DX = PC::DX, P = PC::P;
    struct XStep {
        uint4 raw[4][NV];
    };

    for (;;) {
        const int32_t j0 = tile * TC;
        ColPos cps[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v)
            cps[v] = col_pos<QV>(j0 + vcol[v], m, hw);

        float acc[K][Q];
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int e = 0; e < Q; ++e)
                acc[kk][e] = 0.0f;

        // the bundle in progress and its rows / biases (from LDS)
        int b = bbeg;
        int rb = -1;
        float bv[K];
        auto load_meta = [&](int bb) {
            const int mi = bb * RPW + g;
            rb = meta_lds[mi];
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
                bv[kk] = bias_lds[mi * K + kk];
        };
        if (b < bend)
            load_meta(b);

        auto read_x = [&](const Idx4 &ci, XStep &xs) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                // the flag bit of a channel index shifts out of the 32-bit offset
                const uint32_t base = static_cast<uint32_t>(ci.c[u]) * ROWB;
#pragma unroll
                for (int v = 0; v < NV; ++v)
                    xs.raw[u][v] = *reinterpret_cast<const uint4 *>(lds + base + voff[v]);
            }
        };
        auto fma_step = [&](const XStep &xs, const W4<K> &ws) {
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < NV; ++v) {
                    const T *xe = reinterpret_cast<const T *>(&xs.raw[u][v]);
#pragma unroll
                    for (int e = 0; e < QV; ++e) {
                        const float xf = Elem<F16>::to_f32(xe[e]);
#pragma unroll
                        for (int kk = 0; kk < K; ++kk)
                            acc[kk][v * QV + e] = __builtin_fmaf(ws.w[u][kk], xf, acc[kk][v * QV + e]);
                    }
                }
        };
        // bias, activation, one rounding, store; then start the next bundle
        auto finish_bundle = [&]() {
            if (rb >= 0) {
#pragma unroll
                for (int v = 0; v < NV; ++v) {
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) {
                        T out[QV];
#pragma unroll
                        for (int e = 0; e < QV; ++e)
                            out[e] = Elem<F16>::from_f32(activate(acc[kk][v * QV + e] + bv[kk], act));
                        scatter16<T, QV>(y, cps[v], m, hw, cout, rb * K + kk, vec != 0, out);
                    }
                }
            }
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
#pragma unroll
                for (int e = 0; e < Q; ++e)
                    acc[kk][e] = 0.0f;
            ++b;
            if (b < bend)
                load_meta(b);
        };

        // The pipeline: ring buffers indexed by step modulo their depth; the
        // stage loop is unrolled over P steps so every index is a constant.
        // Fetches past the stream's end read planner padding and are unused.
        Idx4 ci[DI + 1];
        W4<K> wv[DW + 1];
        XStep xr[DX + 1];
#pragma unroll
        for (int t = 0; t < DI; ++t)
            ci[t] = load_idx(ri, lo, sbase + t * SS);
#pragma unroll
        for (int t = 0; t < DW; ++t)
            wv[t] = load_w<K>(rv, lo, sbase + t * SS);
#pragma unroll
        for (int t = 0; t < DX; ++t)
            read_x(ci[t], xr[t]);
        auto stage = [&](int s, int k) {
            ci[(k + DI) % (DI + 1)] = load_idx(ri, lo, sbase + (s + DI) * SS);
            wv[(k + DW) % (DW + 1)] = load_w<K>(rv, lo, sbase + (s + DW) * SS);
            if constexpr (DX > 0)
                read_x(ci[(k + DX) % (DI + 1)], xr[(k + DX) % (DX + 1)]);
            else
                read_x(ci[k % (DI + 1)], xr[0]);
            __builtin_amdgcn_sched_barrier(0);
            fma_step(xr[k % (DX + 1)], wv[k % (DW + 1)]);
            if (__builtin_amdgcn_readfirstlane(ci[k % (DI + 1)].c[0]) & kLastStepFlag)
                finish_bundle();
        };
        int s0 = 0;
        // whole periods; a single-exit loop keeps its bounds in scalar registers
        for (const int np = nsteps - nsteps % P; s0 < np; s0 += P) {
#pragma unroll
            for (int k = 0; k < P; ++k)
                stage(s0 + k, k);
        }
#pragma unroll
        for (int k = 0; k < P - 1; ++k)
            if (s0 + k < nsteps)
                stage(s0 + k, k);

        const int next = tile + gridDim.x;
        __syncthreads();  // done with strip(tile)
        if (next >= tiles)
            break;
        if (self_load)
            copy_strip(next);
        __syncthreads();  // strip(next) ready
        tile = next;
    }
}

// ---------------------------------------------------------------------------
// Direct kernel: X read from global memory, one tile per workgroup.
// ---------------------------------------------------------------------------

template <int G, int K, bool F16>
__global__ void __launch_bounds__(1024)
spmm_direct(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
            const float *__restrict__ val, const int4 *__restrict__ hdr, const int32_t *__restrict__ meta,
            const int32_t *__restrict__ wave_ptr, int32_t cin, int32_t cout, int32_t hw, int32_t m, int32_t act,
            int32_t vec, int32_t idx_bytes, int32_t val_bytes, int32_t nbundles) {
    using T = typename Elem<F16>::T;
    constexpr int QV = 16 / sizeof(T);
    constexpr int TC = G * QV;
    constexpr int RPW = 64 / G;
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);
    const float *bias = reinterpret_cast<const float *>(meta + nbundles * RPW);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int g = lane / G;
    const int li = lane % G;
    const int32_t lo = g * 16;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ColPos cp = col_pos<QV>(static_cast<int32_t>(blockIdx.x) * TC + li * QV, m, hw);
    const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(idx_bytes));
    const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(val_bytes));

    for (int b = wave_ptr[wave]; b < wave_ptr[wave + 1]; ++b) {
        const int4 h = hdr[b];
        float acc[K][QV];
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int e = 0; e < QV; ++e)
                acc[kk][e] = 0.0f;
        for (int t = 0; t < h.y; ++t) {
            const Idx4 ci = load_idx(ri, lo, h.x + t * RPW * 4);
            const W4<K> ws = load_w<K>(rv, lo, h.x + t * RPW * 4);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint4 raw = gather16<T, QV>(x, cp, m, hw, cin, ci.c[u] & (kLastStepFlag - 1), vec != 0);
                const T *xe = reinterpret_cast<const T *>(&raw);
#pragma unroll
                for (int e = 0; e < QV; ++e) {
                    const float xf = Elem<F16>::to_f32(xe[e]);
#pragma unroll
                    for (int kk = 0; kk < K; ++kk)
                        acc[kk][e] = __builtin_fmaf(ws.w[u][kk], xf, acc[kk][e]);
                }
            }
        }
        const int rb = meta[b * RPW + g];
        if (rb < 0)
            continue;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) {
            const float bv = bias[(b * RPW + g) * K + kk];
            T out[QV];
#pragma unroll
            for (int e = 0; e < QV; ++e)
                out[e] = Elem<F16>::from_f32(activate(acc[kk][e] + bv, act));
            scatter16<T, QV>(y, cp, m, hw, cout, rb * K + kk, vec != 0, out);
        }
    }
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------

template <int G, int NV, int K, bool F16>
hipError_t prepare_strip(DevicePlan &p) {
    auto kern = spmm_strip<G, NV, K, F16>;
    const int threads = (p.waves + p.loader_waves) * 64;
    if (p.lds_bytes > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, p.lds_bytes);
        if (e != hipSuccess)
            return e;
    }
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, p.lds_bytes);
    if (e != hipSuccess)
        return e;
    if (per_cu < 1)
        return hipErrorInvalidConfiguration;
    p.blocks_per_cu = per_cu;
    return hipSuccess;
}

template <int G, int NV, int K, bool F16>
hipError_t launch_strip(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                        hipStream_t stream) {
    constexpr int TC = G * NV * 16 / (F16 ? 2 : 4);
    const int threads = (p.waves + p.loader_waves) * 64;
    const int64_t tiles = (static_cast<int64_t>(m) + TC - 1) / TC;
    const int64_t slots = static_cast<int64_t>(p.blocks_per_cu) * p.num_cus;
    if (slots < 1)
        return hipErrorInvalidConfiguration;
    const unsigned grid = static_cast<unsigned>(tiles < slots ? tiles : slots);
    hipLaunchKernelGGL((spmm_strip<G, NV, K, F16>), dim3(grid), dim3(threads), p.lds_bytes, stream, x, y, p.idx,
                       p.val, reinterpret_cast<const int4 *>(p.hdr), p.meta, p.wave_ptr, p.cin, p.cout, hw, m,
                       p.act, vec, p.waves, p.idx_bytes, p.val_bytes, p.strip_bytes, p.meta_words, p.nbundles);
    return hipGetLastError();
}

template <int G, int K, bool F16>
hipError_t launch_direct(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                         hipStream_t stream) {
    constexpr int TC = G * 16 / (F16 ? 2 : 4);
    const int64_t tiles = (static_cast<int64_t>(m) + TC - 1) / TC;
    hipLaunchKernelGGL((spmm_direct<G, K, F16>), dim3(static_cast<unsigned>(tiles)), dim3(p.waves * 64), 0,
                       stream, x, y, p.idx, p.val, reinterpret_cast<const int4 *>(p.hdr), p.meta, p.wave_ptr,
                       p.cin, p.cout, hw, m, p.act, vec, p.idx_bytes, p.val_bytes, p.nbundles);
    return hipGetLastError();
}

template <int K, bool F16>
hipError_t prepare(DevicePlan &p) {
    if (p.kernel == KERNEL_DIRECT)
        return hipSuccess;
    switch (p.lanes_per_row * 10 + p.vecs_per_lane) {
    case 81: return prepare_strip<8, 1, K, F16>(p);
    case 82: return prepare_strip<8, 2, K, F16>(p);
    case 161: return prepare_strip<16, 1, K, F16>(p);
    case 162: return prepare_strip<16, 2, K, F16>(p);
    case 321: return prepare_strip<32, 1, K, F16>(p);
    case 322: return prepare_strip<32, 2, K, F16>(p);
    case 641: return prepare_strip<64, 1, K, F16>(p);
    default: return hipErrorInvalidValue;
    }
}

template <int K, bool F16>
hipError_t dispatch(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                    hipStream_t s) {
    if (p.kernel == KERNEL_DIRECT) {
        switch (p.lanes_per_row) {
        case 8: return launch_direct<8, K, F16>(p, x, y, m, hw, vec, s);
        case 16: return launch_direct<16, K, F16>(p, x, y, m, hw, vec, s);
        case 32: return launch_direct<32, K, F16>(p, x, y, m, hw, vec, s);
        case 64: return launch_direct<64, K, F16>(p, x, y, m, hw, vec, s);
        default: return hipErrorInvalidValue;
        }
    }
    switch (p.lanes_per_row * 10 + p.vecs_per_lane) {
    case 81: return launch_strip<8, 1, K, F16>(p, x, y, m, hw, vec, s);
    case 82: return launch_strip<8, 2, K, F16>(p, x, y, m, hw, vec, s);
    case 161: return launch_strip<16, 1, K, F16>(p, x, y, m, hw, vec, s);
    case 162: return launch_strip<16, 2, K, F16>(p, x, y, m, hw, vec, s);
    case 321: return launch_strip<32, 1, K, F16>(p, x, y, m, hw, vec, s);
    case 322: return launch_strip<32, 2, K, F16>(p, x, y, m, hw, vec, s);
    case 641: return launch_strip<64, 1, K, F16>(p, x, y, m, hw, vec, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t prepare_launch(DevicePlan &p) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    e = hipDeviceGetAttribute(&p.num_cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess)
        return e;
    if (p.storage == 1)
        return p.k == 4 ? prepare<4, true>(p) : prepare<1, true>(p);
    return p.k == 4 ? prepare<4, false>(p) : prepare<1, false>(p);
}

hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                       hipStream_t stream) {
    if (p.storage == 1)
        return p.k == 4 ? dispatch<4, true>(p, x, y, m, hw, vec, stream)
                        : dispatch<1, true>(p, x, y, m, hw, vec, stream);
    return p.k == 4 ? dispatch<4, false>(p, x, y, m, hw, vec, stream)
                    : dispatch<1, false>(p, x, y, m, hw, vec, stream);
}

}  // namespace spconv
