// gfx950 (CDNA4) kernels for the sparse 1x1 convolution
//     Y[n, r, p] = act(b[r] + sum_c W[r, c] * X[n, c, p])
// (Fast Sparse ConvNets, Sec. 3.2 / Fig. 2), over NCHW tensors.
//
// Columns.  The product's dense operand has Cin rows and N*H*W columns; column
// j is (image j / HW, position j % HW).  A workgroup works on one tile of 256
// bytes of consecutive columns at a time (64 fp32 or 128 fp16 columns).
//
// Lane groups.  A wavefront's 64 lanes form 64/G groups of G lanes; each group
// owns one (block) row of the bundle in progress and each lane accumulates
// V = 16/G vectors of 16 bytes of the tile's columns -- the paper's first
// insight (Sec. 3.2: the activations are dense, so load them as vectors along
// H*W) mapped onto wave64.  With 1xk output blocks (Sec. 3.2) one X vector
// feeds k rows from registers.  Each lane keeps its own copy of the channel
// and weight of every slot of its row: the G lanes of a group read the same
// 16-byte records with ordinary vector loads.  On gfx950 that is cheaper than
// handing one lane's weight to the others with DPP, whose FMAs and moves
// issue at a fraction of the plain FMA rate.
//
// Strip kernel.  The second and third insights (Sec. 3.2, Fig. 3: walk the
// output rows in the inner loop while one strip of spatial columns stays in
// the near cache) become: the strip X[:, tile] (Cin x 256 bytes) is copied
// from HBM straight into LDS (buffer loads with the LDS-destination bit, no
// register staging), and every wavefront walks its bundles reading X only from
// LDS: per slot and lane, V address adds, V 16-byte LDS reads and k * V * 16/e
// FMAs.  Lane (q, i) of group q reads vector G * ((q + j) % V) + i of its row
// at its j-th read, so the 16 lanes of each quarter-wavefront touch 16
// distinct 16-byte bank groups whatever channels their rows read (LDS reads
// are free of bank conflicts), and each group stores G consecutive vectors.  Workgroups are persistent: each takes tiles blockIdx.x,
// + gridDim.x, ...; the tiles left over after the last whole round are shared
// by bundle rank: P workgroups each take 1/P of a tile's bundles, so no
// compute unit idles while a few finish a last round alone.
//
// Weight streams.  Each wavefront reads its bundles' steps as one continuous
// stream (planner.hpp); the main loop is a software pipeline that fetches the
// records D steps ahead and does not stop at bundle boundaries: a scalar
// countdown of the bundle's steps triggers its epilogue (bias, activation,
// one rounding, store).  Accumulation is fp32 FMA in ascending input-channel
// order from zero; the bias is added after the sum.
//
// Direct kernel.  When Cin * 256 bytes does not fit in LDS, the same loop
// reads X straight from global memory (L1/L2) instead of the strip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>
#include <utility>

#include "launch.hpp"

namespace spconv {
namespace {

typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

template <bool F16>
struct Elem;
template <>
struct Elem<false> {
    using T = float;
    static __device__ __forceinline__ float from_f32(float v) { return v; }
};
template <>
struct Elem<true> {
    using T = _Float16;
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

__device__ __forceinline__ u4 bload16(Rsrc r, int32_t voff, int32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    u4 o;
    o.x = v[0];
    o.y = v[1];
    o.z = v[2];
    o.w = v[3];
    return o;
}

// An offset no buffer resource of this file reaches: the load returns zeros.
constexpr int32_t kOutOfRange = static_cast<int32_t>(0x80000000u);
// Largest byte size given to a buffer resource (offsets stay below kOutOfRange).
constexpr int64_t kMaxRecords = 0x7ffffff0;


// Call f(std::integral_constant<int, I>) for I = 0 .. N-1, unrolled.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------------------
// Work distribution over persistent workgroups
// ---------------------------------------------------------------------------

struct Args {
    int32_t cin, cout, hw, m, act;
    int32_t xc;          // channels per image of X (the plan's cin, or more for a channel-range pass)
    int32_t accum;       // add Y's values (partial sums of earlier channel ranges) before the bias
    int32_t splits;      // the plan has split rows (row-table entries kRowPiece)
    int32_t vec;         // 16-byte global loads and stores (see launch_spmm)
    int32_t strip_rows;  // LDS strip channels (a multiple of 4); 0 for the direct kernel
    int32_t regions;     // strip parts refilled independently (pipelined kernel)
    int32_t region_rows; // channels per part, a multiple of 4
    int32_t table_off;   // LDS byte offset of the bundle table
    int32_t ctl_off;     // LDS byte offset of the strip-refill counters (pipelined kernel)
    int32_t nbundles;
    int32_t busy_waves;  // wavefronts with at least one bundle
    int32_t idx_bytes, val_bytes;
    int64_t x_bytes, y_bytes;
    int32_t tiles;        // tiles of the launch
    int32_t whole_tiles;  // tiles processed whole: a multiple of the grid
    int32_t tail_parts;   // workgroups sharing each remaining tile (a power of two)
    int32_t nxcd;         // workgroup i runs on XCD i % nxcd; the grid is a multiple of it
    // fused depthwise stage (simple strip kernel, fp32): stride (0 = none), its
    // activation, the input's height and width, the output width, and the
    // taps and biases (kDwParams floats per strip channel)
    int32_t dw_stride, dw_act, in_h, in_w, out_w;
    int32_t stage_off, stage_bytes;  // LDS staging area of its input windows
    const float *dw;
    int32_t *flag;  // the plan's error word: bit 0 set when a bounded wait gives up
    int32_t spin;   // bound of every wait on a counter (sleeps)
};

// Bit 0 of the plan's error word: a bounded wait gave up (the output of that
// launch is not trusted; spconv_plan_check reports it).  One lane, a vector
// atomic.
__device__ __forceinline__ void flag_wait_gave_up(const Args &a, int lane) {
    if (lane == 0)
        __hip_atomic_fetch_or(a.flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A workgroup's unit of work: a tile, whole (part < 0) or one of tail_parts
// parts of its bundles; tile < 0 when none is left.  `round` counts the whole
// tiles (-1 for a shared one).
//
// Tiles are laid out so that the workgroups of one XCD work on neighbouring
// tiles: XCD x owns the whole tiles [x * W, (x + 1) * W), W = whole_tiles /
// nxcd, and its workgroups take them one per round in order.  A strip row of a
// tile rarely starts or ends on a 128-byte line, and the neighbouring tile
// needs the rest of that line: on the same XCD it finds it in L2.  All parts
// of a shared tile run on one XCD, so its strip is fetched from memory once.
struct Work {
    int32_t tile, part, round;
};

__device__ __forceinline__ Work tail_work(const Args &a) {
    const int32_t b = static_cast<int32_t>(blockIdx.x);
    const int32_t x = b % a.nxcd, lb = b / a.nxcd;
    const int32_t u = x + a.nxcd * (lb / a.tail_parts);  // remaining tile of this workgroup
    if (u < a.tiles - a.whole_tiles)
        return Work{a.whole_tiles + u, a.tail_parts > 1 ? lb % a.tail_parts : -1, -1};
    return Work{-1, -1, -1};
}

__device__ __forceinline__ Work whole_work(const Args &a, int32_t r) {
    const int32_t b = static_cast<int32_t>(blockIdx.x);
    const int32_t bpx = static_cast<int32_t>(gridDim.x) / a.nxcd;  // workgroups per XCD
    return Work{(b % a.nxcd) * (a.whole_tiles / a.nxcd) + r * bpx + b / a.nxcd, -1, r};
}

__device__ __forceinline__ Work first_work(const Args &a) {
    return a.whole_tiles > 0 ? whole_work(a, 0) : tail_work(a);
}

__device__ __forceinline__ Work next_work(const Args &a, Work w) {
    if (w.round >= 0)
        return (w.round + 1) * static_cast<int32_t>(gridDim.x) < a.whole_tiles ? whole_work(a, w.round + 1)
                                                                               : tail_work(a);
    return Work{-1, -1, -1};
}

// ---------------------------------------------------------------------------
// Lane geometry, tile addressing, slot arithmetic, epilogue
// ---------------------------------------------------------------------------

template <int G, bool F16>
struct Geo {
    using T = typename Elem<F16>::T;
    static constexpr int E = sizeof(T);
    static constexpr int QE = 16 / E;   // columns per 16-byte vector
    static constexpr int V = 16 / G;    // vectors per lane and slot
    static constexpr int NB = 64 / G;   // block rows per bundle
    static constexpr int TC = 256 / E;  // columns per tile
};

// One step's records as one lane holds them: the channel offsets of its row's
// 4 slots and their weights, slot-major with K weights per slot (K == 1: the 4
// slots' weights; K == 4: w[u] = the 4 rows' weights of slot u).
template <int K>
struct Entry {
    u4 off;
    u4 w[K];
};

// The same from one resource over both streams, the weights `vdelta` bytes
// after the channel offsets (the plan's device image keeps them in that
// order): one buffer descriptor fewer in scalar registers.
template <int G, int K>
__device__ __forceinline__ Entry<K> load_entry_one(Rsrc r, int32_t vdelta, int q, int32_t s) {
    constexpr int NB = 64 / G;
    Entry<K> en;
    en.off = bload16(r, q * 16, s * NB * 16);
#pragma unroll
    for (int kk = 0; kk < K; ++kk)
        en.w[kk] = bload16(r, vdelta + q * 16 * K + 16 * kk, s * NB * 16 * K);
    return en;
}

template <int G, int K>
__device__ __forceinline__ Entry<K> load_entry(Rsrc ri, Rsrc rv, int q, int32_t s) {
    constexpr int NB = 64 / G;
    Entry<K> en;
    en.off = bload16(ri, q * 16, s * NB * 16);
#pragma unroll
    for (int kk = 0; kk < K; ++kk)
        en.w[kk] = bload16(rv, q * 16 * K + 16 * kk, s * NB * 16 * K);
    return en;
}

// The vectors a lane reads and accumulates: its j-th is vector vb[j] of the
// tile row.  For a fixed j the 16 lanes of a quarter-wavefront read 16
// distinct vectors (bank groups) whatever their rows' channels, and the G
// lanes of a group store G consecutive vectors.
template <int G, bool F16>
struct Lane {
    using GE = Geo<G, F16>;
    int q, li;
    int32_t vb[GE::V], lb[GE::V];
    __device__ __forceinline__ explicit Lane(int lane) : q(lane / G), li(lane % G) {
#pragma unroll
        for (int j = 0; j < GE::V; ++j) {
            vb[j] = G * ((q + j) % GE::V) + li;
            lb[j] = 16 * vb[j];
        }
    }
};

// Where one tile's columns of the lane live: X and Y are addressed from the
// tile's first image with 32-bit byte offsets (out of range past the last
// column).
template <int G, bool F16>
struct TileAddr {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    int32_t col0, n0;
    Rsrc rx, ry;
    int32_t xo[GE::V], yo[GE::V];
    __device__ __forceinline__ void set(const Args &a, const Lane<G, F16> &L, const T *x, T *y, int32_t tile) {
        col0 = tile * GE::TC;
        n0 = col0 / a.hw;
        const int64_t xbase = static_cast<int64_t>(n0) * a.xc * a.hw;
        const int64_t ybase = static_cast<int64_t>(n0) * a.cout * a.hw;
        rx = make_rsrc(x + xbase, static_cast<uint32_t>(std::min<int64_t>(a.x_bytes - xbase * GE::E, kMaxRecords)));
        ry = make_rsrc(y + ybase, static_cast<uint32_t>(std::min<int64_t>(a.y_bytes - ybase * GE::E, kMaxRecords)));
#pragma unroll
        for (int j = 0; j < GE::V; ++j) {
            const int32_t c = col0 + L.vb[j] * GE::QE;
            const int32_t n = c / a.hw;
            const int32_t p = c - n * a.hw;
            xo[j] = c < a.m ? ((n - n0) * a.xc * a.hw + p) * GE::E : kOutOfRange;
            yo[j] = c < a.m ? ((n - n0) * a.cout * a.hw + p) * GE::E : kOutOfRange;
        }
    }
};

// X offsets of a lane's columns for the direct kernel without aligned 16-byte
// vectors (H*W not a multiple of the vector width), computed once per tile
// so the inner loop needs no division.  Byte offsets count from channel 0 of
// the tile's first image; kOutOfRange past the last column.
//   fp32 with H*W >= 4 (`pair`): xe[j][0] = offset of element 0 of vector j,
//     xe[j][1] = the number k of its elements in that image, xe[j][2] = an
//     offset whose element e >= k is element e of the vector (the next
//     image's plane, shifted back by k).  A read is one 16-byte load, plus a
//     second only where a vector straddles two images; the loads are 4-byte
//     aligned, and raw buffer loads check bounds per dword.
//   otherwise: xe[j][e] = offset of element e (one 4- or 2-byte load each).
template <int G, bool F16, bool ON>
struct ColOff {
    __device__ __forceinline__ void set(const Args &, const Lane<G, F16> &, int32_t) {}
};
template <int G, bool F16>
struct ColOff<G, F16, true> {
    using GE = Geo<G, F16>;
    int32_t xe[GE::V][GE::QE];
    __device__ __forceinline__ static bool pair(const Args &a) { return !F16 && a.hw >= GE::QE; }
    __device__ __forceinline__ void set(const Args &a, const Lane<G, F16> &L, int32_t tile) {
        const int32_t col0 = tile * GE::TC;
        const int32_t n0 = col0 / a.hw;
        if (pair(a)) {
#pragma unroll
            for (int j = 0; j < GE::V; ++j) {
                const int32_t c = col0 + L.vb[j] * GE::QE;
                const int32_t n = c / a.hw;
                const int32_t p = c - n * a.hw;
                const int32_t k = std::min(GE::QE, a.hw - p);
                xe[j][0] = c < a.m ? ((n - n0) * a.xc * a.hw + p) * GE::E : kOutOfRange;
                xe[j][1] = k;
                xe[j][2] = c + k < a.m ? ((n + 1 - n0) * a.xc * a.hw - k) * GE::E : kOutOfRange;
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < GE::V; ++j)
#pragma unroll
            for (int e = 0; e < GE::QE; ++e) {
                const int32_t c = col0 + L.vb[j] * GE::QE + e;
                const int32_t n = c / a.hw;
                xe[j][e] = c < a.m ? ((n - n0) * a.xc * a.hw + (c - n * a.hw)) * GE::E : kOutOfRange;
            }
    }
};

__device__ __forceinline__ void bstore16(u4 v, Rsrc r, int32_t voff) {
    // plain write-back stores: the lane groups' pieces of a 128-byte line meet in L2
    __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, 0, 0);
}

// acc[k][j][e] += w(slot U, row k) * x[j][e]
template <int G, int K, bool F16, int U>
__device__ __forceinline__ void fma_slot(float (&acc)[K][16 / G][16 / (F16 ? 2 : 4)], const Entry<K> &en,
                                         const u4 (&xr)[16 / G]) {
    using GE = Geo<G, F16>;
#pragma unroll
    for (int kk = 0; kk < K; ++kk) {
        // the step's weights are slot-major, K per slot: weight kk of slot U is
        // float U * K + kk of the lane's 4 K floats
        const float w = __uint_as_float(en.w[(U * K + kk) / 4][(U * K + kk) % 4]);
#pragma unroll
        for (int j = 0; j < GE::V; ++j) {
            if constexpr (F16) {
                const h8 xh = __builtin_bit_cast(h8, xr[j]);
#pragma unroll
                for (int e = 0; e < GE::QE; ++e)
                    acc[kk][j][e] = __builtin_fmaf(w, static_cast<float>(xh[e]), acc[kk][j][e]);
            } else {
                const f4 xf = __builtin_bit_cast(f4, xr[j]);
#pragma unroll
                for (int e = 0; e < GE::QE; ++e)
                    acc[kk][j][e] = __builtin_fmaf(w, xf[e], acc[kk][j][e]);
            }
        }
    }
}

// Bias, activation (a clamp to [lo, hi]), one rounding, store of block row rb;
// then the accumulators restart from zero.  rb_next is the next lane group's
// row-table entry: kRowPiece when this group holds the even nonzeros of a
// split row and the next one its odd nonzeros, whose partial sums are added
// here first.
template <int G, int K, bool F16, bool VEC>
__device__ __forceinline__ void finish_rows(const Args &a, const Lane<G, F16> &L, const TileAddr<G, F16> &ta,
                                            typename Geo<G, F16>::T *y,
                                            float (&acc)[K][16 / G][16 / (F16 ? 2 : 4)], const float (&bv)[K],
                                            int32_t rb, int32_t rb_next, float lo, float hi) {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    if (a.splits) {
        // Every lane reads its counterpart in the next group (lane + G), whose
        // vector j - 1 holds this lane's vector j (the per-group rotation of
        // the vectors).  Only a first piece adds, and it reads a second piece,
        // which never adds, so no lane reads a value another has changed.
        const bool add = rb_next == kRowPiece;
        const int src = ((static_cast<int>(threadIdx.x & 63) + G) & 63) << 2;
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int j = 0; j < GE::V; ++j)
#pragma unroll
                for (int e = 0; e < GE::QE; ++e) {
                    const float pv = __int_as_float(__builtin_amdgcn_ds_bpermute(
                        src, __float_as_int(acc[kk][(j + GE::V - 1) % GE::V][e])));
                    if (add)
                        acc[kk][j][e] += pv;
                }
    }
    if (rb >= 0) {
        const int32_t hwe = a.hw * GE::E;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) {
            const int32_t ro = (rb * K + kk) * hwe;
#pragma unroll
            for (int j = 0; j < GE::V; ++j) {
                T out[GE::QE];
#pragma unroll
                for (int e = 0; e < GE::QE; ++e)
                    out[e] = Elem<F16>::from_f32(fminf(fmaxf(acc[kk][j][e] + bv[kk], lo), hi));
                if constexpr (VEC) {
                    bstore16(*reinterpret_cast<const u4 *>(out), ta.ry, ta.yo[j] + ro);
                } else {
                    // element stores through the tile's Y resource (32-bit
                    // offsets from its first image): the vector's first
                    // column's image and position, then carried forward (one
                    // division per vector)
                    const int32_t c0 = ta.col0 + L.vb[j] * GE::QE;
                    int32_t n = c0 / a.hw;
                    int32_t pp = c0 - n * a.hw;
#pragma unroll
                    for (int e = 0; e < GE::QE; ++e) {
                        const int32_t off = c0 + e < a.m ? (((n - ta.n0) * a.cout + rb * K + kk) * a.hw + pp) * GE::E
                                                         : kOutOfRange;
                        if constexpr (F16)
                            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, out[e]), ta.ry, off, 0, 0);
                        else
                            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, out[e]), ta.ry, off, 0, 0);
                        if (++pp == a.hw) {
                            pp = 0;
                            ++n;
                        }
                    }
                }
            }
        }
    }
#pragma unroll
    for (int kk = 0; kk < K; ++kk)
#pragma unroll
        for (int j = 0; j < GE::V; ++j)
#pragma unroll
            for (int e = 0; e < GE::QE; ++e)
                acc[kk][j][e] = 0.0f;
}

// X vector j of a slot with channel offset o: from the LDS strip, or (direct
// kernel, o = channel) from global memory.
template <int G, bool F16, bool DIRECT, bool VEC>
__device__ __forceinline__ u4 read_x(const Args &a, const Lane<G, F16> &L, const TileAddr<G, F16> &ta,
                                     const ColOff<G, F16, DIRECT && !VEC> &co, const unsigned char *lds,
                                     uint32_t o, int j) {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    if constexpr (DIRECT) {
        const int32_t ro = static_cast<int32_t>(o) * a.hw * GE::E;  // channel o's plane
        if constexpr (VEC) {
            return bload16(ta.rx, ta.xo[j] + ro, 0);
        } else {
            if constexpr (!F16) {
                if (co.pair(a)) {
                    u4 va = bload16(ta.rx, co.xe[j][0] + ro, 0);
                    if (co.xe[j][1] < GE::QE) {
                        // the vector straddles two images: its tail from the next plane
                        const u4 vb = bload16(ta.rx, co.xe[j][2] + ro, 0);
#pragma unroll
                        for (int e = 1; e < GE::QE; ++e)
                            if (e >= co.xe[j][1])
                                va[e] = vb[e];
                    }
                    return va;
                }
            }
            // any HW: element by element (past the last column: zero)
            T v[GE::QE];
#pragma unroll
            for (int e = 0; e < GE::QE; ++e) {
                if constexpr (F16)
                    v[e] = __builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(ta.rx, co.xe[j][e] + ro, 0, 0));
                else
                    v[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ta.rx, co.xe[j][e] + ro, 0, 0));
            }
            return *reinterpret_cast<const u4 *>(v);
        }
    } else {
        return *reinterpret_cast<const u4 *>(lds + (o + L.lb[j]));
    }
}

// ---------------------------------------------------------------------------
// The simple loop: the bundles [b0, b1) of a wavefront's stream over one tile,
// records fetched two steps ahead
// ---------------------------------------------------------------------------

template <int G, int K, bool F16, bool DIRECT, bool VEC, bool ACC = false, int D = 2>
__device__ __forceinline__ void run_simple(const Args &a, const Lane<G, F16> &L, const TileAddr<G, F16> &ta,
                                           const ColOff<G, F16, DIRECT && !VEC> &co, typename Geo<G, F16>::T *y,
                                           const unsigned char *lds, Rsrc ri, Rsrc rv,
                                           const int32_t *__restrict__ hdr, const int32_t *rows_lds,
                                           const float *bias_lds, int32_t b0, int32_t b1, float lo, float hi) {
    using GE = Geo<G, F16>;
    constexpr int NR = D + 1;  // D records fetched ahead
    const int32_t s_first = hdr[2 * b0];
    const int32_t nsteps = hdr[2 * (b1 - 1)] + hdr[2 * (b1 - 1) + 1] - s_first;

    float acc[K][GE::V][GE::QE];
#pragma unroll
    for (int kk = 0; kk < K; ++kk)
#pragma unroll
        for (int j = 0; j < GE::V; ++j)
#pragma unroll
            for (int e = 0; e < GE::QE; ++e)
                acc[kk][j][e] = 0.0f;

    // the bundle in progress: its row and biases (of this lane's group), steps left
    int32_t b = b0, rb = 0, rbn = -1, left = 0;
    float bv[K];
    // Channel-range passes after the first (ACC, fp32): a row's
    // accumulators start from its values in Y, the sums over the earlier
    // channels, so each output is still summed in ascending channel order
    // from zero.  They are loaded one bundle ahead.
    float pn[K][GE::V][GE::QE];
    auto load_part = [&](int32_t bb) __attribute__((always_inline)) {
        const int32_t row = rows_lds[bb * GE::NB + L.q];
        const int32_t hwe = a.hw * GE::E;
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int j = 0; j < GE::V; ++j) {
                if constexpr (VEC) {
                    const u4 v = row >= 0 ? bload16(ta.ry, ta.yo[j] + (row * K + kk) * hwe, 0) : u4{0u, 0u, 0u, 0u};
#pragma unroll
                    for (int e = 0; e < GE::QE; ++e)
                        pn[kk][j][e] = __uint_as_float(v[e]);
                } else {
                    const int32_t c0 = ta.col0 + L.vb[j] * GE::QE;
                    int32_t n = c0 / a.hw;
                    int32_t pp = c0 - n * a.hw;
#pragma unroll
                    for (int e = 0; e < GE::QE; ++e) {
                        const int32_t off = row >= 0 && c0 + e < a.m
                                                ? (((n - ta.n0) * a.cout + row * K + kk) * a.hw + pp) * GE::E
                                                : kOutOfRange;
                        pn[kk][j][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ta.ry, off, 0, 0));
                        if (++pp == a.hw) {
                            pp = 0;
                            ++n;
                        }
                    }
                }
            }
    };
    auto start_bundle = [&]() __attribute__((always_inline)) {
        rb = rows_lds[b * GE::NB + L.q];
        rbn = L.q + 1 < GE::NB ? rows_lds[b * GE::NB + L.q + 1] : -1;
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
            bv[kk] = bias_lds[(b * GE::NB + L.q) * K + kk];
        left = hdr[2 * b + 1];
        if constexpr (ACC) {
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
#pragma unroll
                for (int j = 0; j < GE::V; ++j)
#pragma unroll
                    for (int e = 0; e < GE::QE; ++e)
                        acc[kk][j][e] = pn[kk][j][e];
            if (b + 1 < b1)
                load_part(b + 1);
        }
    };
    if constexpr (ACC)
        load_part(b0);
    start_bundle();

    // A ring of NR entries (step i of the run in entry i % NR), unrolled over
    // NR steps so every index is a constant.  Entries fetched past the stream's
    // end hold other bundles' data or zeros (buffer bounds) and are never used.
    Entry<K> cr[NR];
#pragma unroll
    for (int d = 0; d < D; ++d)
        cr[d] = load_entry<G, K>(ri, rv, L.q, s_first + d);
    for (int32_t s0 = 0; s0 < nsteps; s0 += NR) {
        static_for<NR>([&](auto kc) __attribute__((always_inline)) {
            constexpr int KI = decltype(kc)::value;
            if (s0 + KI < nsteps) {
                cr[(KI + D) % NR] = load_entry<G, K>(ri, rv, L.q, s_first + s0 + KI + D);
                static_for<4>([&](auto uc) __attribute__((always_inline)) {
                    constexpr int U = decltype(uc)::value;
                    u4 xr[GE::V];
#pragma unroll
                    for (int j = 0; j < GE::V; ++j)
                        xr[j] = read_x<G, F16, DIRECT, VEC>(a, L, ta, co, lds, cr[KI].off[U], j);
                    fma_slot<G, K, F16, U>(acc, cr[KI], xr);
                });
                if (--left == 0) {
                    finish_rows<G, K, F16, VEC>(a, L, ta, y, acc, bv, rb, rbn, lo, hi);
                    if (++b < b1)
                        start_bundle();
                }
            }
        });
    }
}

// A wavefront's share of a work item: all of its bundles (whole tile) or its
// bundles of rank % tail_parts == part (shared tile), one run each.
template <int G, int K, bool F16, bool DIRECT, bool VEC, bool ACC = false, int D = 2>
__device__ __forceinline__ void run_item(const Args &a, const Lane<G, F16> &L, const TileAddr<G, F16> &ta,
                                         const ColOff<G, F16, DIRECT && !VEC> &co, typename Geo<G, F16>::T *y,
                                         const unsigned char *lds, Rsrc ri, Rsrc rv, const int32_t *__restrict__ hdr,
                                         const int32_t *__restrict__ rank, const int32_t *rows_lds,
                                         const float *bias_lds, int32_t wb0, int32_t wb1, int32_t part, float lo,
                                         float hi) {
    int32_t bnext = wb0;
    for (;;) {
        int32_t b0, b1;
        if (part < 0) {
            if (bnext >= wb1)
                break;
            b0 = bnext;
            b1 = wb1;
        } else {
            // the wavefront's bundles at positions part, part + tail_parts, ...
            // of its own list: every wavefront of a part gets an equal share
            while (bnext < wb1 && (bnext - wb0) % a.tail_parts != part)
                ++bnext;
            if (bnext >= wb1)
                break;
            b0 = bnext;
            b1 = bnext + 1;
        }
        bnext = b1;
        run_simple<G, K, F16, DIRECT, VEC, ACC, D>(a, L, ta, co, y, lds, ri, rv, hdr, rows_lds, bias_lds, b0, b1, lo,
                                                   hi);
    }
}

typedef int i4 __attribute__((ext_vector_type(4)));

// Buffer resource words for inline assembly: base, byte size, raw-buffer configuration.
__device__ __forceinline__ i4 rsrc_words(const void *p, int64_t bytes) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    i4 r;
    r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(v));
    r.y = __builtin_amdgcn_readfirstlane(static_cast<int>((v >> 32) & 0xffff));
    r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(std::min<int64_t>(bytes, kMaxRecords)));
    r.w = 0x00020000;
    return r;
}

// This wavefront's share of the copies of strip rows [r0, r1) (multiples of 4)
// of `tile` into LDS: instructions i = r0 / 4 + wave, + nwaves, ...; 16 lanes per
// channel row, 4 rows per instruction.
template <int G, bool F16>
__device__ __forceinline__ void copy_share(const Args &a, const typename Geo<G, F16>::T *x, uint32_t lds_base,
                                           int32_t tile, int32_t r0, int32_t r1, int wave, int nwaves, int lane) {
    using GE = Geo<G, F16>;
    const int32_t col0 = tile * GE::TC;
    const int32_t n0 = col0 / a.hw;
    const int64_t xbase = static_cast<int64_t>(n0) * a.xc * a.hw;
    const i4 rs = rsrc_words(x + xbase, a.x_bytes - xbase * GE::E);
    const int32_t cc = col0 + (lane & 15) * GE::QE;
    const int32_t n = cc / a.hw;
    const int32_t p = cc - n * a.hw;
    const int32_t crow = lane >> 4;
    const bool ok = cc < a.m;
    const int32_t hwe = a.hw * GE::E;
    const int32_t lo = ((n - n0) * a.xc * a.hw + crow * a.hw + p) * GE::E;
    for (int i = r0 / 4 + wave; i < r1 / 4; i += nwaves) {
        const int32_t voff = ok && 4 * i + crow < a.cin ? lo + i * 4 * hwe : kOutOfRange;
        const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds_base + 1024 * i);
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                     :
                     : "s"(m0), "v"(voff), "s"(rs)
                     : "memory", "m0");
    }
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt takes 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

// The strip X[:, tile] into LDS for the simple kernel; the caller synchronizes.
template <int G, bool F16, bool VEC>
__device__ __forceinline__ void load_strip_simple(const Args &a, const TileAddr<G, F16> &ta,
                                                  const typename Geo<G, F16>::T *x, unsigned char *lds,
                                                  uint32_t lds_base, int32_t tile, int tid, int nthreads, int wave,
                                                  int nwaves, int lane) {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    if constexpr (VEC) {
        copy_share<G, F16>(a, x, lds_base, tile, 0, a.strip_rows, wave, nwaves, lane);
        wait_vmcnt<0>();  // this wave's copies landed
    } else if (!F16 && a.hw >= GE::QE) {
        // fp32, any HW of at least 4: thread = one 16-byte vector of the tile
        // row (nthreads is a multiple of 16), read with one 16-byte load where
        // its 4 columns lie in one image and a second where they straddle two
        // (offsets computed once; raw buffer loads check bounds per dword, so
        // columns past the last read zero); all of a batch of rows' loads are
        // issued before their LDS writes
        const int vi = tid & 15;
        const int32_t c = ta.col0 + vi * GE::QE;
        int32_t off0 = kOutOfRange, off2 = kOutOfRange, kfirst = GE::QE;
        if (c < a.m) {
            const int32_t n = c / a.hw;
            const int32_t p = c - n * a.hw;
            kfirst = std::min(GE::QE, a.hw - p);
            off0 = ((n - ta.n0) * a.xc * a.hw + p) * GE::E;
            off2 = c + kfirst < a.m ? ((n + 1 - ta.n0) * a.xc * a.hw - kfirst) * GE::E : kOutOfRange;
        }
        const int32_t hwe = a.hw * GE::E;
        const int32_t step = nthreads >> 4;  // rows covered by one pass of the workgroup
        constexpr int U = 4;
        for (int32_t r0 = tid >> 4; r0 < a.strip_rows; r0 += U * step) {
            u4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t row = r0 + u * step;
                const bool in = row < a.cin;
                v[u] = bload16(ta.rx, in ? off0 + row * hwe : kOutOfRange, 0);
                if (kfirst < GE::QE) {
                    const u4 vb = bload16(ta.rx, in ? off2 + row * hwe : kOutOfRange, 0);
#pragma unroll
                    for (int e = 1; e < GE::QE; ++e)
                        if (e >= kfirst)
                            v[u][e] = vb[e];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t row = r0 + u * step;
                if (row < a.strip_rows)
                    *reinterpret_cast<u4 *>(lds + row * kRowBytes + vi * 16) = v[u];
            }
        }
    } else {
        // fp16, or HW below 4: gather element by element
        for (int i = tid; i < a.strip_rows * 16; i += nthreads) {
            const int32_t row = i >> 4;
            T v[GE::QE];
#pragma unroll
            for (int e = 0; e < GE::QE; ++e) {
                const int32_t c = ta.col0 + (i & 15) * GE::QE + e;
                v[e] = T(0);
                if (row < a.cin && c < a.m) {
                    const int32_t n = c / a.hw;
                    v[e] = x[(static_cast<int64_t>(n) * a.xc + row) * a.hw + (c - n * a.hw)];
                }
            }
            *reinterpret_cast<u4 *>(lds + i * 16) = *reinterpret_cast<const u4 *>(v);
        }
    }
}

// The strip of a plan with a depthwise stage, computed instead of copied:
// column j of strip row c is the depthwise output
//     D[n, c, oy, ox] = act1(b1[c] + sum_{dy, dx} K[c][dy][dx] * X[n, c, s*oy + dy - 1, s*ox + dx - 1])
// (zero padding 1, stride s) of output column j = (n, oy * out_w + ox).  The
// taps are fp32 fma in dy, dx order from zero, then the bias, then the clamp.
//
// Lane j owns column j of the tile for every row: its 9 tap offsets (relative
// to the tile's first image) are computed once per tile, a tap in the padding
// gets an offset past the buffer so its load returns 0 without touching
// memory.  Each wavefront computes whole rows, 4 at a time (rows wave,
// wave + nwaves, ...), so a row's taps and bias are wavefront-uniform and one
// load instruction reads 64 neighbouring columns of one input plane.  Rows
// past cin are zero.  The caller synchronizes.
__device__ __forceinline__ void dw_strip(const Args &a, const float *__restrict__ x, unsigned char *lds,
                                         int32_t tile, int wave, int nwaves, int lane) {
    const float lo = a.dw_act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.dw_act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t s = a.dw_stride;
    const int32_t ihw = a.in_h * a.in_w;
    const int32_t col0 = tile * 64;
    const int32_t n0 = col0 / a.hw;
    const int32_t c = col0 + lane;
    const bool ok = c < a.m;
    int32_t off[9];
    {
        const int32_t n = c / a.hw;
        const int32_t pp = c - n * a.hw;
        const int32_t oy = pp / a.out_w;
        const int32_t ox = pp - oy * a.out_w;
        const int32_t plane = (n - n0) * a.cin * ihw;  // (n, channel 0) from (n0, channel 0), elements
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int32_t iy = oy * s + t / 3 - 1;
            const int32_t ix = ox * s + t % 3 - 1;
            const bool in = ok && iy >= 0 && iy < a.in_h && ix >= 0 && ix < a.in_w;
            off[t] = in ? (plane + iy * a.in_w + ix) * 4 : kOutOfRange;
        }
    }
    const int64_t xbase = static_cast<int64_t>(n0) * a.cin * ihw;
    const int64_t xbytes = a.x_bytes - xbase * 4;
    constexpr int R = 4;
    for (int32_t r0 = wave; r0 < a.strip_rows; r0 += R * nwaves) {
        float v[R];
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int32_t row = r0 + u * nwaves;
            v[u] = 0.0f;
            if (row < a.cin) {
                // channel row of the tile's first image: one buffer resource per row
                const int64_t rowoff = static_cast<int64_t>(row) * ihw;
                const Rsrc rx = make_rsrc(x + xbase + rowoff,
                                          static_cast<uint32_t>(std::min<int64_t>(xbytes - rowoff * 4, kMaxRecords)));
                const float *kp = a.dw + row * kDwParams;
                float acc = 0.0f;
#pragma unroll
                for (int t = 0; t < 9; ++t)
                    acc = __builtin_fmaf(kp[t], __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rx, off[t], 0, 0)), acc);
                v[u] = fminf(fmaxf(acc + kp[9], lo), hi);  // columns past the last one: never stored
            }
        }
#pragma unroll
        for (int u = 0; u < R; ++u) {
            const int32_t row = r0 + u * nwaves;
            if (row < a.strip_rows)
                *reinterpret_cast<float *>(lds + row * kRowBytes + lane * 4) = v[u];
        }
    }
}

// The same strip through LDS: a tile's 64 output columns read, per channel, a
// window of input rows -- for each image n0 .. n1 the tile touches, rows
// iy_a(n) .. iy_b(n) of its plane, one contiguous span of memory each.  The
// workgroup stages the windows of `ch` channels at a time with 16-byte loads
// (each input element is fetched once per tile, not once per tap), and each
// wavefront computes whole strip rows from there, lane j column j, 9 LDS
// reads per output.  The loads of the next chunk are issued into registers
// before the current chunk is computed, so their latency overlaps it.  Spans
// start on 16-byte boundaries in LDS (piece n at base(n), lengths rounded up
// to 4 floats), so the staging copy of vector i is simply LDS bytes 16 i ..
// 16 i + 15 and no two threads write one word.  Returns false, doing nothing,
// when one channel's window does not fit in the staging area.  Same
// arithmetic as dw_strip.  The caller synchronizes after it.
constexpr int kStageVecs = 4;  // staged 16-byte vectors per thread and chunk, at most

// The depthwise parameters are read-only for the whole launch: reading them
// through the constant address space lets wavefront-uniform reads become
// scalar loads.
using ConstF = const __attribute__((address_space(4))) float;
__device__ __forceinline__ ConstF *as_constant(const float *p) { return (ConstF *)(p); }

__device__ __forceinline__ bool dw_strip_staged(const Args &a, const float *__restrict__ x, unsigned char *lds,
                                                int32_t tile, int tid, int nthreads, int wave, int nwaves,
                                                int lane) {
    const int32_t s = a.dw_stride;
    const int32_t in_w = a.in_w;
    const int32_t ihw = a.in_h * in_w;
    // the tile's images and the rows of each it needs (uniform)
    const int32_t col0 = tile * 64;
    const int32_t clast = std::min(col0 + 63, a.m - 1);
    const int32_t n0 = col0 / a.hw, n1 = clast / a.hw;
    const int32_t ya0 = std::max(0, (col0 - n0 * a.hw) / a.out_w * s - 1);           // iy_a(n0)
    const int32_t yb1 = std::min(a.in_h - 1, (clast - n1 * a.hw) / a.out_w * s + 1);  // iy_b(n1)
    const int32_t yb0 = n1 == n0 ? yb1 : a.in_h - 1;                                  // iy_b(n0)
    const int32_t ya1 = n1 == n0 ? ya0 : 0;                                           // iy_a(n1)
    const int32_t len0 = (yb0 - ya0 + 1) * in_w, len1 = (yb1 - ya1 + 1) * in_w;
    const int32_t pfull = (ihw + 3) & ~3;     // a whole plane (images between n0 and n1)
    const int32_t p0 = (len0 + 3) & ~3;       // LDS floats of each piece
    const int32_t p1 = (len1 + 3) & ~3;
    const int32_t spc = n1 == n0 ? p0 : p0 + (n1 - n0 - 1) * pfull + p1;  // LDS floats per channel
    const int32_t nv = spc / 4;  // 16-byte vectors per channel
    const int32_t ch = std::min(a.stage_bytes / 4 / spc, kStageVecs * nthreads / nv);
    if (ch == 0)
        return false;

    // this lane's taps: LDS float offsets in its channel's window, -1 in the padding
    const int32_t c = col0 + lane;
    const bool ok = c < a.m;
    int32_t toff[9];
    {
        const int32_t n = ok ? c / a.hw : n0;
        const int32_t pp = c - n * a.hw;
        const int32_t oy = pp / a.out_w;
        const int32_t ox = pp - oy * a.out_w;
        const int32_t ya = n == n0 ? ya0 : 0;
        const int32_t base = n == n0 ? 0 : p0 + (n - n0 - 1) * pfull;
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int32_t iy = oy * s + t / 3 - 1;
            const int32_t ix = ox * s + t % 3 - 1;
            const bool in = ok && iy >= 0 && iy < a.in_h && ix >= 0 && ix < in_w;
            toff[t] = in ? base + (iy - ya) * in_w + ix : -1;
        }
    }
    // this thread's staging vectors i = tid + j * nthreads of a chunk: their
    // channel within the chunk and their byte offset from channel 0 of the
    // tile's first image (chunk c0 adds c0 planes)
    int32_t vr[kStageVecs], vg[kStageVecs];
#pragma unroll
    for (int j = 0; j < kStageVecs; ++j) {
        const int32_t i = tid + j * nthreads;
        const int32_t r = i / nv;
        const int32_t f = (i - r * nv) * 4;  // LDS float offset in the channel's window
        int32_t n, off;
        if (f < p0) {
            n = n0;
            off = f;
        } else if (f < spc - p1) {
            n = n0 + 1 + (f - p0) / pfull;
            off = (f - p0) % pfull;
        } else {
            n = n1;
            off = f - (spc - p1);
        }
        vr[j] = r < ch ? r : INT32_MAX;
        vg[j] = r < ch ? (((n - n0) * a.cin + r) * ihw + (n == n0 ? ya0 : 0) * in_w + off) * 4 : 0;
    }
    const float lo = a.dw_act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.dw_act == 2 ? 6.0f : __builtin_huge_valf();
    const int64_t xbase = static_cast<int64_t>(n0) * a.cin * ihw;
    const int64_t xrel = a.x_bytes - xbase * 4;  // bytes of x from the tile's first image on
    const Rsrc rx = make_rsrc(x + xbase, static_cast<uint32_t>(std::min<int64_t>(xrel, kMaxRecords)));
    float *stage = reinterpret_cast<float *>(lds + a.stage_off);

    // A vector past the last element of x is padding, never read back; raw
    // buffer loads check their bounds per dword, so the elements of a vector
    // that straddles the end of x still arrive and the rest read 0.
    u4 v[kStageVecs];
    auto fetch = [&](int32_t c0) __attribute__((always_inline)) {
        const int32_t nch = std::min(ch, a.cin - c0);
#pragma unroll
        for (int j = 0; j < kStageVecs; ++j)
            v[j] = bload16(rx, vr[j] < nch ? vg[j] + c0 * ihw * 4 : kOutOfRange, 0);
    };
    fetch(0);
    for (int32_t c0 = 0; c0 < a.cin; c0 += ch) {
        const int32_t nch = std::min(ch, a.cin - c0);
#pragma unroll
        for (int j = 0; j < kStageVecs; ++j)
            if (vr[j] < nch)
                *reinterpret_cast<u4 *>(stage + 4 * (tid + j * nthreads)) = v[j];
        __syncthreads();  // chunk staged
        if (c0 + ch < a.cin)
            fetch(c0 + ch);
        // two rows per pass, their 18 LDS reads issued together; columns past
        // the last one hold act1(b1), never stored
        for (int32_t r0 = wave; r0 < nch; r0 += 2 * nwaves) {
            float xv[2][9];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const float *w = stage + std::min(r0 + u * nwaves, nch - 1) * spc;
#pragma unroll
                for (int t = 0; t < 9; ++t)
                    xv[u][t] = w[toff[t] < 0 ? 0 : toff[t]];
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int32_t r = r0 + u * nwaves;
                if (r < nch) {
                    const ConstF *kp = as_constant(a.dw) + (c0 + r) * kDwParams;
                    float acc = 0.0f;
#pragma unroll
                    for (int t = 0; t < 9; ++t)
                        acc = __builtin_fmaf(kp[t], toff[t] < 0 ? 0.0f : xv[u][t], acc);
                    *reinterpret_cast<float *>(lds + (c0 + r) * kRowBytes + lane * 4) =
                        fminf(fmaxf(acc + kp[9], lo), hi);
                }
            }
        }
        __syncthreads();  // staging free again
    }
    // channel rows past cin read as zero
    for (int32_t row = a.cin + wave; row < a.strip_rows; row += nwaves)
        *reinterpret_cast<float *>(lds + row * kRowBytes + lane * 4) = 0.0f;
    return true;
}

// ---------------------------------------------------------------------------
// Simple kernel: for each work item, copy the strip (strip kernel; computed by
// the depthwise stage when the plan has one), then every wavefront runs its
// bundles; workgroup barriers around each strip.
// ---------------------------------------------------------------------------

// DWS: the plan has a depthwise stage (its strip is computed); without one
// the kernel carries none of that code and its registers, and fetches records
// further ahead (short runs of shared tiles would otherwise wait on them).
template <int G, int K, bool F16, bool DIRECT, bool VEC, bool ACC = false, bool DWS = false>
__global__ void __launch_bounds__(1024)
spmm_kernel(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
            const float *__restrict__ val, const int32_t *__restrict__ hdr, const int32_t *__restrict__ table,
            const int32_t *__restrict__ rank, const int32_t *__restrict__ wave_ptr, const int32_t *, const float *,
            const uint32_t *, const int32_t *, const int32_t *, Args a) {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    extern __shared__ __align__(16) unsigned char lds[];
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nwaves = static_cast<int>(blockDim.x >> 6);
    const Lane<G, F16> L(lane);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char *)lds));

    // the bundle table into LDS (once per launch)
    int32_t *rows_lds = reinterpret_cast<int32_t *>(lds + a.table_off);
    const float *bias_lds = reinterpret_cast<const float *>(rows_lds + a.nbundles * GE::NB);
    for (int i = tid; i < a.nbundles * GE::NB * (1 + K); i += blockDim.x)
        rows_lds[i] = table[i];
    if constexpr (!DIRECT) {
        // the row of zeros that padding slots read
        if (tid < kRowBytes / 16)
            *reinterpret_cast<u4 *>(lds + a.strip_rows * kRowBytes + 16 * tid) = u4{0u, 0u, 0u, 0u};
    }
    const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(a.idx_bytes));
    const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(a.val_bytes));
    // the activation as a clamp: [-inf, inf] none, [0, inf] ReLU, [0, 6] ReLU6
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t wb0 = wave_ptr[wave], wb1 = wave_ptr[wave + 1];

    Work wk = first_work(a);
    __syncthreads();  // table ready
    TileAddr<G, F16> ta;
    ColOff<G, F16, DIRECT && !VEC> co;
    while (wk.tile >= 0) {
        ta.set(a, L, x, y, wk.tile);
        if constexpr (!DIRECT) {
            bool computed = false;
            if constexpr (!F16 && DWS) {
                if (a.dw_stride) {
                    if (!dw_strip_staged(a, x, lds, wk.tile, tid, blockDim.x, wave, nwaves, lane))
                        dw_strip(a, x, lds, wk.tile, wave, nwaves, lane);
                    computed = true;
                }
            }
            if (!computed)
                load_strip_simple<G, F16, VEC>(a, ta, x, lds, lds_base, wk.tile, tid, blockDim.x, wave, nwaves,
                                               lane);
            __syncthreads();  // strip ready
        }
        co.set(a, L, wk.tile);
        // records fetched ahead: as deep as the registers allow
        constexpr int DR = K == 1 && !F16 && !DWS && !DIRECT ? (VEC ? (ACC ? 3 : 4) : (ACC ? 2 : 3)) : 2;
        run_item<G, K, F16, DIRECT, VEC, ACC, DR>(a, L, ta, co, y, lds, ri, rv, hdr, rank, rows_lds, bias_lds, wb0,
                                                  wb1, wk.part, lo, hi);
        const Work nx = next_work(a, wk);
        if constexpr (!DIRECT)
            __syncthreads();  // done with strip(wk)
        wk = nx;
    }
}

// ---------------------------------------------------------------------------
// Pipelined strip kernel (16-byte vectors): the strip is a ring of `regions`
// parts, each refilled with the next tile's channels while the wavefronts
// compute on the others.
//
// Each wavefront walks its interleaved stream (planner.hpp): its bundles, two
// at a time with one accumulator set each, merged so that the wavefront reads
// a tile's channels roughly in ascending order once.  Per strip part q, two
// LDS counters coordinate the workgroup:
//   free[q]  wavefronts (with bundles) done with part q, summed over tiles
//   fill[q]  copies of part q that have landed, summed over tiles
// A wavefront waits for fill[q] >= nwaves * (t + 1) before its first read of
// part q in tile t (a "need" event) and counts free[q] after its last one (a
// "release" event).  Every wavefront copies a 1/nwaves share of each part of
// every tile, in order: part q of tile t once free[q] >= busy * t, with
// buffer loads that write LDS directly.  It counts the share in fill[q] one
// ring turn later, when a record fetched after the share has arrived (vector
// memory operations complete in issue order), or at once when waiting.  Each
// part of tile t + 1 can thus stream in while the wavefronts are still busy
// with other parts of tile t, and fast wavefronts run ahead into tile t + 1
// without a workgroup barrier.
//
// The copies are issued with inline assembly: the compiler would otherwise
// drain every vector-memory access before the next LDS read.  Every wait on a
// counter is bounded, so a logic error cannot hang the device.  The tiles
// left after the whole rounds take the simple path.
// ---------------------------------------------------------------------------

// Steps of records fetched ahead: as many as fit beside the accumulators and
// X vectors in an 88-register budget (each entry costs 4 + 4k registers).
template <int G, int K, bool F16, int M>
struct PipeDepth {
    static constexpr int A = M * K * (16 / G) * (16 / (F16 ? 2 : 4));  // accumulators
    static constexpr int FREE = 88 - A - 4 * (16 / G);
    static constexpr int RAW = FREE / (4 + 4 * K) - 1;
    static constexpr int D = RAW < 2 ? 2 : (RAW > 6 ? 6 : RAW);
    static constexpr int NR = D + 1;
};

__device__ __forceinline__ int32_t lds_load_volatile(const int32_t *p) {
    return __atomic_load_n(p, __ATOMIC_RELAXED);
}

// One increment per wavefront (an atomic from every lane would add 64).
__device__ __forceinline__ void count_once(int32_t *p, int lane) {
    if (lane == 0)
        atomicAdd(p, 1);
}

template <int G, int K, bool F16, int M>
__global__ void __launch_bounds__(1024)
spmm_pipe(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
          const float *__restrict__ val, const int32_t *__restrict__ hdr, const int32_t *__restrict__ table,
          const int32_t *__restrict__ rank, const int32_t *__restrict__ wave_ptr,
          const int32_t *__restrict__ pidx, const float *__restrict__ pval, const uint32_t *__restrict__ psel,
          const int32_t *__restrict__ sel_ptr, const int32_t *__restrict__ wave_ev, Args a) {
    using GE = Geo<G, F16>;
    using T = typename GE::T;
    using DP = PipeDepth<G, K, F16, M>;
    constexpr int D = DP::D, NR = DP::NR;
    constexpr int LPE = 1 + K;          // vector loads per ring entry

    extern __shared__ __align__(16) unsigned char lds[];
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nwaves = static_cast<int>(blockDim.x >> 6);
    const Lane<G, F16> L(lane);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char *)lds));

    int32_t *rows_lds = reinterpret_cast<int32_t *>(lds + a.table_off);
    const float *bias_lds = reinterpret_cast<const float *>(rows_lds + a.nbundles * GE::NB);
    for (int i = tid; i < a.nbundles * GE::NB * (1 + K); i += blockDim.x)
        rows_lds[i] = table[i];
    if (tid < kRowBytes / 16)
        *reinterpret_cast<u4 *>(lds + a.strip_rows * kRowBytes + 16 * tid) = u4{0u, 0u, 0u, 0u};
    int32_t *ctl = reinterpret_cast<int32_t *>(lds + a.ctl_off);  // free[kMaxRegions], fill[kMaxRegions]
    if (tid < kMaxRegions) {
        ctl[tid] = 0;
        ctl[kMaxRegions + tid] = 0;
    }
    // the weight stream follows the channel-offset stream in the plan's image
    // (checked on the host: 0 <= pval - pidx and the end below 2^31)
    const int32_t vdelta = static_cast<int32_t>(reinterpret_cast<const char *>(pval) -
                                                reinterpret_cast<const char *>(pidx));
    const Rsrc rpr = make_rsrc(pidx, static_cast<uint32_t>(vdelta) + static_cast<uint32_t>(a.val_bytes));
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t wb0 = wave_ptr[wave], wb1 = wave_ptr[wave + 1];
    const int32_t R = a.whole_tiles / static_cast<int32_t>(gridDim.x);  // whole rounds of every workgroup

    __syncthreads();  // table, zero row and counters ready

    // ---- whole rounds ----
    // the next share this wave copies (part cq of tile ct) and the parts whose
    // shares are in flight.  Tile 0 streams in part by part like every other
    // tile: a wavefront starts on part 0 as soon as all of its shares have
    // landed, while the later parts are still on their way.
    int32_t cq = 0, ct = 0;
    uint32_t pend = 0;
    auto publish = [&]() __attribute__((always_inline)) {
        static_for<kMaxRegions>([&](auto qc) __attribute__((always_inline)) {
            constexpr int Q = decltype(qc)::value;
            if (pend & (1u << Q))
                count_once(&ctl[kMaxRegions + Q], lane);
        });
        pend = 0;
    };
    // copy the next share if its part is free; `idle`: count it at once
    auto service = [&](bool idle) __attribute__((always_inline)) {
        if (ct < R && lds_load_volatile(&ctl[cq]) >= a.busy_waves * ct) {
            const int32_t r0 = cq * a.region_rows;
            const int32_t r1 = std::min(r0 + a.region_rows, a.strip_rows);
            copy_share<G, F16>(a, x, lds_base, whole_work(a, ct).tile, r0, r1, wave, nwaves, lane);
            pend |= 1u << cq;
            if (++cq == a.regions) {
                cq = 0;
                ++ct;
            }
            if (idle) {
                wait_vmcnt<0>();
                publish();
            }
        }
    };
    auto wait_fill = [&](int32_t q, int32_t target) __attribute__((always_inline)) {
        if (pend) {
            wait_vmcnt<0>();
            publish();
        }
        int32_t n = 0;
        for (; n < a.spin && lds_load_volatile(&ctl[kMaxRegions + q]) < target; ++n) {
            service(true);
            __builtin_amdgcn_s_sleep(1);
        }
        if (n == a.spin && lds_load_volatile(&ctl[kMaxRegions + q]) < target)
            flag_wait_gave_up(a, lane);
        // strip reads stay after the wait
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    };
    // done with a part: earlier strip reads stay before the count
    auto release = [&](int32_t q) __attribute__((always_inline)) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        count_once(&ctl[q], lane);
    };

    if (R > 0 && wb0 < wb1) {
        const int32_t ws0 = hdr[2 * wb0];
        const int32_t len = hdr[2 * (wb1 - 1)] + hdr[2 * (wb1 - 1) + 1] - ws0;  // steps per tile
        const int32_t total = R * len;
        const uint32_t *__restrict__ sel = psel + sel_ptr[wave];
        const int32_t *__restrict__ ev = wave_ev + kWaveEvents * wave;
        // LDS byte addresses of the lane's vectors in strip row 0
        uint32_t lrow[GE::V];
#pragma unroll
        for (int j = 0; j < GE::V; ++j)
            lrow[j] = lds_base + static_cast<uint32_t>(L.lb[j]);

        float acc[M][K][GE::V][GE::QE];
#pragma unroll
        for (int s = 0; s < M; ++s)
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
#pragma unroll
                for (int j = 0; j < GE::V; ++j)
#pragma unroll
                    for (int e = 0; e < GE::QE; ++e)
                        acc[s][kk][j][e] = 0.0f;
        int32_t bset[M];  // bundle in progress of each set
        // this tile's next need and release events and their indices in ev
        int32_t need = INT32_MAX, rel = INT32_MAX, ni = 0, ri_ = 0;
        uint32_t selw = 0;  // selector bits of the steps ahead (2 per step)
        TileAddr<G, F16> ta;
        // one step of set S: 4 slots of strip reads and FMAs
        auto step = [&](auto sc, const Entry<K> &en) __attribute__((always_inline)) {
            constexpr int S = decltype(sc)::value;
            static_for<4>([&](auto uc) __attribute__((always_inline)) {
                constexpr int U = decltype(uc)::value;
                u4 xr[GE::V];
#pragma unroll
                for (int j = 0; j < GE::V; ++j)
                    xr[j] = *reinterpret_cast<const __attribute__((address_space(3))) u4 *>(
                        static_cast<uintptr_t>(en.off[U] + lrow[j]));
                fma_slot<G, K, F16, U>(acc[S], en, xr);
            });
        };
        // after a bundle's last step: bias, activation and store from set S,
        // which continues with its next bundle
        auto finish = [&](auto sc) __attribute__((always_inline)) {
            constexpr int S = decltype(sc)::value;
            const int32_t b = bset[S];
            float bv[K];
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
                bv[kk] = bias_lds[(b * GE::NB + L.q) * K + kk];
            finish_rows<G, K, F16, true>(a, L, ta, y, acc[S], bv, rows_lds[b * GE::NB + L.q],
                                         L.q + 1 < GE::NB ? rows_lds[b * GE::NB + L.q + 1] : -1, lo, hi);
            bset[S] = b + M;
        };

        int32_t it = 0, pos = 0;   // tile (round) and step within the wave's stream
        int32_t pre = 0;           // next step with tile-start, selector or need-event work
        int32_t lpos = D % len;    // stream position of the next record fetch
        Entry<K> cr[NR];
#pragma unroll
        for (int dd = 0; dd < D; ++dd)
            cr[dd] = load_entry_one<G, K>(rpr, vdelta, L.q, ws0 + dd % len);
        for (int32_t g0 = 0; g0 < total; g0 += NR) {
            static_for<NR>([&](auto kc) __attribute__((always_inline)) {
                constexpr int KI = decltype(kc)::value;
                if (g0 + KI < total) {
                    cr[(KI + D) % NR] = load_entry_one<G, K>(rpr, vdelta, L.q, ws0 + lpos);
                    lpos = lpos + 1 == len ? 0 : lpos + 1;
                    if (pos == pre) {
                        if (pos == 0) {
                            ni = ri_ = 0;
                            need = ev[0];
                            rel = ev[kMaxRegions];
                            ta.set(a, L, x, y, whole_work(a, it).tile);
#pragma unroll
                            for (int s2 = 0; s2 < M; ++s2)
                                bset[s2] = wb0 + s2;
                        }
                        if ((pos & (kSelSteps - 1)) == 0)
                            selw = sel[pos / kSelSteps];
                        while ((need >> 4) == pos) {
                            wait_fill(need & 15, nwaves * (it + 1));
                            need = ++ni < kMaxRegions ? ev[ni] : INT32_MAX;
                        }
                        pre = std::min(need >> 4, (pos | (kSelSteps - 1)) + 1);
                    }
                    // the step's set as two one-sided branches on conditions the
                    // compiler cannot relate: with an if / else it copies one
                    // set's accumulators at the join
                    uint32_t c1 = selw & 1u, c0 = c1 ^ 1u;
                    asm volatile("" : "+s"(c1), "+s"(c0));
                    if constexpr (M > 1) {
                        if (c1)
                            step(std::integral_constant<int, M - 1>{}, cr[KI]);
                    }
                    if (M == 1 || c0)
                        step(std::integral_constant<int, 0>{}, cr[KI]);
                    if constexpr (KI == 0) {
                        // shares issued one ring turn ago precede the record just used
                        if (pend) {
                            wait_vmcnt<D * LPE>();
                            publish();
                        }
                        service(false);
                    }
                    if (selw & 2u) {
                        if constexpr (M > 1) {
                            if (c1)
                                finish(std::integral_constant<int, M - 1>{});
                        }
                        if (M == 1 || c0)
                            finish(std::integral_constant<int, 0>{});
                    }
                    selw >>= 2;
                    if ((rel >> 4) == pos) {
                        do {
                            release(rel & 15);
                            rel = ++ri_ < kMaxRegions ? ev[kMaxRegions + ri_] : INT32_MAX;
                        } while ((rel >> 4) == pos);
                    }
                    if (++pos == len) {
                        pos = 0;
                        pre = 0;
                        ++it;
                    }
                }
            });
        }
    }
    // shares not issued yet (a wave without bundles issues all of its shares here)
    int32_t n_left = 0;
    for (; n_left < a.spin && ct < R; ++n_left) {
        service(true);
        __builtin_amdgcn_s_sleep(1);
    }
    if (ct < R)
        flag_wait_gave_up(a, lane);
    wait_vmcnt<0>();
    if (pend)
        publish();
    __syncthreads();  // every copy landed and every wave is done with the strip

    // ---- the shared tiles left after the whole rounds ----
    const Work wk = tail_work(a);
    if (wk.tile >= 0) {
        TileAddr<G, F16> ta;
        ta.set(a, L, x, y, wk.tile);
        copy_share<G, F16>(a, x, lds_base, wk.tile, 0, a.strip_rows, wave, nwaves, lane);
        wait_vmcnt<0>();
        __syncthreads();  // strip ready
        const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(a.idx_bytes));
        const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(a.val_bytes));
        run_item<G, K, F16, false, true>(a, L, ta, ColOff<G, F16, false>{}, y, lds, ri, rv, hdr, rank, rows_lds,
                                         bias_lds, wb0, wb1, wk.part, lo, hi);
    }
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------

using KernelFn = void (*)(const void *, void *, const int32_t *, const float *, const int32_t *, const int32_t *,
                          const int32_t *, const int32_t *, const int32_t *, const float *, const uint32_t *,
                          const int32_t *, const int32_t *, Args);

template <int K, bool F16, bool DIRECT, bool VEC, bool DWS>
KernelFn pick_g2(int g) {
    switch (g) {
    case 4:
        if constexpr (K * 4 * (16 / (F16 ? 2 : 4)) <= 64)
            return spmm_kernel<4, K, F16, DIRECT, VEC, false, DWS>;
        return nullptr;
    case 8: return spmm_kernel<8, K, F16, DIRECT, VEC, false, DWS>;
    case 16: return spmm_kernel<16, K, F16, DIRECT, VEC, false, DWS>;
    default: return nullptr;
    }
}

// dws: the plan has a depthwise stage (fp32 LDS-strip plans only)
template <int K, bool F16, bool DIRECT, bool VEC>
KernelFn pick_g(int g, bool dws = false) {
    if constexpr (!F16 && !DIRECT) {
        if (dws)
            return pick_g2<K, F16, DIRECT, VEC, true>(g);
    }
    return pick_g2<K, F16, DIRECT, VEC, false>(g);
}

// Accumulators of one set of a lane.
template <int G, int K, bool F16>
constexpr int kSetAcc = K * (16 / G) * (16 / (F16 ? 2 : 4));

template <int G, int K, bool F16>
KernelFn pick_pipe_m(int m) {
    if constexpr (kSetAcc<G, K, F16> <= 64) {
        if (m == 1)
            return spmm_pipe<G, K, F16, 1>;
        if constexpr (2 * kSetAcc<G, K, F16> <= 32) {
            if (m == 2)
                return spmm_pipe<G, K, F16, 2>;
        }
    }
    return nullptr;
}

template <int K, bool F16>
KernelFn pick_pipe(int g, int m) {
    switch (g) {
    case 4: return pick_pipe_m<4, K, F16>(m);
    case 8: return pick_pipe_m<8, K, F16>(m);
    case 16: return pick_pipe_m<16, K, F16>(m);
    default: return nullptr;
    }
}

template <int K, bool F16>
KernelFn pick_kv(const DevicePlan &p, bool vec) {
    if (p.kernel == KERNEL_DIRECT)
        return vec ? pick_g<K, F16, true, true>(p.group_lanes) : pick_g<K, F16, true, false>(p.group_lanes);
    // 1xk blocks keep the simple loop: their records take too many registers
    // for the pipelined kernel's fetch depth
    // (a depthwise stage computes the strip in the simple kernel)
    // an accumulating channel-range pass (fp32, 1x1 rows) reads Y in the simple kernel
    if constexpr (K == 1 && !F16) {
        if (p.accum) {
            switch (p.group_lanes) {
            case 4: return vec ? spmm_kernel<4, 1, false, false, true, true> : spmm_kernel<4, 1, false, false, false, true>;
            case 8: return vec ? spmm_kernel<8, 1, false, false, true, true> : spmm_kernel<8, 1, false, false, false, true>;
            case 16: return vec ? spmm_kernel<16, 1, false, false, true, true> : spmm_kernel<16, 1, false, false, false, true>;
            default: return nullptr;
            }
        }
    }
    if (p.accum)
        return nullptr;
    if (vec && K == 1 && !p.dw_stride)
        return pick_pipe<K, F16>(p.group_lanes, p.pipe_sets);
    const bool dws = p.dw_stride != 0;
    return vec ? pick_g<K, F16, false, true>(p.group_lanes, dws) : pick_g<K, F16, false, false>(p.group_lanes, dws);
}

KernelFn pick(const DevicePlan &p, bool vec) {
    if (p.k == 4)
        return p.storage == 1 ? pick_kv<4, true>(p, vec) : pick_kv<4, false>(p, vec);
    if (p.k == 2)
        return p.storage == 1 ? pick_kv<2, true>(p, vec) : pick_kv<2, false>(p, vec);
    return p.storage == 1 ? pick_kv<1, true>(p, vec) : pick_kv<1, false>(p, vec);
}

// XCDs of an MI355X: consecutive workgroups of a launch go to consecutive XCDs.
constexpr int64_t kXcds = 8;

int64_t pow2_floor(int64_t v) {
    int64_t r = 1;
    while (r * 2 <= v)
        r *= 2;
    return r;
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
    int per_cu = 1 << 30;
    for (bool vec : {false, true}) {
        KernelFn kern = pick(p, vec);
        if (!kern)
            return hipErrorInvalidValue;
        if (p.lds_bytes > 64 * 1024) {
            e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, p.lds_bytes);
            if (e != hipSuccess)
                return e;
        }
        int n = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void *>(kern), p.waves * 64,
                                                         p.lds_bytes);
        if (e != hipSuccess)
            return e;
        per_cu = std::min(per_cu, n);
    }
    if (per_cu < 1)
        return hipErrorInvalidConfiguration;
    p.blocks_per_cu = per_cu;
    return hipSuccess;
}

hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                       int64_t x_bytes, int64_t y_bytes, int32_t in_h, int32_t in_w, int32_t out_w,
                       hipStream_t stream) {
    KernelFn kern = pick(p, vec != 0);
    if (!kern)
        return hipErrorInvalidValue;
    const int64_t tc = p.tile_cols;
    const int64_t tiles = (static_cast<int64_t>(m) + tc - 1) / tc;
    const int64_t slots = static_cast<int64_t>(p.blocks_per_cu) * p.num_cus;
    if (slots < 1)
        return hipErrorInvalidConfiguration;
    // whole rounds of `slots` tiles, then each remaining tile shared by up to
    // (workgroups per XCD) / (remaining tiles per XCD) workgroups of one XCD
    // (a power of two, at most the plan's max_parts).  The grid is always
    // `slots` workgroups; those left without work leave at once.
    const int64_t nxcd = slots % kXcds == 0 ? kXcds : 1;
    const int64_t whole = tiles / slots * slots;
    const int64_t rest = tiles - whole;
    const int64_t per_xcd = (rest + nxcd - 1) / nxcd;
    const int64_t parts =
        rest ? std::max<int64_t>(1, std::min<int64_t>(pow2_floor(slots / nxcd / per_xcd), p.max_parts)) : 1;
    Args a;
    a.cin = p.cin;
    a.xc = p.xc > 0 ? p.xc : p.cin;
    a.accum = p.accum;
    a.splits = p.splits;
    a.cout = p.cout;
    a.hw = hw;
    a.m = m;
    a.act = p.act;
    a.vec = vec;
    a.strip_rows = p.strip_rows;
    a.regions = p.regions;
    a.region_rows = p.region_rows;
    a.table_off = p.kernel == KERNEL_DIRECT ? 0 : (p.strip_rows + 1) * kRowBytes;
    a.ctl_off = p.lds_bytes - kCtlBytes;
    a.nbundles = p.nbundles;
    a.busy_waves = p.busy_waves;
    a.idx_bytes = p.idx_bytes;
    a.val_bytes = p.val_bytes;
    if (p.pidx && p.pval) {
        // the pipelined kernel reads both interleaved streams through one
        // resource based at pidx
        const int64_t vdelta = reinterpret_cast<const char *>(p.pval) - reinterpret_cast<const char *>(p.pidx);
        if (vdelta < 0 || vdelta + p.val_bytes > INT32_MAX)
            return hipErrorInvalidValue;
    }
    a.x_bytes = x_bytes;
    a.y_bytes = y_bytes;
    a.tiles = static_cast<int32_t>(tiles);
    a.whole_tiles = static_cast<int32_t>(whole);
    a.tail_parts = static_cast<int32_t>(parts);
    a.nxcd = static_cast<int32_t>(nxcd);
    a.dw_stride = p.dw_stride;
    a.dw_act = p.dw_act;
    a.in_h = p.dw_stride ? in_h : 0;
    a.in_w = p.dw_stride ? in_w : 0;
    a.out_w = p.dw_stride ? out_w : 0;
    a.dw = p.dw;
    a.flag = p.flag;
    a.spin = p.spin_limit;
    a.stage_off = p.stage_off;
    a.stage_bytes = p.stage_bytes;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(slots)), dim3(p.waves * 64), p.lds_bytes, stream, x, y,
                       p.idx, p.val, p.hdr, p.table, p.rank, p.wave_ptr, p.pidx, p.pval, p.psel, p.sel_ptr,
                       p.wave_ev, a);
    return hipGetLastError();
}

}  // namespace spconv
