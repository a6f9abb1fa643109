// gfx950 (CDNA4) kernels for the sparse 1x1 convolution
//     Y[n, r, p] = act(b[r] + sum_c W[r, c] * X[n, c, p])
// (Fast Sparse ConvNets, Sec. 3.2 / Fig. 2), over NCHW tensors.
//
// Columns.  The product's dense operand has Cin rows and N*H*W columns; column
// j is (image j / HW, position j % HW).  A workgroup works on one tile of TC
// consecutive columns at a time.  A wavefront's 64 lanes form four groups of
// 16 (the four DPP rows of the wavefront); each group works on one (block)
// row, and each lane accumulates the QV columns of one VB-byte vector.  This is
// the paper's first insight (Sec. 3.2: the activations are dense, so load them
// as vectors along H*W) mapped onto wave64 lanes.
//
// Strip kernel.  The second and third insights (Sec. 3.2, Fig. 3: walk the
// output rows in the inner loop while one strip of spatial columns stays in
// the near cache, and prefetch the next strip) become:
//   * the strip X[:, tile] (Cin x TC elements) sits in LDS and compute
//     wavefronts walk their rows reading X only from there: per nonzero and
//     lane, one address add, one VB-byte LDS read and QV * K FMAs; with 1xK
//     output blocks (Sec. 3.2) one X vector feeds K rows from registers;
//   * loader wavefronts fetch the NEXT tile's strip from HBM into their
//     registers while the compute wavefronts work, and copy it into LDS
//     between two workgroup barriers (vector-memory operations of one
//     wavefront complete in order, so a compute wavefront that issued the
//     strip loads would stall its own weight loads behind them);
//   * workgroups are persistent: each takes tiles blockIdx.x, + gridDim.x, ...;
//     the tiles left over after the last whole round are shared: P workgroups
//     each take 1/P of a tile's rows, so no compute unit idles while a few
//     finish a last round alone.
//
// Weight streams.  The host planner (planner.hpp) packs each wavefront's rows
// into bundles of 4 rows (one per lane group) stored back to back, so a
// wavefront reads one continuous stream of steps (4 slots per row), kept in
// chunks of 4 steps.  Lane i of a group loads slot i of its group's 16 slots
// of a chunk -- one coalesced 4-byte load per lane for the channel offsets and
// one for the weights -- and a DPP row broadcast (row_newbcast) hands slot u
// to all 16 lanes of the group inside the instructions that use it.  So the
// weight stream costs each lane 8 (K = 1) or 20 (K = 4) bytes per 16 slots
// rather than per slot.  The main loop is a software pipeline over the stream
// that does not stop at bundle boundaries: chunks are fetched DC chunks ahead
// and X vectors read from LDS one step ahead; a scalar countdown of the
// bundle's steps triggers its epilogue (bias, activation, one rounding,
// store).  Accumulation is fp32 FMA in ascending input-channel order from
// zero; the bias is added after the sum.
//
// Direct kernel.  When Cin * TC does not fit in LDS, a simpler loop reads X
// straight from global memory (L1/L2), one tile per workgroup.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>
#include <utility>

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

// ---------------------------------------------------------------------------
// Vectors of VB bytes (16 or 8) in registers, LDS and global memory
// ---------------------------------------------------------------------------
template <int VB>
struct VecT;
template <>
struct VecT<16> {
    typedef unsigned int type __attribute__((ext_vector_type(4)));
};
template <>
struct VecT<8> {
    typedef unsigned int type __attribute__((ext_vector_type(2)));
};

template <int VB>
struct Raw {
    uint32_t w[VB / 4];
};

// X is read once and Y written once: stream them past the caches with
// non-temporal accesses, so the weight stream that every workgroup re-reads
// keeps its place in L2.
template <int VB>
__device__ __forceinline__ Raw<VB> load_stream(const void *p) {
    using V = typename VecT<VB>::type;
    const V v = __builtin_nontemporal_load(static_cast<const V *>(p));
    Raw<VB> r;
#pragma unroll
    for (int i = 0; i < VB / 4; ++i)
        r.w[i] = v[i];
    return r;
}

template <int VB>
__device__ __forceinline__ void store_stream(void *p, const Raw<VB> &r) {
    using V = typename VecT<VB>::type;
    V v;
#pragma unroll
    for (int i = 0; i < VB / 4; ++i)
        v[i] = r.w[i];
    __builtin_nontemporal_store(v, static_cast<V *>(p));
}

template <int VB>
__device__ __forceinline__ Raw<VB> lds_load(const unsigned char *lds, uint32_t byte) {
    using V = typename VecT<VB>::type;
    const V v = *reinterpret_cast<const V *>(lds + byte);
    Raw<VB> r;
#pragma unroll
    for (int i = 0; i < VB / 4; ++i)
        r.w[i] = v[i];
    return r;
}

template <int VB>
__device__ __forceinline__ void lds_store(unsigned char *lds, uint32_t byte, const Raw<VB> &r) {
    using V = typename VecT<VB>::type;
    V v;
#pragma unroll
    for (int i = 0; i < VB / 4; ++i)
        v[i] = r.w[i];
    *reinterpret_cast<V *>(lds + byte) = v;
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

// Read the QV columns of `cp` in channel c (of `ch`).  VEC promises that HW
// is a multiple of 16 bytes' worth of columns and the tensors are 16-byte
// aligned, so every run that starts before m is whole and aligned; runs past
// m read zeros.  Otherwise whole runs are read element by element from one
// base address, and runs that cross an image or the end are gathered with
// bounds checks (zeros past the end).
template <typename T, int QV, bool VEC>
__device__ __forceinline__ Raw<QV * sizeof(T)> gather(const T *__restrict__ x, const ColPos &cp, int32_t m,
                                                      int32_t hw, int32_t ch, int32_t c) {
    constexpr int VB = QV * sizeof(T);
    if constexpr (VEC) {
        Raw<VB> r = {};
        if (cp.j < m)
            r = load_stream<VB>(x + (static_cast<int64_t>(cp.img) * ch + c) * hw + cp.p);
        return r;
    } else {
        T v[QV];
        if (cp.whole) {
            const T *src = x + (static_cast<int64_t>(cp.img) * ch + c) * hw + cp.p;
#pragma unroll
            for (int e = 0; e < QV; ++e)
                v[e] = src[e];
        } else {
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
        }
        return *reinterpret_cast<const Raw<VB> *>(v);
    }
}

// Store QV columns of `cp` in output channel r (of `ch`); same cases as gather.
template <typename T, int QV, bool VEC>
__device__ __forceinline__ void scatter(T *__restrict__ y, const ColPos &cp, int32_t m, int32_t hw, int32_t ch,
                                        int32_t r, const T (&out)[QV]) {
    constexpr int VB = QV * sizeof(T);
    if constexpr (VEC) {
        if (cp.j < m)
            store_stream<VB>(y + (static_cast<int64_t>(cp.img) * ch + r) * hw + cp.p,
                             *reinterpret_cast<const Raw<VB> *>(out));
    } else if (cp.whole) {
        T *dst = y + (static_cast<int64_t>(cp.img) * ch + r) * hw + cp.p;
#pragma unroll
        for (int e = 0; e < QV; ++e)
            dst[e] = out[e];
    } else {
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

// Lane N of each 16-lane row of the wavefront, handed to every lane of that
// row (DPP row_newbcast:N).  The compiler folds it into the instruction that
// consumes the value where that instruction has a DPP form.
template <int N>
__device__ __forceinline__ int32_t row_bcast(int32_t v) {
    static_assert(N >= 0 && N < 16, "row_newbcast takes a lane of the row");
    return __builtin_amdgcn_update_dpp(0, v, 0x150 + N, 0xf, 0xf, false);
}

template <int N>
__device__ __forceinline__ float row_bcast(float v) {
    return __int_as_float(row_bcast<N>(__float_as_int(v)));
}

// FMAs whose weight comes from lane N of the 16-lane row, as v_fmac_f32 with
// the DPP broadcast on its first source.  The compiler does not form these
// itself when one broadcast value feeds several FMAs, and a separate
// v_mov_b32_dpp per weight would cost one extra VALU instruction per slot and
// weight.  Each block starts with s_nop 1: a DPP source written by a VALU
// instruction needs two wait states, and the compiler cannot see inside the
// block to insert them.
#define SPCONV_DPP(N) " row_newbcast:" #N " row_mask:0xf bank_mask:0xf\n\t"
#define SPCONV_FMAC(D, W, X, N) "v_fmac_f32_dpp %" #D ", %" #W ", %" #X SPCONV_DPP(N)

// One step of unstructured rows (K = 1, 4 fp32 columns per lane): slots
// N0..N3 of the chunk, acc[e] += w[slot] * x[slot][e], slot by slot.
#define SPCONV_STEP_K1(N0, N1, N2, N3)                                                                          \
    "s_nop 1\n\t" SPCONV_FMAC(0, 4, 5, N0) SPCONV_FMAC(1, 4, 6, N0) SPCONV_FMAC(2, 4, 7, N0)                   \
        SPCONV_FMAC(3, 4, 8, N0) SPCONV_FMAC(0, 4, 9, N1) SPCONV_FMAC(1, 4, 10, N1) SPCONV_FMAC(2, 4, 11, N1)  \
            SPCONV_FMAC(3, 4, 12, N1) SPCONV_FMAC(0, 4, 13, N2) SPCONV_FMAC(1, 4, 14, N2)                      \
                SPCONV_FMAC(2, 4, 15, N2) SPCONV_FMAC(3, 4, 16, N2) SPCONV_FMAC(0, 4, 17, N3)                  \
                    SPCONV_FMAC(1, 4, 18, N3) SPCONV_FMAC(2, 4, 19, N3) SPCONV_FMAC(3, 4, 20, N3)

template <int J>
__device__ __forceinline__ void fmac_step_k1(float (&acc)[4], float w, const Raw<16> (&xs)[4]) {
#define SPCONV_K1_ASM(N0, N1, N2, N3)                                                                           \
    asm(SPCONV_STEP_K1(N0, N1, N2, N3)                                                                          \
        : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])                                                \
        : "v"(w), "v"(xs[0].w[0]), "v"(xs[0].w[1]), "v"(xs[0].w[2]), "v"(xs[0].w[3]), "v"(xs[1].w[0]),         \
          "v"(xs[1].w[1]), "v"(xs[1].w[2]), "v"(xs[1].w[3]), "v"(xs[2].w[0]), "v"(xs[2].w[1]), "v"(xs[2].w[2]), \
          "v"(xs[2].w[3]), "v"(xs[3].w[0]), "v"(xs[3].w[1]), "v"(xs[3].w[2]), "v"(xs[3].w[3]))
    if constexpr (J == 0)
        SPCONV_K1_ASM(0, 1, 2, 3);
    else if constexpr (J == 1)
        SPCONV_K1_ASM(4, 5, 6, 7);
    else if constexpr (J == 2)
        SPCONV_K1_ASM(8, 9, 10, 11);
    else
        SPCONV_K1_ASM(12, 13, 14, 15);
#undef SPCONV_K1_ASM
}

// One slot N of 1x4 blocks (4 rows x 4 fp32 columns per lane):
// acc[r][e] += w[r] * x[e].
#define SPCONV_SLOT_K4(N)                                                                                       \
    "s_nop 1\n\t" SPCONV_FMAC(0, 16, 20, N) SPCONV_FMAC(1, 16, 21, N) SPCONV_FMAC(2, 16, 22, N)                \
        SPCONV_FMAC(3, 16, 23, N) SPCONV_FMAC(4, 17, 20, N) SPCONV_FMAC(5, 17, 21, N)                          \
            SPCONV_FMAC(6, 17, 22, N) SPCONV_FMAC(7, 17, 23, N) SPCONV_FMAC(8, 18, 20, N)                      \
                SPCONV_FMAC(9, 18, 21, N) SPCONV_FMAC(10, 18, 22, N) SPCONV_FMAC(11, 18, 23, N)                \
                    SPCONV_FMAC(12, 19, 20, N) SPCONV_FMAC(13, 19, 21, N) SPCONV_FMAC(14, 19, 22, N)           \
                        SPCONV_FMAC(15, 19, 23, N)

template <int N>
__device__ __forceinline__ void fmac_slot_k4(float (&acc)[4][4], const float (&w)[4], const Raw<16> &x) {
#define SPCONV_K4_ASM(NN)                                                                                        \
    asm(SPCONV_SLOT_K4(NN)                                                                                       \
        : "+v"(acc[0][0]), "+v"(acc[0][1]), "+v"(acc[0][2]), "+v"(acc[0][3]), "+v"(acc[1][0]), "+v"(acc[1][1]), \
          "+v"(acc[1][2]), "+v"(acc[1][3]), "+v"(acc[2][0]), "+v"(acc[2][1]), "+v"(acc[2][2]), "+v"(acc[2][3]), \
          "+v"(acc[3][0]), "+v"(acc[3][1]), "+v"(acc[3][2]), "+v"(acc[3][3])                                    \
        : "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(x.w[0]), "v"(x.w[1]), "v"(x.w[2]), "v"(x.w[3]))
    static_assert(N >= 0 && N < 16, "row_newbcast takes a lane of the row");
    switch (N) {
    case 0: SPCONV_K4_ASM(0); break;
    case 1: SPCONV_K4_ASM(1); break;
    case 2: SPCONV_K4_ASM(2); break;
    case 3: SPCONV_K4_ASM(3); break;
    case 4: SPCONV_K4_ASM(4); break;
    case 5: SPCONV_K4_ASM(5); break;
    case 6: SPCONV_K4_ASM(6); break;
    case 7: SPCONV_K4_ASM(7); break;
    case 8: SPCONV_K4_ASM(8); break;
    case 9: SPCONV_K4_ASM(9); break;
    case 10: SPCONV_K4_ASM(10); break;
    case 11: SPCONV_K4_ASM(11); break;
    case 12: SPCONV_K4_ASM(12); break;
    case 13: SPCONV_K4_ASM(13); break;
    case 14: SPCONV_K4_ASM(14); break;
    default: SPCONV_K4_ASM(15); break;
    }
#undef SPCONV_K4_ASM
}

// One lane's share of a chunk: the LDS byte offset (or channel) and the K
// weights of slot `lane % 16` of its group's 16 slots.
template <int K>
struct Chunk {
    int32_t off;
    float w[K];
};

template <int K>
__device__ __forceinline__ Chunk<K> load_chunk(Rsrc ri, Rsrc rv, int32_t lane, int32_t chunk) {
    Chunk<K> c;
    c.off = static_cast<int32_t>(bload4(ri, lane * 4, chunk * 256));
    if constexpr (K == 1) {
        c.w[0] = __uint_as_float(bload4(rv, lane * 4, chunk * 256));
    } else {
        static_assert(K == 4, "1x1 and 1x4 blocks");
        const uint4 v = bload16(rv, lane * 16, chunk * 1024);
        c.w[0] = __uint_as_float(v.x);
        c.w[1] = __uint_as_float(v.y);
        c.w[2] = __uint_as_float(v.z);
        c.w[3] = __uint_as_float(v.w);
    }
    return c;
}

// Chunks fetched ahead of their first use.  Each costs 1 + K registers.
template <int K>
struct ChunkDepth {
    static constexpr int DC = K == 1 ? 3 : 2;
    static constexpr int NR = DC + 1;  // ring entries
    static constexpr int P = 4 * NR;   // steps in one unrolled period
};

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
// Strip kernel
// ---------------------------------------------------------------------------

struct StripArgs {
    int32_t cin, cout, hw, m, act;
    int32_t cwaves;  // compute wavefronts (the rest of the workgroup loads strips)
    int32_t idx_bytes, val_bytes;
    int32_t strip_bytes, meta_words, nbundles;
    int32_t tiles;        // tiles of the launch
    int32_t whole_tiles;  // tiles processed whole: a multiple of the grid
    int32_t tail_parts;   // workgroups sharing each remaining tile (a power of two)
    int32_t nxcd;         // workgroup i runs on XCD i % nxcd; the grid is a multiple of it
};

// A workgroup's unit of work: a tile, whole (part < 0) or one of tail_parts
// parts of its rows; tile < 0 when none is left.  `round` counts the whole
// tiles (-1 for a shared one).
//
// Tiles are laid out so that the workgroups of one XCD work on neighbouring
// tiles: XCD x owns the whole tiles [x * W, (x + 1) * W), W = whole_tiles /
// nxcd, and its workgroups take them 1 per round in order.  A strip row of a
// tile rarely starts or ends on a 128-byte line, and the neighbouring tile
// needs the rest of that line: on the same XCD it finds it in L2.  All parts
// of a shared tile run on one XCD, so its strip is fetched from memory once.
struct Work {
    int32_t tile, part, round;
};

__device__ __forceinline__ Work tail_work(const StripArgs &a) {
    const int32_t b = static_cast<int32_t>(blockIdx.x);
    const int32_t x = b % a.nxcd, lb = b / a.nxcd;
    const int32_t u = x + a.nxcd * (lb / a.tail_parts);  // remaining tile of this workgroup
    if (u < a.tiles - a.whole_tiles)
        return Work{a.whole_tiles + u, a.tail_parts > 1 ? lb % a.tail_parts : -1, -1};
    return Work{-1, -1, -1};
}

__device__ __forceinline__ Work whole_work(const StripArgs &a, int32_t r) {
    const int32_t b = static_cast<int32_t>(blockIdx.x);
    const int32_t bpx = static_cast<int32_t>(gridDim.x) / a.nxcd;  // workgroups per XCD
    return Work{(b % a.nxcd) * (a.whole_tiles / a.nxcd) + r * bpx + b / a.nxcd, -1, r};
}

__device__ __forceinline__ Work first_work(const StripArgs &a) {
    return a.whole_tiles > 0 ? whole_work(a, 0) : tail_work(a);
}

__device__ __forceinline__ Work next_work(const StripArgs &a, Work w) {
    if (w.round >= 0)
        return (w.round + 1) * static_cast<int32_t>(gridDim.x) < a.whole_tiles ? whole_work(a, w.round + 1)
                                                                               : tail_work(a);
    return Work{-1, -1, -1};
}

constexpr int kLoaderVecs = 16;  // 16-byte strip vectors one loader lane holds

template <int VB, int K, bool F16, bool VEC>
__global__ void __launch_bounds__(1024)
spmm_strip(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
           const float *__restrict__ val, const int32_t *__restrict__ hdr, const int32_t *__restrict__ meta,
           const int32_t *__restrict__ wave_ptr, const int32_t *__restrict__ wave_chunk,
           const int32_t *__restrict__ split, StripArgs a) {
    using T = typename Elem<F16>::T;
    constexpr int E = sizeof(T);
    constexpr int QV = VB / E;      // columns per lane
    constexpr int TC = 16 * QV;     // columns per tile
    constexpr int ROWB = 16 * VB;   // bytes of one strip row in LDS
    constexpr int QL = 16 / E;      // columns per 16-byte loader vector
    constexpr int CPR = ROWB / 16;  // 16-byte vectors per strip row
    static_assert(64 % CPR == 0, "a loader lane must keep one column vector");

    extern __shared__ __align__(16) unsigned char lds[];
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    Work wk = first_work(a);
    if (wk.tile < 0)
        return;  // the whole workgroup leaves: no barrier is skipped by part of it

    if (wave >= a.cwaves) {
        // ----- loader wavefront -----
        const int nl = static_cast<int>(blockDim.x >> 6) - a.cwaves;
        const int ll = (wave - a.cwaves) * 64 + lane;
        const int cc = ll % CPR;          // which 16-byte vector of a strip row
        const int c0 = ll / CPR;          // first channel
        const int cstep = nl * 64 / CPR;  // channel stride between this lane's vectors
        Raw<16> pf[kLoaderVecs];
        auto fetch = [&](int t) {
            const ColPos cp = col_pos<QL>(t * TC + cc * QL, a.m, a.hw);
#pragma unroll
            for (int i = 0; i < kLoaderVecs; ++i) {
                const int c = c0 + i * cstep;
                if (c < a.cin)
                    pf[i] = gather<T, QL, VEC>(x, cp, a.m, a.hw, a.cin, c);
            }
        };
        auto deposit = [&]() {
#pragma unroll
            for (int i = 0; i < kLoaderVecs; ++i) {
                const int c = c0 + i * cstep;
                if (c < a.cin)
                    lds_store<16>(lds, c * ROWB + cc * 16, pf[i]);
            }
        };
        fetch(wk.tile);
        deposit();
        __syncthreads();  // strip(wk) ready
        for (;;) {
            const Work nx = next_work(a, wk);
            if (nx.tile >= 0)
                fetch(nx.tile);
            __syncthreads();  // compute wavefronts done with strip(wk)
            if (nx.tile < 0)
                break;
            deposit();
            __syncthreads();  // strip(nx) ready
            wk = nx;
        }
        return;
    }

    // ----- compute wavefront -----
    const int g = lane >> 4;   // lane group: one DPP row
    const int li = lane & 15;  // lane within the group
    const int32_t voff = li * VB;
    int32_t *rows_lds = reinterpret_cast<int32_t *>(lds + a.strip_bytes);
    const float *bias_lds = reinterpret_cast<const float *>(rows_lds + a.nbundles * 4);
    const int32_t *steps_lds = reinterpret_cast<const int32_t *>(bias_lds + a.nbundles * 4 * K);

    // Without loader wavefronts, every wavefront copies strips between tiles.
    const bool self_load = static_cast<int>(blockDim.x >> 6) == a.cwaves;
    auto copy_strip = [&](int t) {
        const int cc = tid % CPR;
        const int cstep = static_cast<int>(blockDim.x) / CPR;
        const ColPos cp = col_pos<QL>(t * TC + cc * QL, a.m, a.hw);
        int c = tid / CPR;
        for (; c + 3 * cstep < a.cin; c += 4 * cstep) {
            Raw<16> v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] = gather<T, QL, VEC>(x, cp, a.m, a.hw, a.cin, c + i * cstep);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                lds_store<16>(lds, (c + i * cstep) * ROWB + cc * 16, v[i]);
        }
        for (; c < a.cin; c += cstep)
            lds_store<16>(lds, c * ROWB + cc * 16, gather<T, QL, VEC>(x, cp, a.m, a.hw, a.cin, c));
    };

    const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(a.idx_bytes));
    const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(a.val_bytes));
    const int32_t wbeg = wave_ptr[wave];
    const int32_t wend = wave_ptr[wave + 1];
    const int32_t wchunk = wave_chunk[wave];

    // the bundle table into LDS (once per launch)
    for (int i = tid; i < a.meta_words; i += a.cwaves * 64)
        rows_lds[i] = meta[i];
    if (self_load)
        copy_strip(wk.tile);
    __syncthreads();  // strip(wk) and the bundle table ready

    using CD = ChunkDepth<K>;
    constexpr int DC = CD::DC, NR = CD::NR, P = CD::P;

    for (;;) {
        // this work item's bundles: all of the wavefront's, or one part of them
        int32_t b0 = wbeg, b1 = wend;
        if (wk.part >= 0) {
            const int32_t f = kMaxParts / a.tail_parts;
            b0 = split[wave * (kMaxParts + 1) + wk.part * f];
            b1 = split[wave * (kMaxParts + 1) + (wk.part + 1) * f];
        }
        if (b0 < b1) {
            const int32_t s_first = hdr[2 * b0];
            const int32_t s_end = hdr[2 * (b1 - 1)] + hdr[2 * (b1 - 1) + 1];
            // start at the chunk holding s_first; the steps before it belong to
            // an earlier bundle and are multiplied into a discarded sum
            const int32_t s_begin = s_first & ~(kChunkSteps - 1);
            const int32_t nsteps = s_end - s_begin;
            const int32_t chunk0 = wchunk + s_begin / kChunkSteps;
            const ColPos cp = col_pos<QV>(wk.tile * TC + li * QV, a.m, a.hw);

            float acc[K][QV];
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
#pragma unroll
                for (int e = 0; e < QV; ++e)
                    acc[kk][e] = 0.0f;

            // the bundle in progress: its rows and biases, and its steps left
            int32_t b = b0 - 1;
            int32_t rb = -1;
            float bv[K];
#pragma unroll
            for (int kk = 0; kk < K; ++kk)
                bv[kk] = 0.0f;
            int32_t left = s_first - s_begin;
            auto start_bundle = [&]() __attribute__((always_inline)) {
                const int mi = b * 4 + g;
                rb = rows_lds[mi];
#pragma unroll
                for (int kk = 0; kk < K; ++kk)
                    bv[kk] = bias_lds[mi * K + kk];
                left = __builtin_amdgcn_readfirstlane(steps_lds[b]);
            };
            if (left == 0) {
                b = b0;
                start_bundle();
            }
            // bias, activation, one rounding, store; then the next bundle
            auto finish_bundle = [&]() __attribute__((always_inline)) {
                if (rb >= 0) {
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) {
                        T out[QV];
#pragma unroll
                        for (int e = 0; e < QV; ++e)
                            out[e] = Elem<F16>::from_f32(activate(acc[kk][e] + bv[kk], a.act));
                        scatter<T, QV, VEC>(y, cp, a.m, a.hw, a.cout, rb * K + kk, out);
                    }
                }
#pragma unroll
                for (int kk = 0; kk < K; ++kk)
#pragma unroll
                    for (int e = 0; e < QV; ++e)
                        acc[kk][e] = 0.0f;
                ++b;
                if (b < b1)
                    start_bundle();
            };

            // X vectors of the 4 slots of step J of a chunk, at the lane's columns
            auto read_x = [&](auto jc, const Chunk<K> &ch, Raw<VB>(&xs)[4]) __attribute__((always_inline)) {
                constexpr int J = decltype(jc)::value;
                static_for<4>([&](auto uc) __attribute__((always_inline)) {
                    constexpr int U = decltype(uc)::value;
                    const uint32_t byte = static_cast<uint32_t>(row_bcast<4 * J + U>(ch.off) + voff);
                    xs[U] = lds_load<VB>(lds, byte);
                });
            };
            auto fma_step = [&](auto jc, const Chunk<K> &ch, const Raw<VB>(&xs)[4]) __attribute__((always_inline)) {
                constexpr int J = decltype(jc)::value;
                if constexpr (!F16 && VB == 16 && K == 1) {
                    fmac_step_k1<J>(acc[0], ch.w[0], xs);
                    return;
                } else if constexpr (!F16 && VB == 16 && K == 4) {
                    static_for<4>([&](auto uc) __attribute__((always_inline)) {
                        fmac_slot_k4<4 * J + decltype(uc)::value>(acc, ch.w, xs[decltype(uc)::value]);
                    });
                    return;
                }
                static_for<4>([&](auto uc) __attribute__((always_inline)) {
                    constexpr int U = decltype(uc)::value;
                    const T *xe = reinterpret_cast<const T *>(xs[U].w);
#pragma unroll
                    for (int kk = 0; kk < K; ++kk) {
                        const float w = row_bcast<4 * J + U>(ch.w[kk]);
#pragma unroll
                        for (int e = 0; e < QV; ++e)
                            acc[kk][e] = __builtin_fmaf(w, Elem<F16>::to_f32(xe[e]), acc[kk][e]);
                    }
                });
            };

            // The pipeline: a ring of NR chunks (chunk q in entry q % NR) and
            // two sets of X vectors (step s in set s % 2); the stage loop is
            // unrolled over P = 4 * NR steps so every index is a constant.
            // Chunks fetched past the stream's end hold other wavefronts' data
            // or zeros (buffer bounds) and are never multiplied in.
            Chunk<K> cr[NR];
            Raw<VB> xr[2][4];
#pragma unroll
            for (int q = 0; q < DC; ++q)
                cr[q] = load_chunk<K>(ri, rv, lane, chunk0 + q);
            read_x(std::integral_constant<int, 0>{}, cr[0], xr[0]);

            int32_t s0 = 0;
            auto stage = [&](auto kc) __attribute__((always_inline)) {
                constexpr int KI = decltype(kc)::value;  // step within the period
                constexpr int J = KI % 4, Q = KI / 4;
                constexpr int KN = KI + 1, JN = KN % 4, QN = (KN / 4) % NR;
                if constexpr (J == 0)
                    cr[(Q + DC) % NR] = load_chunk<K>(ri, rv, lane, chunk0 + s0 / 4 + Q + DC);
                read_x(std::integral_constant<int, JN>{}, cr[QN], xr[KN % 2]);
                __builtin_amdgcn_sched_barrier(0);
                fma_step(std::integral_constant<int, J>{}, cr[Q], xr[KI % 2]);
                if (--left == 0)
                    finish_bundle();
            };
            // one copy of the unrolled period; each step is guarded by a
            // scalar test, and the single-exit loop keeps its bounds scalar
            for (; s0 < nsteps; s0 += P)
                static_for<P>([&](auto kc) __attribute__((always_inline)) {
                    if (s0 + decltype(kc)::value < nsteps)
                        stage(kc);
                });
        }

        const Work nx = next_work(a, wk);
        __syncthreads();  // done with strip(wk)
        if (nx.tile < 0)
            break;
        if (self_load)
            copy_strip(nx.tile);
        __syncthreads();  // strip(nx) ready
        wk = nx;
    }
}

// ---------------------------------------------------------------------------
// Direct kernel: X read from global memory, one tile per workgroup.
// ---------------------------------------------------------------------------

struct DirectArgs {
    int32_t cin, cout, hw, m, act;
    int32_t idx_bytes, val_bytes, nbundles;
};

template <int K, bool F16, bool VEC>
__global__ void __launch_bounds__(1024)
spmm_direct(const void *__restrict__ xv, void *__restrict__ yv, const int32_t *__restrict__ idx,
            const float *__restrict__ val, const int32_t *__restrict__ hdr, const int32_t *__restrict__ meta,
            const int32_t *__restrict__ wave_ptr, const int32_t *__restrict__ wave_chunk, DirectArgs a) {
    using T = typename Elem<F16>::T;
    constexpr int QV = 16 / sizeof(T);
    constexpr int TC = 16 * QV;
    const T *__restrict__ x = static_cast<const T *>(xv);
    T *__restrict__ y = static_cast<T *>(yv);
    const int32_t *rows = meta;
    const float *bias = reinterpret_cast<const float *>(meta + a.nbundles * 4);

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int g = lane >> 4;
    const int li = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ColPos cp = col_pos<QV>(static_cast<int32_t>(blockIdx.x) * TC + li * QV, a.m, a.hw);
    const Rsrc ri = make_rsrc(idx, static_cast<uint32_t>(a.idx_bytes));
    const Rsrc rv = make_rsrc(val, static_cast<uint32_t>(a.val_bytes));
    const int32_t wchunk = wave_chunk[wave];

    for (int b = wave_ptr[wave]; b < wave_ptr[wave + 1]; ++b) {
        const int32_t s_first = hdr[2 * b];
        const int32_t n = hdr[2 * b + 1];
        float acc[K][QV];
#pragma unroll
        for (int kk = 0; kk < K; ++kk)
#pragma unroll
            for (int e = 0; e < QV; ++e)
                acc[kk][e] = 0.0f;
        for (int t = 0; t < n; ++t) {
            const int32_t s = s_first + t;
            const int32_t chunk = wchunk + s / kChunkSteps;
            const int32_t slot0 = 16 * g + 4 * (s % kChunkSteps);  // this group's step within the chunk
            const uint4 c4 = bload16(ri, slot0 * 4, chunk * 256);
            const int32_t cu[4] = {static_cast<int32_t>(c4.x), static_cast<int32_t>(c4.y),
                                   static_cast<int32_t>(c4.z), static_cast<int32_t>(c4.w)};
            float w[4][K];
            if constexpr (K == 1) {
                const uint4 w4 = bload16(rv, slot0 * 4, chunk * 256);
                w[0][0] = __uint_as_float(w4.x);
                w[1][0] = __uint_as_float(w4.y);
                w[2][0] = __uint_as_float(w4.z);
                w[3][0] = __uint_as_float(w4.w);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const uint4 w4 = bload16(rv, (slot0 + u) * 16, chunk * 1024);
                    w[u][0] = __uint_as_float(w4.x);
                    w[u][1] = __uint_as_float(w4.y);
                    w[u][2] = __uint_as_float(w4.z);
                    w[u][3] = __uint_as_float(w4.w);
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const Raw<16> raw = gather<T, QV, VEC>(x, cp, a.m, a.hw, a.cin, cu[u]);
                const T *xe = reinterpret_cast<const T *>(raw.w);
#pragma unroll
                for (int e = 0; e < QV; ++e) {
                    const float xf = Elem<F16>::to_f32(xe[e]);
#pragma unroll
                    for (int kk = 0; kk < K; ++kk)
                        acc[kk][e] = __builtin_fmaf(w[u][kk], xf, acc[kk][e]);
                }
            }
        }
        const int rb = rows[b * 4 + g];
        if (rb < 0)
            continue;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) {
            const float bv = bias[(b * 4 + g) * K + kk];
            T out[QV];
#pragma unroll
            for (int e = 0; e < QV; ++e)
                out[e] = Elem<F16>::from_f32(activate(acc[kk][e] + bv, a.act));
            scatter<T, QV, VEC>(y, cp, a.m, a.hw, a.cout, rb * K + kk, out);
        }
    }
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------

template <int VB, int K, bool F16>
hipError_t prepare_strip(DevicePlan &p) {
    const void *kerns[2] = {reinterpret_cast<const void *>(spmm_strip<VB, K, F16, false>),
                            reinterpret_cast<const void *>(spmm_strip<VB, K, F16, true>)};
    const int threads = (p.waves + p.loader_waves) * 64;
    int per_cu = 1 << 30;
    for (const void *kern : kerns) {
        if (p.lds_bytes > 64 * 1024) {
            hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, p.lds_bytes);
            if (e != hipSuccess)
                return e;
        }
        int n = 0;
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kern, threads, p.lds_bytes);
        if (e != hipSuccess)
            return e;
        per_cu = std::min(per_cu, n);
    }
    if (per_cu < 1)
        return hipErrorInvalidConfiguration;
    p.blocks_per_cu = per_cu;
    return hipSuccess;
}

// XCDs of an MI355X: consecutive workgroups of a launch go to consecutive XCDs.
constexpr int64_t kXcds = 8;

int64_t pow2_floor(int64_t v) {
    int64_t r = 1;
    while (r * 2 <= v)
        r *= 2;
    return r;
}

template <int VB, int K, bool F16>
hipError_t launch_strip(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                        hipStream_t stream) {
    constexpr int TC = 16 * VB / (F16 ? 2 : 4);
    const int threads = (p.waves + p.loader_waves) * 64;
    const int64_t tiles = (static_cast<int64_t>(m) + TC - 1) / TC;
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
    const int64_t grid = slots;
    StripArgs a;
    a.cin = p.cin;
    a.cout = p.cout;
    a.hw = hw;
    a.m = m;
    a.act = p.act;
    a.cwaves = p.waves;
    a.idx_bytes = p.idx_bytes;
    a.val_bytes = p.val_bytes;
    a.strip_bytes = p.strip_bytes;
    a.meta_words = p.meta_words;
    a.nbundles = p.nbundles;
    a.tiles = static_cast<int32_t>(tiles);
    a.whole_tiles = static_cast<int32_t>(whole);
    a.tail_parts = static_cast<int32_t>(parts);
    a.nxcd = static_cast<int32_t>(nxcd);
    if (vec)
        hipLaunchKernelGGL((spmm_strip<VB, K, F16, true>), dim3(static_cast<unsigned>(grid)), dim3(threads),
                           p.lds_bytes, stream, x, y, p.idx, p.val, p.hdr, p.meta, p.wave_ptr, p.wave_chunk, p.split,
                           a);
    else
        hipLaunchKernelGGL((spmm_strip<VB, K, F16, false>), dim3(static_cast<unsigned>(grid)), dim3(threads),
                           p.lds_bytes, stream, x, y, p.idx, p.val, p.hdr, p.meta, p.wave_ptr, p.wave_chunk, p.split,
                           a);
    return hipGetLastError();
}

template <int K, bool F16>
hipError_t launch_direct(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                         hipStream_t stream) {
    constexpr int TC = 16 * 16 / (F16 ? 2 : 4);
    const int64_t tiles = (static_cast<int64_t>(m) + TC - 1) / TC;
    DirectArgs a;
    a.cin = p.cin;
    a.cout = p.cout;
    a.hw = hw;
    a.m = m;
    a.act = p.act;
    a.idx_bytes = p.idx_bytes;
    a.val_bytes = p.val_bytes;
    a.nbundles = p.nbundles;
    if (vec)
        hipLaunchKernelGGL((spmm_direct<K, F16, true>), dim3(static_cast<unsigned>(tiles)), dim3(p.waves * 64), 0,
                           stream, x, y, p.idx, p.val, p.hdr, p.meta, p.wave_ptr, p.wave_chunk, a);
    else
        hipLaunchKernelGGL((spmm_direct<K, F16, false>), dim3(static_cast<unsigned>(tiles)), dim3(p.waves * 64), 0,
                           stream, x, y, p.idx, p.val, p.hdr, p.meta, p.wave_ptr, p.wave_chunk, a);
    return hipGetLastError();
}

template <int K, bool F16>
hipError_t prepare(DevicePlan &p) {
    if (p.kernel == KERNEL_DIRECT)
        return hipSuccess;
    switch (p.vec_bytes) {
    case 16: return prepare_strip<16, K, F16>(p);
    case 8: return prepare_strip<8, K, F16>(p);
    default: return hipErrorInvalidValue;
    }
}

template <int K, bool F16>
hipError_t dispatch(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                    hipStream_t s) {
    if (p.kernel == KERNEL_DIRECT)
        return launch_direct<K, F16>(p, x, y, m, hw, vec, s);
    switch (p.vec_bytes) {
    case 16: return launch_strip<16, K, F16>(p, x, y, m, hw, vec, s);
    case 8: return launch_strip<8, K, F16>(p, x, y, m, hw, vec, s);
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
