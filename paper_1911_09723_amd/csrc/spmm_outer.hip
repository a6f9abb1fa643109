// Outer-product kernel for 1 x 4 blocks on the matrix cores (format in
// planner.hpp, "Outer-product kernel").
//
// The paper's 1 x k output-channel blocks (Sec. 3.2) let one X value feed k
// output rows from registers.  For k = 4 that product, one stored block times
// one X vector of 4 columns, is a 4 x 4 outer product, and the fp32 4x4x1
// matrix instruction computes 16 of them per wavefront, each lane block of 4
// lanes with its own operands: lane 4b + t supplies weight t of its block (A)
// and the X value of its column (B), and its accumulator register r becomes
// A[4b + r] * B[4b + t] + C with a single rounding.  On MI355X that costs
// about as much issue time as 3 wave-wide VALU FMAs while doing the work of 4,
// and it needs no per-row register indexing, because every lane group carries
// its own block row.
//
// Work layout.  A workgroup of `waves` wavefronts owns tiles of 32 columns,
// round-robin over the grid (XCD-aware).  A tile's X rows sit in one of two
// LDS buffers; a wavefront walks the octs (8 block rows) the planner gave it
// for that tile parity: per step, group g (8 lanes) reads the 16-byte vector
// of its block's channel row and issues 4 matrix instructions, one per column
// of the vector.  Weights come from global memory, one 16-byte load per lane
// per 4 steps; the channel-row offsets from the workgroup's LDS copy of the
// offset table (global memory when it does not fit).
//
// Refills.  The last wavefront to leave a buffer publishes the tile it takes
// next; each wavefront copies its share of that tile at its next check and
// counts it as landed at the check after (Refill below).  fp32 input with
// H*W a multiple of 4 is copied by 16-byte global-to-LDS loads; fp16 input
// (converted to fp32 on the way) and H*W not a multiple of 4 (4-column
// vectors that straddle two images, read element by element) go through
// registers, kStageMax instructions per phase.  A wavefront starts a tile
// once every share of it has been counted: a bounded wait that sets the
// plan's error word if it gives up.  fp16 output is rounded once, to nearest
// even, after the bias and the activation.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "launch.hpp"

namespace spconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef unsigned int u2 __attribute__((ext_vector_type(2)));

struct OArgs {
    const void *x;
    void *y;
    const float *bias;  // every output channel
    const f4 *rec;      // weights, 16 bytes per (quad, slot)
    const i4 *off;      // channel-row offsets, 16 bytes per (quad, group)
    int32_t off_bytes;  // size of the offset table (with its read-ahead quads)
    int32_t off_lds;    // LDS byte address of its copy (table in LDS), else -1
    const int32_t *oct;
    const int32_t *wave_ptr;
    const int32_t *wave_oct;
    int32_t *flag;  // the plan's error word: bit 0 set when a bounded wait gives up
    int32_t spin;   // bound of every wait (sleeps)
    int32_t cin, cout, hw, m, act;
    int32_t ntiles, grid, nx;  // tiles, workgroups, XCD groups of the tile map (grid % nx == 0)
    int32_t rounds, rem;       // whole rounds of the grid, tiles left after them
    int32_t parts;             // workgroups sharing each of those tiles (grid / rem when at least 2, else 1)
    int32_t noct;
    int32_t waves, ozrow, buf_bytes;
    int32_t ctl_off;  // LDS byte address of the control words
    int64_t x_bytes;
};

// LDS control words after the buffers (and the offset table), per buffer:
// wavefronts done with it, copy shares of it landed (one per wavefront per
// tile), and the tile sequence number it is free to take next (set by the
// last wavefront out).
constexpr int kCtlRel = 0, kCtlFill = 2, kCtlFree = 4, kCtlWords = 6;
// Copy instructions a wavefront holds in registers per phase (staged copies):
// 4 with one load per lane each, 2 with 4 element loads each.
template <bool VEC>
constexpr int stage_max() { return VEC ? 4 : 2; }

// Geometry of a mode (0 matrix, 1 vector) and tile width TW: lanes per group
// (4 columns each), groups per wavefront, bytes per LDS row, rows per 1 KB
// copy instruction, weight slots per group and per quad.
template <int MODE, int TW>
struct LGeo {
    static constexpr int LPG = TW / 4;
    static constexpr int G = 64 / LPG;
    static constexpr int RB = TW * 4;
    static constexpr int RPI = 1024 / RB;
    static constexpr int KW = MODE == 0 ? 4 : 1;
    static constexpr int SLOTS = G * KW;
};
constexpr int32_t kOutOfRange = static_cast<int32_t>(0x80000000u);
constexpr int64_t kMaxRecords = 0x7ffffff0;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt takes 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

__device__ __forceinline__ i4 rsrc_words(const void *p, int64_t bytes) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    i4 r;
    r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(v));
    r.y = __builtin_amdgcn_readfirstlane(static_cast<int>((v >> 32) & 0xffff));
    r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes < kMaxRecords ? bytes : kMaxRecords));
    r.w = 0x00020000;
    return r;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0),
                                             static_cast<int>(bytes < kMaxRecords ? bytes : kMaxRecords),
                                             0x00020000);
}

// Workgroup wg's position in the tile map: XCD x (= wg % nx) takes the
// neighbouring tiles x * (grid / nx) .. of every round, so the 128-byte lines
// two neighbouring tiles share meet in one L2.
__device__ __forceinline__ int32_t tile_slot(const OArgs &a, int32_t wg) {
    return (wg % a.nx) * (a.grid / a.nx) + wg / a.nx;
}

// Tile of workgroup position `slot` at its k-th tile: one per whole round,
// then, of the tiles left, the one its group of `parts` neighbouring
// positions (one XCD) shares, each position taking every parts-th oct.
__device__ __forceinline__ int32_t tile_of(const OArgs &a, int32_t slot, int32_t k) {
    return k < a.rounds ? k * a.grid + slot : a.rounds * a.grid + slot / a.parts;
}

__device__ __forceinline__ int32_t tiles_of(const OArgs &a, int32_t slot) {
    return a.rounds + (a.rem > 0 && slot / a.parts < a.rem ? 1 : 0);
}

// The 4 columns of lane vector (lane % (TW / 4)) of a tile, counted from channel 0
// of the tile's first image n0 (the images one tile touches span less than
// 2^31 bytes): X byte offsets (kOutOfRange past the last column) and Y
// element offsets from ybase (-1 past it).  With VEC the 4 columns lie in one
// image and only element 0 is kept.
template <int TW, bool F16, bool VEC>
struct Cols {
    static constexpr int NE = VEC ? 1 : 4;
    int32_t n0;
    int64_t ybase;
    int32_t xo[NE];
    int32_t yo[NE];
    __device__ __forceinline__ void set(const OArgs &a, int32_t tile, int lane) {
        constexpr int E = F16 ? 2 : 4;
        const int32_t col0 = tile * TW;
        n0 = col0 / a.hw;
        ybase = static_cast<int64_t>(n0) * a.cout * a.hw;
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int32_t c = col0 + (lane % (TW / 4)) * 4 + e;
            const int32_t n = c / a.hw;
            const int32_t p = c - n * a.hw;
            xo[e] = c < a.m ? ((n - n0) * a.cin * a.hw + p) * E : kOutOfRange;
            yo[e] = c < a.m ? (n - n0) * a.cout * a.hw + p : -1;
        }
    }
};

__device__ __forceinline__ int32_t lds_load_acquire(const int32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ f4 lds_vec(const unsigned char *lds, uint32_t byte) {
    return *reinterpret_cast<const f4 *>(lds + byte);
}

// A wavefront's part in filling the two buffers.  Copy instruction i of a
// tile moves channel rows 8i .. 8i + 7 (lane l: row 8i + l / 8, the 4 columns
// of vector l % 8) to LDS bytes buf + 1024 i + 16 l, as fp32; channels past
// cin and columns past m give zeros.  A wavefront's share of a tile is
// instructions wave, wave + waves, ...; it starts the share when it sees the
// buffer freed for that tile, and once its last copy has landed adds one to
// the buffer's fill count.  One share (or one phase of a staged share) is in
// flight at a time.  Checks inside an oct come after at least N newer loads,
// and loads complete in order, so a wait for vmcnt <= N finds the copies done.
template <int TW, bool DMA, bool F16, bool VEC>
struct Refill {
    using GE = LGeo<1, TW>;  // copy geometry (the same in both modes)
    int32_t issued0, issued1;  // sequence number of the last tile whose share this wave started, per buffer
    int32_t sb;         // buffer of the copy in flight, -1 for none
    int32_t sk;         // its tile sequence number
    int32_t sfirst;     // first share instruction of the phase in flight (staged)
    int32_t sn;         // instructions in it (staged)
    static constexpr int kStageMax = stage_max<VEC>();
    uint32_t st[kStageMax][4];

    __device__ __forceinline__ void start(const OArgs &a, int32_t slot, int wave, int lane, int b, int32_t k,
                                          int32_t first) {
        sb = b;
        sk = k;
        sfirst = first;
        const int ninstr = a.ozrow / GE::RPI;
        Cols<TW, F16, VEC> cols;
        cols.set(a, tile_of(a, slot, k), lane);
        constexpr int E = F16 ? 2 : 4;
        const int64_t xbase = static_cast<int64_t>(cols.n0) * a.cin * a.hw;
        const int32_t crow = lane / GE::LPG;
        const int32_t step = GE::RPI * a.hw * E;
        if constexpr (DMA) {
            const i4 rs = rsrc_words(static_cast<const float *>(a.x) + xbase, a.x_bytes - xbase * 4);
            const int32_t lo = cols.xo[0] == kOutOfRange ? kOutOfRange : cols.xo[0] + crow * a.hw * 4;
            const uint32_t buf = b * a.buf_bytes;
            for (int i = wave; i < ninstr; i += a.waves) {
                const int32_t voff = lo != kOutOfRange && GE::RPI * i + crow < a.cin ? lo + i * step : kOutOfRange;
                const uint32_t m0 = __builtin_amdgcn_readfirstlane(buf + 1024 * i);
                asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                             :
                             : "s"(m0), "v"(voff), "s"(rs)
                             : "memory", "m0");
            }
        } else {
            const auto rs = make_rsrc(static_cast<const unsigned char *>(a.x) + xbase * E, a.x_bytes - xbase * E);
            sn = 0;
#pragma unroll
            for (int s = 0; s < kStageMax; ++s) {
                const int i = wave + (first + s) * a.waves;
                if (i < ninstr) {
                    const bool row_ok = GE::RPI * i + crow < a.cin;
                    const int32_t ro = (GE::RPI * i + crow) * a.hw * E;
                    if constexpr (VEC) {
                        const int32_t o = row_ok && cols.xo[0] != kOutOfRange ? cols.xo[0] + ro : kOutOfRange;
                        if constexpr (F16) {
                            const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs, o, 0, 0);
                            st[s][0] = v[0];
                            st[s][1] = v[1];
                        } else {
                            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rs, o, 0, 0);
                            st[s][0] = v[0];
                            st[s][1] = v[1];
                            st[s][2] = v[2];
                            st[s][3] = v[3];
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int32_t o = row_ok && cols.xo[e] != kOutOfRange ? cols.xo[e] + ro : kOutOfRange;
                            if constexpr (F16)
                                st[s][e] = __builtin_amdgcn_raw_buffer_load_b16(rs, o, 0, 0);
                            else
                                st[s][e] = __builtin_amdgcn_raw_buffer_load_b32(rs, o, 0, 0);
                        }
                    }
                    sn = s + 1;
                }
            }
        }
    }
    // The copy in flight has completed: write a staged phase to LDS, then start
    // the share's next phase or count the share as landed.
    __device__ __forceinline__ void advance(const OArgs &a, unsigned char *lds, int32_t *ctl, int32_t slot,
                                            int wave, int lane) {
        if constexpr (!DMA) {
            const uint32_t buf = sb * a.buf_bytes;
#pragma unroll
            for (int s = 0; s < kStageMax; ++s) {
                if (s < sn) {
                    const int i = wave + (sfirst + s) * a.waves;
                    f4 v;
                    if constexpr (F16) {
                        uint32_t h[4];
                        if constexpr (VEC) {
                            h[0] = st[s][0] & 0xffff;
                            h[1] = st[s][0] >> 16;
                            h[2] = st[s][1] & 0xffff;
                            h[3] = st[s][1] >> 16;
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                h[e] = st[s][e];
                        }
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            v[e] = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h[e])));
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            v[e] = __uint_as_float(st[s][e]);
                    }
                    *reinterpret_cast<f4 *>(lds + buf + 1024 * i + 16 * lane) = v;
                }
            }
            if (wave + (sfirst + sn) * a.waves < a.ozrow / GE::RPI) {
                start(a, slot, wave, lane, sb, sk, sfirst + sn);
                return;
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the LDS writes are done
        }
        if (lane == 0)
            __hip_atomic_fetch_add(&ctl[kCtlFill + sb], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        sb = -1;
    }
    // Start this wave's share of a tile a buffer was freed for, if any (one at a time).
    __device__ __forceinline__ void try_start(const OArgs &a, int32_t *ctl, int32_t slot, int wave, int lane) {
        if (sb >= 0)
            return;
        const int32_t g0 = __builtin_amdgcn_readfirstlane(lds_load_acquire(&ctl[kCtlFree + 0]));
        if (g0 > issued0) {
            issued0 = g0;
            start(a, slot, wave, lane, 0, g0, 0);
            return;
        }
        const int32_t g1 = __builtin_amdgcn_readfirstlane(lds_load_acquire(&ctl[kCtlFree + 1]));
        if (g1 > issued1) {
            issued1 = g1;
            start(a, slot, wave, lane, 1, g1, 0);
        }
    }
    // Inside an oct, at least N loads after the copy in flight was issued.
    template <int N>
    __device__ __forceinline__ void check(const OArgs &a, unsigned char *lds, int32_t *ctl, int32_t slot, int wave,
                                          int lane) {
        if (sb >= 0) {
            wait_vmcnt<N>();
            advance(a, lds, ctl, slot, wave, lane);
        }
        try_start(a, ctl, slot, wave, lane);
    }
    // Before tile k in buffer bw: finish the copy in flight, and this wave's
    // whole share of tile k once the buffer is free for it; then start
    // whatever else is free.
    __device__ __forceinline__ void flush(const OArgs &a, unsigned char *lds, int32_t *ctl, int32_t slot, int wave,
                                          int lane, int bw, int32_t k) {
        for (;;) {
            if (sb >= 0) {
                wait_vmcnt<0>();
                advance(a, lds, ctl, slot, wave, lane);
                continue;
            }
            if ((bw ? issued1 : issued0) < k) {
                const int32_t g = __builtin_amdgcn_readfirstlane(lds_load_acquire(&ctl[kCtlFree + bw]));
                if (g >= k) {
                    if (bw)
                        issued1 = g;
                    else
                        issued0 = g;
                    start(a, slot, wave, lane, bw, g, 0);
                    continue;
                }
            }
            break;
        }
        try_start(a, ctl, slot, wave, lane);
    }
};

// One group set on the tile in the buffer at byte `buf`: lockstep steps,
// then bias, activation and stores of the lane's rows (matrix: 4, vector: 1)
// and 4 columns.  OFF_LDS: the channel-row offsets come from the
// workgroup's LDS copy of the table, else from global memory.
template <int MODE, int TW, bool OFF_LDS, bool DMA, bool F16, bool VEC>
__device__ __forceinline__ void run_oct(const OArgs &a, unsigned char *lds, int32_t o, uint32_t buf,
                                        const Cols<TW, F16, VEC> &cols, float lo, float hi, int lane, int32_t *ctl,
                                        Refill<TW, DMA, F16, VEC> &rf, int32_t slot, int wave) {
    using GE = LGeo<MODE, TW>;
    const int32_t *tab = a.oct + o * kOctWords;
    const int32_t q0 = __builtin_amdgcn_readfirstlane(tab[0]);
    const int32_t nq = __builtin_amdgcn_readfirstlane(tab[1]);
    const int g = lane / GE::LPG;
    const int32_t rb = tab[2 + g];
    const int wslot = MODE == 0 ? g * 4 + (lane & 3) : g;
    const f4 *wp = a.rec + (static_cast<int64_t>(q0) * GE::SLOTS + wslot);
    const int64_t og = static_cast<int64_t>(q0) * GE::G + g;  // (quad, group) index of the offsets
    auto offs = [&](int32_t j) -> i4 {
        if constexpr (OFF_LDS)
            return *reinterpret_cast<const i4 *>(lds + a.off_lds + (og + int64_t(j) * GE::G) * 16);
        else
            return a.off[og + int64_t(j) * GE::G];
    };
    const uint32_t xl = buf + (lane % GE::LPG) * 16;
    f4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0, acc2 = acc0, acc3 = acc0;
    auto mma = [&](float w, const f4 x) {
        if constexpr (MODE == 0) {
            acc0 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.x, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.y, acc1, 0, 0, 0);
            acc2 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.z, acc2, 0, 0, 0);
            acc3 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.w, acc3, 0, 0, 0);
        } else {
            // fused multiply-adds kept in program order (volatile): otherwise
            // the compiler sinks them below the refill checks and holds every
            // X vector of several quads in registers
            asm volatile("v_fmac_f32 %0, %4, %5\n\tv_fmac_f32 %1, %4, %6\n\tv_fmac_f32 %2, %4, %7\n\t"
                         "v_fmac_f32 %3, %4, %8"
                         : "+v"(acc0.x), "+v"(acc0.y), "+v"(acc0.z), "+v"(acc0.w)
                         : "v"(w), "v"(x.x), "v"(x.y), "v"(x.z), "v"(x.w));
        }
    };
    auto xrow = [&](int32_t off) { return lds_vec(lds, xl + static_cast<uint32_t>(off)); };
    // Software pipeline: weights and channel-row offsets kOuterAhead quads
    // ahead in registers (the arrays are padded for it; the offsets of the
    // widest layers come from global memory, so they need the same lead as
    // the weights).  Each step's X vector is read XA steps before its
    // arithmetic, from a ring of four register sets (one per step of the
    // quad): vector mode reads three steps ahead, which covers the LDS
    // latency with the fused multiply-adds of the three steps in between;
    // matrix mode reads one step ahead (its matrix instructions already cover
    // the latency; a deeper ring only costs registers there).
    constexpr int XA = MODE == 1 ? 3 : 1;
    f4 wq[kOuterAhead];
    i4 oqs[kOuterAhead];
#pragma unroll
    for (int i = 0; i < kOuterAhead; ++i) {
        wq[i] = wp[i * GE::SLOTS];
        oqs[i] = offs(i);
    }
    wp += kOuterAhead * GE::SLOTS;
    f4 xs[4];
#pragma unroll
    for (int t = 0; t < XA; ++t)
        xs[t] = xrow(oqs[0][t]);
    // one quad (offsets oq): its 4 steps; step t reads the X vector of step
    // t + XA (in the next quad, offsets nx, once t + XA passes 3)
    auto quad = [&](const f4 w, const i4 oq, const i4 nx) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = t + XA;
            xs[r % 4] = xrow(r < 4 ? oq[r] : nx[r - 4]);
            __builtin_amdgcn_sched_barrier(0);
            mma(w[t], xs[t]);
        }
    };
    int32_t j = 0;
    for (; j + kOuterAhead <= nq; j += kOuterAhead) {
#pragma unroll
        for (int i = 0; i < kOuterAhead; ++i) {
            quad(wq[i], oqs[i], oqs[(i + 1) % kOuterAhead]);
            // after their last use: no copies of the old records
            wq[i] = wp[i * GE::SLOTS];
            oqs[i] = offs(j + i + kOuterAhead);
            __builtin_amdgcn_sched_barrier(0);
        }
        wp += kOuterAhead * GE::SLOTS;
        // loads since the last check: kOuterAhead weight loads (and as many offset loads)
        rf.template check<OFF_LDS ? kOuterAhead : 2 * kOuterAhead>(a, lds, ctl, slot, wave, lane);
    }
#pragma unroll
    for (int i = 0; i < kOuterAhead - 1; ++i)
        if (j + i < nq)
            quad(wq[i], oqs[i], oqs[i + 1]);
    if (rb < 0)
        return;
    constexpr int NR = MODE == 0 ? 4 : 1;  // rows of this lane
    float bz[NR];
    if constexpr (MODE == 0) {
        const f4 b4 = *reinterpret_cast<const f4 *>(a.bias + 4 * rb);
        bz[0] = b4.x;
        bz[1] = b4.y;
        bz[2] = b4.z;
        bz[3] = b4.w;
    } else {
        bz[0] = a.bias[rb];
    }
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        f4 v;
        if constexpr (MODE == 0) {
            v.x = fminf(fmaxf(acc0[r] + bz[r], lo), hi);
            v.y = fminf(fmaxf(acc1[r] + bz[r], lo), hi);
            v.z = fminf(fmaxf(acc2[r] + bz[r], lo), hi);
            v.w = fminf(fmaxf(acc3[r] + bz[r], lo), hi);
        } else {
            v.x = fminf(fmaxf(acc0.x + bz[0], lo), hi);
            v.y = fminf(fmaxf(acc0.y + bz[0], lo), hi);
            v.z = fminf(fmaxf(acc0.z + bz[0], lo), hi);
            v.w = fminf(fmaxf(acc0.w + bz[0], lo), hi);
        }
        const int32_t ro = (NR * rb + r) * a.hw;
        if constexpr (VEC) {
            if (cols.yo[0] >= 0) {
                if constexpr (F16) {
                    u2 h;
                    h.x = __builtin_bit_cast(uint16_t, static_cast<_Float16>(v.x)) |
                          static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(v.y))) << 16;
                    h.y = __builtin_bit_cast(uint16_t, static_cast<_Float16>(v.z)) |
                          static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(v.w))) << 16;
                    *reinterpret_cast<u2 *>(static_cast<_Float16 *>(a.y) + cols.ybase + (cols.yo[0] + ro)) = h;
                } else {
                    *reinterpret_cast<f4 *>(static_cast<float *>(a.y) + cols.ybase + (cols.yo[0] + ro)) = v;
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (cols.yo[e] >= 0) {
                    if constexpr (F16)
                        static_cast<_Float16 *>(a.y)[cols.ybase + (cols.yo[e] + ro)] = static_cast<_Float16>(v[e]);
                    else
                        static_cast<float *>(a.y)[cols.ybase + (cols.yo[e] + ro)] = v[e];
                }
        }
    }
}

template <int MODE, int TW, bool OFF_LDS, bool F16, bool VEC>
__global__ void __launch_bounds__(1024) outer_kernel(OArgs a) {
    using GE = LGeo<MODE, TW>;
    constexpr bool DMA = !F16 && VEC;
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int32_t slot = tile_slot(a, blockIdx.x);
    const int32_t nt = tiles_of(a, slot);
    if (nt == 0)
        return;
    int32_t *ctl = reinterpret_cast<int32_t *>(lds + a.ctl_off);
    // zero rows of both buffers; control words: buffer 0 free for tile 0,
    // buffer 1 for tile 1; the offset table
    if (threadIdx.x < 2 * GE::LPG) {
        const int b = threadIdx.x / GE::LPG;
        *reinterpret_cast<f4 *>(lds + b * a.buf_bytes + a.ozrow * GE::RB + (threadIdx.x % GE::LPG) * 16) =
            f4{0.f, 0.f, 0.f, 0.f};
    }
    if (threadIdx.x < kCtlWords)
        ctl[threadIdx.x] = threadIdx.x == kCtlFree ? 0 : threadIdx.x == kCtlFree + 1 ? (nt > 1 ? 1 : -1) : 0;
    if constexpr (OFF_LDS) {
        // 1 KB per instruction (reads past the table's end give zeros)
        const i4 rs = rsrc_words(a.off, a.off_bytes);
        for (int i = wave; i < (a.off_bytes + 1023) / 1024; i += a.waves) {
            const uint32_t m0 = __builtin_amdgcn_readfirstlane(a.off_lds + 1024 * i);
            asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                         :
                         : "s"(m0), "v"(1024 * i + lane * 16), "s"(rs)
                         : "memory", "m0");
        }
        wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): zero rows and control words written
    __syncthreads();

    Refill<TW, DMA, F16, VEC> rf;
    rf.issued0 = -1;
    rf.issued1 = -1;
    rf.sb = -1;
    rf.try_start(a, ctl, slot, wave, lane);
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    for (int32_t k = 0; k < nt; ++k) {
        const int b = k & 1;
        const uint32_t buf = b * a.buf_bytes;
        {
            // every wavefront's share of tile k landed (this wave's own share
            // may still be owed: flush copies and counts it)
            const int32_t target = a.waves * (k / 2 + 1);
            int32_t spins = 0;
            for (;;) {
                rf.flush(a, lds, ctl, slot, wave, lane, b, k);
                if (lds_load_acquire(&ctl[kCtlFill + b]) >= target)
                    break;
                __builtin_amdgcn_s_sleep(1);
                if (++spins > a.spin) {
                    if (lane == 0)
                        __hip_atomic_fetch_or(a.flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
            }
        }
        Cols<TW, F16, VEC> cols;
        cols.set(a, tile_of(a, slot, k), lane);
        if (k < a.rounds || a.parts == 1) {
            const int q = k & 1;
            const int32_t e0 = __builtin_amdgcn_readfirstlane(a.wave_ptr[q * a.waves + wave]);
            const int32_t e1 = __builtin_amdgcn_readfirstlane(a.wave_ptr[q * a.waves + wave + 1]);
            for (int32_t e = e0; e < e1; ++e)
                run_oct<MODE, TW, OFF_LDS>(a, lds, __builtin_amdgcn_readfirstlane(a.wave_oct[e]), buf, cols, lo, hi,
                                           lane, ctl, rf, slot, wave);
        } else {
            // a shared last tile: this position's octs, one per wavefront in turn
            for (int32_t o = slot % a.parts + a.parts * wave; o < a.noct; o += a.parts * a.waves)
                run_oct<MODE, TW, OFF_LDS>(a, lds, o, buf, cols, lo, hi, lane, ctl, rf, slot, wave);
        }
        if (k + 2 < nt) {
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's reads of the buffer are done
            int32_t old = 0;
            if (lane == 0)
                old = __hip_atomic_fetch_add(&ctl[kCtlRel + b], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
            old = __builtin_amdgcn_readfirstlane(old);
            if (old == a.waves * (k / 2 + 1) - 1 && lane == 0)  // the last one out frees the buffer for tile k + 2
                __hip_atomic_store(&ctl[kCtlFree + b], k + 2, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        rf.try_start(a, ctl, slot, wave, lane);
    }
    // every share this wave started was counted before the tile that needed
    // it; nothing is left in flight but stores
}

// LDS layout: two tile buffers, the offset table when it fits, the control words.
struct OuterLds {
    int32_t buf_bytes, off_lds, ctl_off, total;
};

OuterLds outer_lds(const DevicePlan &p) {
    OuterLds l;
    l.buf_bytes = (p.ozrow + 1) * 4 * p.otw;
    const int32_t table = (p.ooff_bytes + 1023) / 1024 * 1024;
    if (2 * l.buf_bytes + table + kCtlWords * 4 <= kMaxLdsBytes) {
        l.off_lds = 2 * l.buf_bytes;
        l.ctl_off = l.off_lds + table;
    } else {
        l.off_lds = -1;
        l.ctl_off = 2 * l.buf_bytes;
    }
    l.total = l.ctl_off + kCtlWords * 4;
    return l;
}

typedef void (*OKernel)(OArgs);

template <int MODE, int TW, bool OFF_LDS>
OKernel pick3(bool f16, bool vec) {
    if constexpr (MODE == 0) {
        if (f16)
            return vec ? outer_kernel<MODE, TW, OFF_LDS, true, true> : outer_kernel<MODE, TW, OFF_LDS, true, false>;
    }
    return vec ? outer_kernel<MODE, TW, OFF_LDS, false, true> : outer_kernel<MODE, TW, OFF_LDS, false, false>;
}

// The instantiation for a plan's mode and tile width, the table's place, the
// storage type and the vector path (fp16 only in matrix mode).
OKernel pick_outer(int mode, int tw, bool off_lds, bool f16, bool vec) {
    if (mode == 0)
        return off_lds ? pick3<0, 32, true>(f16, vec) : pick3<0, 32, false>(f16, vec);
    if (tw == 32)
        return off_lds ? pick3<1, 32, true>(f16, vec) : pick3<1, 32, false>(f16, vec);
    return off_lds ? pick3<1, 16, true>(f16, vec) : pick3<1, 16, false>(f16, vec);
}

}  // namespace

hipError_t prepare_outer(const DevicePlan &p) {
    for (int v = 0; v < 8; ++v) {
        const OKernel k = pick_outer(p.omode, p.otw, v & 4, (v & 1) && p.omode == 0, v & 2);
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 static_cast<int>(kMaxLdsBytes));
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

int32_t outer_lds_bytes(const DevicePlan &p) { return outer_lds(p).total; }

hipError_t launch_outer(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                        int64_t x_bytes, hipStream_t stream) {
    const OuterLds l = outer_lds(p);
    OArgs a;
    a.x = x;
    a.y = y;
    a.bias = p.rrow_bias;
    a.rec = reinterpret_cast<const f4 *>(p.orec);
    a.off = reinterpret_cast<const i4 *>(p.ooff);
    a.off_bytes = p.ooff_bytes;
    a.off_lds = l.off_lds;
    a.oct = p.ooct;
    a.wave_ptr = p.owave_ptr;
    a.wave_oct = p.owave_oct;
    a.flag = p.flag;
    a.spin = p.spin_limit;
    a.cin = p.cin;
    a.cout = p.cout;
    a.hw = hw;
    a.m = m;
    a.act = p.act;
    a.ntiles = (m + p.otw - 1) / p.otw;
    const int32_t cus = p.num_cus > 0 ? p.num_cus : 256;
    a.noct = p.oocts;
    if (a.ntiles >= cus) {
        // whole rounds of the grid, then each left-over tile shared among as
        // many workgroups as the grid holds for it, at most one per set
        a.grid = cus;
        a.rounds = a.ntiles / a.grid;
        a.rem = a.ntiles % a.grid;
        a.parts = 1;
        if (a.rem > 0)
            a.parts = std::max(1, std::min(a.grid / a.rem, p.oocts));
    } else {
        // fewer tiles than compute units: every tile shared that way
        a.rounds = 0;
        a.rem = a.ntiles;
        a.parts = std::max(1, std::min(cus / a.ntiles, p.oocts));
        a.grid = a.ntiles * a.parts;
    }
    a.nx = a.grid % 8 == 0 ? 8 : 1;
    a.waves = p.owaves;
    a.ozrow = p.ozrow;
    a.buf_bytes = l.buf_bytes;
    a.ctl_off = l.ctl_off;
    a.x_bytes = x_bytes;
    const OKernel k = pick_outer(p.omode, p.otw, l.off_lds >= 0, p.storage == 1, vec != 0);
    hipLaunchKernelGGL(k, dim3(a.grid), dim3(64 * a.waves), l.total, stream, a);
    return hipGetLastError();
}

}  // namespace spconv
