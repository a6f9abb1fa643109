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
// next; each wavefront copies its share of that tile (16-byte global-to-LDS
// loads) at its next check and counts it as landed at the check after
// (Refill below).  A wavefront starts a tile once every share of it has been
// counted: a bounded wait that sets the plan's error word if it gives up.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "launch.hpp"

namespace spconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i4 __attribute__((ext_vector_type(4)));

struct OArgs {
    const float *x;
    float *y;
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
    int32_t waves, ozrow, buf_bytes;
    int32_t ctl_off;  // LDS byte address of the control words
    int64_t x_bytes;
};

// LDS control words after the two buffers, per buffer: wavefronts done with
// it, copy shares of it landed (one per wavefront per tile), and the tile
// sequence number it is free to take next (set by the last wavefront out).
constexpr int kCtlRel = 0, kCtlFill = 2, kCtlFree = 4, kCtlWords = 6;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt takes 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

constexpr int32_t kOutOfRange = static_cast<int32_t>(0x80000000u);
constexpr int64_t kMaxRecords = 0x7ffffff0;

__device__ __forceinline__ i4 rsrc_words(const void *p, int64_t bytes) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    i4 r;
    r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(v));
    r.y = __builtin_amdgcn_readfirstlane(static_cast<int>((v >> 32) & 0xffff));
    r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes < kMaxRecords ? bytes : kMaxRecords));
    r.w = 0x00020000;
    return r;
}

// Workgroup wg's position in the tile map: XCD x (= wg % nx) takes the
// neighbouring tiles x * (grid / nx) .. of every round, so the 128-byte lines
// two neighbouring tiles share meet in one L2.
__device__ __forceinline__ int32_t tile_slot(const OArgs &a, int32_t wg) {
    return (wg % a.nx) * (a.grid / a.nx) + wg / a.nx;
}

// Copy instructions [i0, i1) step `di` of tile `tile` into the LDS buffer at
// byte `buf`: instruction i moves channel rows 8i .. 8i + 7 (lane l: row
// 8i + l / 8, vector l % 8), 1 KB, to buf + 1024 i.  Columns past m and
// channels past cin read zeros.
__device__ __forceinline__ void copy_tile(const OArgs &a, int32_t tile, uint32_t buf, int i0, int i1, int di,
                                          int lane) {
    const int32_t col0 = tile * kOuterCols;
    const int32_t n0 = col0 / a.hw;
    const int64_t xbase = static_cast<int64_t>(n0) * a.cin * a.hw;
    const i4 rs = rsrc_words(a.x + xbase, a.x_bytes - xbase * 4);
    const int32_t cc = col0 + (lane & 7) * 4;
    const int32_t n = cc / a.hw;
    const int32_t p = cc - n * a.hw;
    const int32_t crow = lane >> 3;
    const bool ok = cc < a.m;
    const int32_t lo = ((n - n0) * a.cin * a.hw + crow * a.hw + p) * 4;
    const int32_t step = 8 * a.hw * 4;
    for (int i = i0; i < i1; i += di) {
        const int32_t voff = ok && 8 * i + crow < a.cin ? lo + i * step : kOutOfRange;
        const uint32_t m0 = __builtin_amdgcn_readfirstlane(buf + 1024 * i);
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                     :
                     : "s"(m0), "v"(voff), "s"(rs)
                     : "memory", "m0");
    }
}

__device__ __forceinline__ int32_t lds_load_acquire(const int32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// A wavefront's part in refilling the two buffers.  When a buffer's last
// wavefront leaves it, it publishes the tile sequence number the buffer takes
// next; every wavefront, at its next check, copies its share of that tile
// (instructions wave, wave + waves, ...) and, at the check after that, counts
// the share as landed.  Checks run every kOuterAhead pairs inside an oct (the
// record loads issued in between guarantee that older copies have completed:
// loads complete in order), at the end of each tile and while waiting.
struct Refill {
    int32_t issued[2];  // sequence number of the last tile whose share this wave copied, per buffer
    int32_t pend;       // buffers with copied shares not yet counted (bit b)

    __device__ __forceinline__ void count(int32_t *ctl, int lane) {
        if (lane == 0) {
            if (pend & 1)
                __hip_atomic_fetch_add(&ctl[kCtlFill + 0], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            if (pend & 2)
                __hip_atomic_fetch_add(&ctl[kCtlFill + 1], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        pend = 0;
    }
    // Copy this wave's share of any tile a buffer was freed for.
    __device__ __forceinline__ void issue(const OArgs &a, int32_t *ctl, int32_t slot, int wave, int lane) {
        for (int b = 0; b < 2; ++b) {
            const int32_t g = __builtin_amdgcn_readfirstlane(lds_load_acquire(&ctl[kCtlFree + b]));
            if (g > issued[b]) {
                copy_tile(a, g * a.grid + slot, b * a.buf_bytes, wave, a.ozrow / 8, a.waves, lane);
                issued[b] = g;
                pend |= 1 << b;
            }
        }
    }
    // Inside an oct: at least N loads were issued since the last check.
    template <int N>
    __device__ __forceinline__ void check(const OArgs &a, int32_t *ctl, int32_t slot, int wave, int lane) {
        if (pend) {
            wait_vmcnt<N>();
            count(ctl, lane);
        }
        issue(a, ctl, slot, wave, lane);
    }
    // Anywhere: wait for this wave's copies, count them, issue new shares.
    __device__ __forceinline__ void flush(const OArgs &a, int32_t *ctl, int32_t slot, int wave, int lane) {
        if (pend) {
            wait_vmcnt<0>();
            count(ctl, lane);
        }
        issue(a, ctl, slot, wave, lane);
    }
};

__device__ __forceinline__ f4 lds_vec(const unsigned char *lds, uint32_t byte) {
    return *reinterpret_cast<const f4 *>(lds + byte);
}

// One oct on the tile in the buffer at byte `buf`: lockstep steps, then bias,
// activation and 16-byte stores of the lane's 4 rows x 4 columns.  OFF_LDS:
// the channel-row offsets come from the workgroup's LDS copy of the table,
// else from global memory.
template <bool OFF_LDS>
__device__ __forceinline__ void run_oct(const OArgs &a, const unsigned char *lds, int32_t o, uint32_t buf,
                                        float *ylane, bool col_ok, float lo, float hi, int lane, int32_t *ctl,
                                        Refill &rf, int32_t slot, int wave) {
    const int32_t *tab = a.oct + o * kOctWords;
    const int32_t q0 = __builtin_amdgcn_readfirstlane(tab[0]);
    const int32_t nq = __builtin_amdgcn_readfirstlane(tab[1]);
    const int g = lane >> 3;
    const int32_t rb = tab[2 + g];
    const f4 *wp = a.rec + (static_cast<int64_t>(q0) * kOuterSlots + g * 4 + (lane & 3));
    const int64_t og = static_cast<int64_t>(q0) * kOctRows + g;  // (quad, group) index of the offsets
    auto offs = [&](int32_t j) -> i4 {
        if constexpr (OFF_LDS)
            return *reinterpret_cast<const i4 *>(lds + a.off_lds + (og + int64_t(j) * kOctRows) * 16);
        else
            return a.off[og + int64_t(j) * kOctRows];
    };
    const uint32_t xl = buf + (lane & 7) * 16;
    f4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0, acc2 = acc0, acc3 = acc0;
    auto mma = [&](float w, const f4 x) {
        acc0 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.x, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.y, acc1, 0, 0, 0);
        acc2 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.z, acc2, 0, 0, 0);
        acc3 = __builtin_amdgcn_mfma_f32_4x4x1f32(w, x.w, acc3, 0, 0, 0);
    };
    auto xrow = [&](int32_t off) { return lds_vec(lds, xl + static_cast<uint32_t>(off)); };
    // Software pipeline: weights kOuterAhead quads ahead in registers (the
    // arrays are padded for it), the next quad's offsets one quad ahead, and
    // each step's X vector read before the previous step's matrix
    // instructions (two register sets, alternating by step).
    f4 wq[kOuterAhead];
#pragma unroll
    for (int i = 0; i < kOuterAhead; ++i)
        wq[i] = wp[i * kOuterSlots];
    wp += kOuterAhead * kOuterSlots;
    i4 oq = offs(0);
    f4 xs[2];
    xs[0] = xrow(oq.x);
    // one quad: its 4 steps, the first X of the next quad read during the last
    auto quad = [&](const f4 w, const i4 nx) {
        xs[1] = xrow(oq.y);
        __builtin_amdgcn_sched_barrier(0);
        mma(w.x, xs[0]);
        xs[0] = xrow(oq.z);
        __builtin_amdgcn_sched_barrier(0);
        mma(w.y, xs[1]);
        xs[1] = xrow(oq.w);
        __builtin_amdgcn_sched_barrier(0);
        mma(w.z, xs[0]);
        xs[0] = xrow(nx.x);
        __builtin_amdgcn_sched_barrier(0);
        mma(w.w, xs[1]);
    };
    int32_t j = 0;
    for (; j + kOuterAhead <= nq; j += kOuterAhead) {
#pragma unroll
        for (int i = 0; i < kOuterAhead; ++i) {
            const i4 nx = offs(j + i + 1);
            quad(wq[i], nx);
            wq[i] = wp[i * kOuterSlots];  // after its last use: no copy of the old weights
            oq = nx;
            __builtin_amdgcn_sched_barrier(0);
        }
        wp += kOuterAhead * kOuterSlots;
        // loads since the last check: kOuterAhead weight loads (and as many offset loads)
        rf.template check<OFF_LDS ? kOuterAhead : 2 * kOuterAhead>(a, ctl, slot, wave, lane);
    }
#pragma unroll
    for (int i = 0; i < kOuterAhead - 1; ++i) {
        if (j + i < nq) {
            const i4 nx = offs(j + i + 1);
            quad(wq[i], nx);
            oq = nx;
        }
    }
    if (rb >= 0 && col_ok) {
        const f4 bz = *reinterpret_cast<const f4 *>(a.bias + 4 * rb);
        float *yr = ylane + static_cast<int64_t>(4 * rb) * a.hw;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            f4 v;
            v.x = fminf(fmaxf(acc0[r] + bz[r], lo), hi);
            v.y = fminf(fmaxf(acc1[r] + bz[r], lo), hi);
            v.z = fminf(fmaxf(acc2[r] + bz[r], lo), hi);
            v.w = fminf(fmaxf(acc3[r] + bz[r], lo), hi);
            *reinterpret_cast<f4 *>(yr + static_cast<int64_t>(r) * a.hw) = v;
        }
    }
}

template <bool OFF_LDS>
__global__ void __launch_bounds__(1024) outer_kernel(OArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int32_t slot = tile_slot(a, blockIdx.x);
    const int32_t nt = slot < a.ntiles ? (a.ntiles - slot + a.grid - 1) / a.grid : 0;
    if (nt == 0)
        return;
    int32_t *ctl = reinterpret_cast<int32_t *>(lds + a.ctl_off);
    const int ninstr = a.ozrow / 8;
    // zero rows of both buffers, control words, the first two tiles: tile 0
    // behind a barrier, tile 1 counted by each wavefront's share
    if (threadIdx.x < 16) {
        const int b = threadIdx.x >> 3;
        *reinterpret_cast<f4 *>(lds + b * a.buf_bytes + a.ozrow * kOuterRowBytes + (threadIdx.x & 7) * 16) =
            f4{0.f, 0.f, 0.f, 0.f};
    }
    if (threadIdx.x < kCtlWords)  // tile 0 is complete at the barrier below: count its shares
        ctl[threadIdx.x] = threadIdx.x == kCtlFill ? a.waves : 0;
    if constexpr (OFF_LDS) {
        // the offset table, 1 KB per instruction (reads past its end give zeros)
        const i4 rs = rsrc_words(a.off, a.off_bytes);
        for (int i = wave; i < (a.off_bytes + 1023) / 1024; i += a.waves) {
            const uint32_t m0 = __builtin_amdgcn_readfirstlane(a.off_lds + 1024 * i);
            asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                         :
                         : "s"(m0), "v"(1024 * i + lane * 16), "s"(rs)
                         : "memory", "m0");
        }
    }
    copy_tile(a, slot, 0, wave, ninstr, a.waves, lane);
    Refill rf;
    rf.issued[0] = 0;
    rf.issued[1] = 0;
    rf.pend = 0;
    if (nt > 1) {
        copy_tile(a, slot + a.grid, a.buf_bytes, wave, ninstr, a.waves, lane);
        rf.issued[1] = 1;
        rf.pend = 2;
        // this wavefront's tile-0 copies are the older ones: wait until at most
        // its tile-1 copies (or fewer) are in flight
        const int mine = (ninstr - wave + a.waves - 1) / a.waves;
        if (mine >= 8)
            wait_vmcnt<8>();
        else if (mine >= 4)
            wait_vmcnt<4>();
        else if (mine >= 2)
            wait_vmcnt<2>();
        else
            wait_vmcnt<0>();
    } else {
        wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): zero rows and control words written
    __syncthreads();

    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    for (int32_t k = 0; k < nt; ++k) {
        const int b = k & 1;
        const uint32_t buf = b * a.buf_bytes;
        if (k >= 1) {
            // every wavefront's share of tile k's copy landed (this wave's own
            // share may still be owed: flush issues and counts it)
            const int32_t target = a.waves * (k / 2 + 1);
            int32_t spins = 0;
            for (;;) {
                rf.flush(a, ctl, slot, wave, lane);
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
        const int32_t tile = k * a.grid + slot;
        const int32_t cc = tile * kOuterCols + (lane & 7) * 4;
        const bool col_ok = cc < a.m;
        const int32_t n = cc / a.hw;
        float *ylane = a.y + (static_cast<int64_t>(n) * a.cout * a.hw + (cc - n * a.hw));
        const int q = k & 1;
        const int32_t e0 = __builtin_amdgcn_readfirstlane(a.wave_ptr[q * a.waves + wave]);
        const int32_t e1 = __builtin_amdgcn_readfirstlane(a.wave_ptr[q * a.waves + wave + 1]);
        for (int32_t e = e0; e < e1; ++e)
            run_oct<OFF_LDS>(a, lds, __builtin_amdgcn_readfirstlane(a.wave_oct[e]), buf, ylane, col_ok, lo, hi,
                             lane, ctl, rf, slot, wave);
        if (k + 2 < nt) {
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's reads of the buffer are done
            int32_t old = 0;
            if (lane == 0)
                old = __hip_atomic_fetch_add(&ctl[kCtlRel + b], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
            old = __builtin_amdgcn_readfirstlane(old);
            if (old == a.waves * (k / 2 + 1) - 1 && lane == 0)  // the last one out frees the buffer for tile k + 2
                __hip_atomic_store(&ctl[kCtlFree + b], k + 2, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        rf.issue(a, ctl, slot, wave, lane);
    }
    // every copy this wave issued was counted before the tile that needed it;
    // nothing is left in flight but stores
}

// LDS layout: two tile buffers, the offset table when it fits, the control words.
struct OuterLds {
    int32_t buf_bytes, off_lds, ctl_off, total;
};

OuterLds outer_lds(const DevicePlan &p) {
    OuterLds l;
    l.buf_bytes = (p.ozrow + 1) * kOuterRowBytes;
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

}  // namespace

hipError_t prepare_outer(const DevicePlan &p) {
    (void)p;
    for (const void *k : {reinterpret_cast<const void *>(outer_kernel<true>),
                          reinterpret_cast<const void *>(outer_kernel<false>)}) {
        const hipError_t e =
            hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kMaxLdsBytes));
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

int32_t outer_lds_bytes(const DevicePlan &p) { return outer_lds(p).total; }

hipError_t launch_outer(const DevicePlan &p, const float *x, float *y, int32_t m, int32_t hw, int64_t x_bytes,
                        hipStream_t stream) {
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
    a.ntiles = (m + kOuterCols - 1) / kOuterCols;
    const int32_t cus = p.num_cus > 0 ? p.num_cus : 256;
    a.grid = a.ntiles < cus ? a.ntiles : cus;
    a.nx = a.grid % 8 == 0 ? 8 : 1;
    a.waves = p.owaves;
    a.ozrow = p.ozrow;
    a.buf_bytes = l.buf_bytes;
    a.ctl_off = l.ctl_off;
    a.x_bytes = x_bytes;
    if (l.off_lds >= 0)
        hipLaunchKernelGGL(outer_kernel<true>, dim3(a.grid), dim3(64 * a.waves), l.total, stream, a);
    else
        hipLaunchKernelGGL(outer_kernel<false>, dim3(a.grid), dim3(64 * a.waves), l.total, stream, a);
    return hipGetLastError();
}

}  // namespace spconv
