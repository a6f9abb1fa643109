// Register-indexed kernel for the sparse 1x1 convolution on gfx950
//     Y[n, r, p] = act(b[r] + sum_c W[r, c] * X[n, c, p])
// (Fast Sparse ConvNets, Sec. 3.2 / Fig. 2), over NCHW fp32 tensors.
//
// The paper's kernel walks the output rows of one strip of spatial columns
// and reads every nonzero's activations from the near cache (Sec. 3.2,
// insights 2 and 3).  On gfx950 that costs one LDS read and one address add
// per nonzero and lane, and the vector ALU (one wave64 fp32 FMA per ~4.5
// cycles per SIMD, no packed FMA here) becomes the limit long before HBM.
// This kernel turns the loop around:
//
//   * A wavefront owns a *slot* of 16 output channels and C columns per lane
//     (64 C columns per tile, lane l holding columns 64 k + l).  Its 16 x C
//     fp32 accumulators stay in registers for the whole tile.
//   * It walks the slot's nonzeros by ascending input channel (CSC order
//     inside the slot).  For one channel it reads the C activations of its
//     columns once from LDS and adds them, times the weight, into the
//     accumulator of each row that has a nonzero there.  The row is chosen
//     at run time with register-relative addressing: with s_set_gpr_idx_on
//     the FMA's accumulator operand (source 2 and destination) is offset by
//     the index in M0, and s_set_gpr_idx_idx moves it to the next row.
//   * Records (planner.hpp) carry, per channel, the slot rows and weights of
//     up to 3 (1x1), 2 (1x2) or 1 (1x4 block) nonzeros, two records per
//     64-byte batch.  The stream is software-pipelined with one wait per
//     batch: at the start of batch b the wavefront waits once (for the
//     records of batch b + 1 and the activations of batch b), then loads the
//     records of batch b + 2 into the third of three scalar buffers and
//     starts the LDS reads of batch b + 1's activations into the second of
//     two register sets, and only then runs batch b.  Scalar loads and LDS
//     reads share one wait counter and scalar loads return out of order, so
//     a single full wait per batch, a whole batch after the loads it covers,
//     is what keeps both latencies hidden.
//   * X reaches LDS by buffer loads that write LDS directly, into a ring of
//     96 channel rows (1536 bytes each: 6 column slots of 64 fp32) in 6
//     chunks of 16.  The last wavefront to finish with a chunk refills its
//     ring rows with the chunk 6 ahead (16 bytes per lane and load when every
//     image's column count is a multiple of 4, one dword otherwise) and
//     publishes it at its next chunk boundary; a wavefront waits only for the
//     chunk it is about to read, so the fastest may run up to about four
//     chunks ahead of the slowest.  The first record of each batch flags the
//     last batch of a chunk and of the stream.
//
// Every row sums its products in ascending input channel from zero with fp32
// FMA and adds the bias last, exactly as the other kernels of this library do
// (padding records of weight 0 add +0, which leaves every finite sum as it
// is), so the result does not depend on the kernel, the slot assignment or
// the tile split.
//
// Register plan (per C): compiler-managed v0 .. A-1 and s0 .. s33; reserved
// accumulators v[A + 16 k + r] (column k, slot row r), two activation sets of
// two records each (C registers per record, rounded up to even), two
// temporaries (also the LDS addresses of a batch's reads); s34 .. s47
// control, s48 .. s95 three 16-dword record buffers.
//
// Columns left over after the last whole tile round are computed by row
// pairs: each wavefront takes two output channels over 64 columns, with a
// plain loop reading the columns' activations from an LDS strip and the
// pair's (channel, weight, weight) entries from a per-wavefront LDS area,
// both filled by LDS-direct loads before the loop.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>
#include <utility>

#include "launch.hpp"

// M0 is written by the indexing and LDS-copy instructions; the clobber says so.
#pragma clang diagnostic ignored "-Winline-asm"

namespace spconv {
namespace {

using Rsrc = __amdgpu_buffer_rsrc_t;
typedef int i4 __attribute__((ext_vector_type(4)));

constexpr int32_t kOOR = static_cast<int32_t>(0x80000000u);  // an offset past every buffer: loads read 0
constexpr int64_t kMaxRec = 0x7ffffff0;
constexpr int32_t kRingChunks = kRing / kChunk;             // 6 chunks in the ring
static_assert(kRingRowBytes == 6 * 256, "a ring row holds 6 column slots");
static_assert(kRingChunks == 6, "the stream statement counts ring chunks modulo 6");

template <int C>
struct Lay {
    static constexpr int XS = (C + 1) & ~1;                // one record's activations, even-aligned
    static constexpr int A = 128 - 16 * C - 4 * XS - 2;     // accumulators v[A + 16 k + r]
    static constexpr int XA0 = A + 16 * C;                  // activation set a: records 0 and 1
    static constexpr int XA1 = XA0 + XS;
    static constexpr int XB0 = XA1 + XS;                    // activation set b
    static constexpr int XB1 = XB0 + XS;
    static constexpr int T = XB1 + XS;                      // two temporaries, up to v127
    static_assert(T == 126, "register plan must end at v127");
    static_assert(A >= 6, "the compiler keeps at least v0 .. v5");
};

template <typename F, int... I>
__device__ __forceinline__ void sfor_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void sfor(F &&f) {
    sfor_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ Rsrc make_rsrc(const void *p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0),
                                             static_cast<int>(std::min<int64_t>(bytes, kMaxRec)), 0x00020000);
}

__device__ __forceinline__ i4 rsrc_words(const void *p, int64_t bytes) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    i4 r;
    r.x = __builtin_amdgcn_readfirstlane(static_cast<int>(v));
    r.y = __builtin_amdgcn_readfirstlane(static_cast<int>((v >> 32) & 0xffff));
    r.z = __builtin_amdgcn_readfirstlane(static_cast<int>(std::min<int64_t>(bytes, kMaxRec)));
    r.w = 0x00020000;
    return r;
}

// A pointer every lane holds the same value of, in scalar registers.
template <typename T>
__device__ __forceinline__ T *uniform_ptr(T *p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return reinterpret_cast<T *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Read-only plan data every lane of a wavefront reads at the same address:
// through the constant address space these become scalar loads.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(4))) T *cst(const T *p) {
    return (const __attribute__((address_space(4))) T *)(uniform_ptr(p));
}

// One dword per lane from global memory straight into LDS at m0 + 4 * lane.
__device__ __forceinline__ void dma_dword(uint32_t m0, int32_t voff, i4 rs, int32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(rs),
                   "s"(__builtin_amdgcn_readfirstlane(soff))
                 : "memory", "m0");
}

// Sixteen bytes per lane from global memory straight into LDS at m0 + 16 * lane.
__device__ __forceinline__ void dma_x4(uint32_t m0, int32_t voff, i4 rs, int32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(m0)), "v"(voff), "s"(rs),
                   "s"(__builtin_amdgcn_readfirstlane(soff))
                 : "memory", "m0");
}

// s_waitcnt vmcnt(0) (lgkmcnt and expcnt left at their maximum)
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0f70); }

__device__ __forceinline__ int32_t imin(int32_t a, int32_t b) { return a < b ? a : b; }

struct IArgs {
    const float *x;
    float *y;
    int32_t cin, cout, hw, m, act;
    int64_t x_bytes, y_bytes;
    int32_t nch, slots, groups, waves;
    int32_t main_tasks;   // tiles * groups
    int32_t lcol0;        // first column of the row-pair phase
    int32_t lpieces;      // (64-column group, row pair) pieces
    int32_t lper;         // pieces per workgroup
    int32_t pairs;        // row pairs
    int32_t v4;           // 16-byte copies (every image's column count a multiple of 4, x 16-byte aligned)
    int32_t ctl_off;      // LDS byte offsets: counters, lane column tables, copy patterns (the ring at 0)
    int32_t xo_off, pat_off;
    int32_t ent_off;      // row pairs: LDS byte offset of the entry areas (the strip at 0)
    int32_t epw;          // row pairs: entries per wavefront area
    const uint32_t *rec;
    const int32_t *slot_batch, *slot_rows;
    const float *slot_bias;
    const int32_t *pair_ptr;
    const uint32_t *pair_ent;
    int64_t pair_ent_bytes;
    const float *row_bias;
    int32_t *flag;        // set when a bounded wait gives up
    int32_t spin;         // bound of those waits, in sleeps
};

// The launch arguments, read afresh from the kernel-argument segment: the
// pointer passes through an empty asm statement, so the compiler reloads the
// fields where each phase of the kernel uses them instead of holding every
// argument in scalar registers for the whole kernel (the stream statement
// leaves it 34).
typedef const __attribute__((address_space(4))) IArgs KArgs;

__device__ __forceinline__ KArgs &kargs() {
    const IArgs *p = (const IArgs *)(__builtin_amdgcn_kernarg_segment_ptr());
    asm volatile("" : "+s"(p));
    return *cst(p);
}

// Clobber lists of the stream statement: every register it uses for itself.
#define IY_CLOBV1 "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBV2 "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBV3 "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBV4 "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBV5 "v22", "v23", "v24", "v25", "v26", "v27", "v28", "v29", "v30", "v31", "v32", "v33", "v34", "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45", "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBV6 "v6", "v7", "v8", "v9", "v10", "v11", "v12", "v13", "v14", "v15", "v16", "v17", "v18", "v19", "v20", "v21", "v22", "v23", "v24", "v25", "v26", "v27", "v28", "v29", "v30", "v31", "v32", "v33", "v34", "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45", "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IY_CLOBS "s34", "s35", "s36", "s37", "s38", "s39", "s40", "s41", "s42", "s43", "s44", "s45", "s46", "s47", "s48", "s49", "s50", "s51", "s52", "s53", "s54", "s55", "s56", "s57", "s58", "s59", "s60", "s61", "s62", "s63", "s64", "s65", "s66", "s67", "s68", "s69", "s70", "s71", "s72", "s73", "s74", "s75", "s76", "s77", "s78", "s79", "s80", "s81", "s82", "s83", "s84", "s85", "s86", "s87", "s88", "s89", "s90", "s91", "s92", "s93", "s94", "s95"

// ---------------------------------------------------------------------------
// The stream statement.  One inline-assembly statement runs a wavefront's
// whole slot over one tile: zero the accumulators, walk the batches (wait,
// prefetch, compute; at a chunk's last batch enter the next chunk before the
// prefetch and release this one after the compute, refilling its ring
// rows when this wavefront is the last to release it), then bias,
// activation and store.  Inside it the compiler places nothing, so the
// accumulators, activation sets and record buffers are simply registers it
// was told are clobbered.
//
// Scalar registers: s34 chunk q, s35 byte offset of the next record load,
// s36:37 saved exec, s38 ring chunks loaded by this wavefront but not yet
// published (bit per ring chunk; on entry the set-up's chunks 1 .. 5), s39 spin count / temporary, s40 ring chunk of q (q mod 6), s41
// round of q (q div 6), s42 - s45 temporaries, s46 / s47 ring chunk and round
// of q + 1, s48 - s63 / s64 - s79 / s80 - s95 the record buffers (batch b in
// buffer b % 3; record 0 at +0, record 1 at +8).  LDS counters: free[j] at
// ctl + 4 j (wavefronts done with ring chunk j, all rounds), fill[j] at ctl +
// 32 + 4 j (set-up wavefronts that published their share of ring chunk j's
// first round, plus one per later round).
// Vector: accumulators v[a + 16 k + r], activation sets xa0 / xa1 and xb0 /
// xb1 (batch b in set b % 2), temporaries t, t + 1.
// ---------------------------------------------------------------------------

#define RY_F(k, i, X, R, W) \
    "v_fma_f32 v[%[a]+16*" #k "+" #i "], v[%[" #X "]+" #k "], s[" #R "+" #W "], v[%[a]+16*" #k "+" #i "]\n"
#define RY_C1(i, X, R, W) RY_F(0, i, X, R, W)
#define RY_C2(i, X, R, W) RY_C1(i, X, R, W) RY_F(1, i, X, R, W)
#define RY_C3(i, X, R, W) RY_C2(i, X, R, W) RY_F(2, i, X, R, W)
#define RY_C4(i, X, R, W) RY_C3(i, X, R, W) RY_F(3, i, X, R, W)
#define RY_C5(i, X, R, W) RY_C4(i, X, R, W) RY_F(4, i, X, R, W)
#define RY_C6(i, X, R, W) RY_C5(i, X, R, W) RY_F(5, i, X, R, W)

// One record at SGPR R (indexing on): up to 3 rows (1x1), 2 blocks (1x2) or
// 1 block (1x4).  L: a label name unique within the statement.
#define RY_REC_K1(COLS, X, R, L)            \
    "s_set_gpr_idx_idx s[" #R "+1]\n"       \
    COLS(0, X, R, 4)                        \
    "s_bitcmp1_b32 s[" #R "+1], 8\n"        \
    "s_cbranch_scc0 " L "_%=\n"             \
    "s_set_gpr_idx_idx s[" #R "+2]\n"       \
    COLS(0, X, R, 5)                        \
    "s_bitcmp1_b32 s[" #R "+1], 9\n"        \
    "s_cbranch_scc0 " L "_%=\n"             \
    "s_set_gpr_idx_idx s[" #R "+3]\n"       \
    COLS(0, X, R, 6)                        \
    L "_%=:\n"
#define RY_REC_K2(COLS, X, R, L)            \
    "s_set_gpr_idx_idx s[" #R "+1]\n"       \
    COLS(0, X, R, 4) COLS(1, X, R, 5)       \
    "s_bitcmp1_b32 s[" #R "+1], 8\n"        \
    "s_cbranch_scc0 " L "_%=\n"             \
    "s_set_gpr_idx_idx s[" #R "+2]\n"       \
    COLS(0, X, R, 6) COLS(1, X, R, 7)       \
    L "_%=:\n"
#define RY_REC_K4(COLS, X, R, L)            \
    "s_set_gpr_idx_idx s[" #R "+1]\n"       \
    COLS(0, X, R, 4) COLS(1, X, R, 5) COLS(2, X, R, 6) COLS(3, X, R, 7)

// The activations of one record: C dwords, a column slot (256 B) apart, from
// the LDS address in t + VA.
#define RY_XL1(X, VA) "ds_read_b32 v[%[" #X "]], v[%[t]+" #VA "]\n"
#define RY_XL2(X, VA) "ds_read2st64_b32 v[%[" #X "]:%[" #X "]+1], v[%[t]+" #VA "] offset1:1\n"
#define RY_XL3(X, VA) RY_XL2(X, VA) "ds_read_b32 v[%[" #X "]+2], v[%[t]+" #VA "] offset:512\n"
#define RY_XL4(X, VA) RY_XL2(X, VA) "ds_read2st64_b32 v[%[" #X "]+2:%[" #X "]+3], v[%[t]+" #VA "] offset0:2 offset1:3\n"
#define RY_XL5(X, VA) RY_XL4(X, VA) "ds_read_b32 v[%[" #X "]+4], v[%[t]+" #VA "] offset:1024\n"
#define RY_XL6(X, VA) RY_XL4(X, VA) "ds_read2st64_b32 v[%[" #X "]+4:%[" #X "]+5], v[%[t]+" #VA "] offset0:4 offset1:5\n"

// Start the activation reads of the batch whose records are at SGPR RN into
// set (X0, X1).  The index must be 0 (these two adds are indexed too).
#define RY_PREF(XL, RN, X0, X1)                                  \
    "v_add_u32 v[%[t]], s[" #RN "], %[vl]\n"                     \
    "v_add_u32 v[%[t]+1], s[" #RN "+8], %[vl]\n"                 \
    XL(X0, 0) XL(X1, 1)

// Wait until ring chunk s46 holds round s47: its fill count reaches nws + s47
// (the first round is counted once per wavefront that loaded a share of it,
// each later round once by its copier); a bounded wait that sets the plan's
// flag on giving up.  Indexing off.
#define RY_WAITFILL(L)                                             \
    "s_add_u32 s42, s47, %[nws]\n"                                 \
    "s_lshl_b32 s43, s46, 2\n"                                     \
    "s_add_u32 s43, s43, %[ctl]\n"                                 \
    "s_add_u32 s43, s43, 32\n"                                     \
    "v_mov_b32 v[%[t]], s43\n"                                     \
    "s_mov_b32 s39, 0\n"                                           \
    L "sp_%=:\n"                                                   \
    "ds_read_b32 v[%[t]+1], v[%[t]]\n"                             \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "v_readfirstlane_b32 s44, v[%[t]+1]\n"                         \
    "s_cmp_ge_i32 s44, s42\n"                                      \
    "s_cbranch_scc1 " L "ok_%=\n"                                  \
    "s_add_u32 s39, s39, 1\n"                                      \
    "s_cmp_gt_u32 s39, %[spin]\n"                                  \
    "s_cbranch_scc1 " L "bad_%=\n"                                 \
    "s_sleep 1\n"                                                  \
    "s_branch " L "sp_%=\n"                                        \
    L "bad_%=:\n"                                                  \
    "s_mov_b64 s[36:37], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "v_mov_b32 v[%[t]], 0\n"                                       \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    "global_atomic_or v[%[t]], v[%[t]+1], %[flag]\n"               \
    "s_mov_b64 exec, s[36:37]\n"                                   \
    L "ok_%=:\n"
// Count the landing of every ring chunk copied earlier (after the copies'
// loads are complete), one lane adding to its fill counter.
#define RY_PUB1(j, L)                                                    \
    "s_bitcmp1_b32 s38, " #j "\n"                                        \
    "s_cbranch_scc0 " L #j "_%=\n"                                       \
    "s_add_u32 s42, %[ctl], 32+4*" #j "\n"                               \
    "v_mov_b32 v[%[t]], s42\n"                                           \
    "ds_add_u32 v[%[t]], v[%[t]+1]\n"                                    \
    L #j "_%=:\n"
#define RY_PUBLISH(L)                                              \
    "s_cmp_eq_u32 s38, 0\n"                                        \
    "s_cbranch_scc1 " L "_%=\n"                                    \
    "s_waitcnt vmcnt(0)\n"                                         \
    "s_mov_b64 s[36:37], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    RY_PUB1(0, L) RY_PUB1(1, L) RY_PUB1(2, L) RY_PUB1(3, L) RY_PUB1(4, L) RY_PUB1(5, L) \
    "s_mov_b64 exec, s[36:37]\n"                                   \
    "s_mov_b32 s38, 0\n"                                           \
    L "_%=:\n"

// Enter chunk q + 1: publish this wavefront's landed loads (the set-up's
// shares of the first ring are published here at the latest, before any
// wavefront can need them), put chunk q + 1's ring chunk and round into
// s46 / s47, then wait for it.
#define RY_ENTER(L)                                                \
    RY_PUBLISH(L "p")                                              \
    "s_add_u32 s46, s40, 1\n"                                      \
    "s_mov_b32 s47, s41\n"                                         \
    "s_cmp_eq_u32 s46, 6\n"                                        \
    "s_cbranch_scc0 " L "nx_%=\n"                                  \
    "s_mov_b32 s46, 0\n"                                           \
    "s_add_u32 s47, s47, 1\n"                                      \
    L "nx_%=:\n"                                                   \
    RY_WAITFILL(L)

// Chunk q + 6 into ring chunk s40: channels [s42, s43) into the 16 ring rows
// starting at LDS byte s44; v[t + 1] = 4 * lane.
#define RY_CP_HEAD                                                 \
    "s_add_u32 s42, s34, 6\n"                                      \
    "s_lshl_b32 s42, s42, 4\n"                                     \
    "s_add_u32 s43, s42, 16\n"                                     \
    "s_min_u32 s43, s43, %[cin]\n"                                 \
    "s_mul_i32 s44, s40, %[cbytes]\n"                              \
    "s_add_u32 s44, s44, %[base]\n"                                \
    "v_subrev_u32 v[%[t]+1], %[base], %[vl]\n"
// 16 bytes per lane: two ring rows are 3 KiB, three loads with lane source
// offsets (copy patterns) j = 0, 1, 2 from LDS; pass j covers load j of every
// row pair.
#define RY_CPX_PASS(L, j, OFF, MOFF)                               \
    "v_add_u32 v[%[t]], %[pat], v[%[t]+1]\n"                       \
    "ds_read_b32 v[%[t]], v[%[t]] offset:" #OFF "\n"               \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b32 s45, s42\n"                                         \
    L #j "_%=:\n"                                                  \
    "s_sub_u32 s39, s45, s42\n"                                    \
    "s_mul_i32 s39, s39, 1536\n"                                   \
    "s_add_u32 s39, s39, s44\n"                                    \
    "s_add_u32 m0, s39, " #MOFF "\n"                               \
    "s_mul_i32 s39, s45, %[hw4]\n"                                 \
    "s_nop 0\n"                                                    \
    "buffer_load_dwordx4 v[%[t]], %[rs], s39 offen lds\n"          \
    "s_add_u32 s45, s45, 2\n"                                      \
    "s_cmp_lt_u32 s45, s43\n"                                      \
    "s_cbranch_scc1 " L #j "_%=\n"
#define RY_CPX(L) RY_CP_HEAD RY_CPX_PASS(L, 0, 0, 0) RY_CPX_PASS(L, 1, 256, 1024) RY_CPX_PASS(L, 2, 512, 2048)
// One dword per lane: pass k copies column slot k of every row, lane offsets
// from the LDS column table.
#define RY_CPW(L, k, OFF)                                          \
    "v_add_u32 v[%[t]], %[xo], v[%[t]+1]\n"                        \
    "ds_read_b32 v[%[t]], v[%[t]] offset:" #OFF "\n"               \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b32 s45, s42\n"                                         \
    L #k "_%=:\n"                                                  \
    "s_sub_u32 s39, s45, s42\n"                                    \
    "s_mul_i32 s39, s39, 1536\n"                                   \
    "s_add_u32 s39, s39, s44\n"                                    \
    "s_add_u32 m0, s39, " #OFF "\n"                                \
    "s_mul_i32 s39, s45, %[hw4]\n"                                 \
    "s_nop 0\n"                                                    \
    "buffer_load_dword v[%[t]], %[rs], s39 offen lds\n"            \
    "s_add_u32 s45, s45, 1\n"                                      \
    "s_cmp_lt_u32 s45, s43\n"                                      \
    "s_cbranch_scc1 " L #k "_%=\n"
#define RY_CPW1(L) RY_CP_HEAD RY_CPW(L, 0, 0)
#define RY_CPW2(L) RY_CPW1(L) RY_CPW(L, 1, 256)
#define RY_CPW3(L) RY_CPW2(L) RY_CPW(L, 2, 512)
#define RY_CPW4(L) RY_CPW3(L) RY_CPW(L, 3, 768)
#define RY_CPW5(L) RY_CPW4(L) RY_CPW(L, 4, 1024)
#define RY_CPW6(L) RY_CPW5(L) RY_CPW(L, 5, 1280)
#define RY_COPY(L, CPW)                                            \
    "s_cmp_eq_u32 %[v4], 0\n"                                      \
    "s_cbranch_scc1 " L "w_%=\n"                                   \
    RY_CPX(L "x")                                                  \
    "s_branch " L "d_%=\n"                                         \
    L "w_%=:\n"                                                    \
    CPW(L "y")                                                     \
    L "d_%=:\n"

// Issue priority from the order of release (s44 - s43 wavefronts release
// this chunk after this one): the later a wavefront releases, the higher its
// priority until its next release.  Wavefronts of a SIMD otherwise drift
// apart under oldest-first issue, and the ring makes the ones ahead wait.
#define RY_RANK_PRIO(L)                                            \
    "s_sub_u32 s45, s44, s43\n"                                    \
    "s_setprio 0\n"                                                \
    "s_cmp_lt_u32 s45, 8\n"                                        \
    "s_cbranch_scc0 " L "q_%=\n"                                   \
    "s_setprio 1\n"                                                \
    "s_cmp_lt_u32 s45, 4\n"                                        \
    "s_cbranch_scc0 " L "q_%=\n"                                   \
    "s_setprio 2\n"                                                \
    "s_cmp_lt_u32 s45, 1\n"                                        \
    "s_cbranch_scc0 " L "q_%=\n"                                   \
    "s_setprio 3\n"                                                \
    L "q_%=:\n"

// Release chunk q (ring chunk s40, round s41; publish earlier copies first);
// the last wavefront to release it copies chunk q + 6 into its ring rows.
// Indexing off.
#define RY_LEAVE(L, CPW)                                           \
    RY_PUBLISH(L "p")                                              \
    "s_lshl_b32 s42, s40, 2\n"                                     \
    "s_add_u32 s42, s42, %[ctl]\n"                                 \
    "v_mov_b32 v[%[t]], s42\n"                                     \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    "s_mov_b64 s[36:37], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "ds_add_rtn_u32 v[%[t]+1], v[%[t]], v[%[t]+1]\n"               \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b64 exec, s[36:37]\n"                                   \
    "v_readfirstlane_b32 s43, v[%[t]+1]\n"                         \
    "s_add_u32 s43, s43, 1\n"                                      \
    "s_add_u32 s44, s41, 1\n"                                      \
    "s_mul_i32 s44, s44, %[nw]\n"                                  \
    RY_RANK_PRIO(L)                                                \
    "s_cmp_lg_u32 s43, s44\n"                                      \
    "s_cbranch_scc1 " L "n_%=\n"                                   \
    "s_add_u32 s44, s34, 6\n"                                      \
    "s_cmp_ge_u32 s44, %[nch]\n"                                   \
    "s_cbranch_scc1 " L "n_%=\n"                                   \
    RY_COPY(L "c", CPW)                                            \
    "s_lshl_b32 s42, 1, s40\n"                                     \
    "s_or_b32 s38, s38, s42\n"                                     \
    L "n_%=:\n"

// Bias, activation and store of the slot's 16 rows (rows in s48 - s63,
// biases in s64 - s79, the lane's C column offsets from the LDS table in
// xa0), unrolled over the rows.
#define RY_EPK(i, k)                                                                 \
    "v_add_f32 v[%[a]+16*" #k "+" #i "], s[64+" #i "], v[%[a]+16*" #k "+" #i "]\n"   \
    "v_max_f32 v[%[a]+16*" #k "+" #i "], v[%[a]+16*" #k "+" #i "], %[lo]\n"           \
    "v_min_f32 v[%[a]+16*" #k "+" #i "], v[%[a]+16*" #k "+" #i "], %[hi]\n"           \
    "buffer_store_dword v[%[a]+16*" #k "+" #i "], v[%[xa0]+" #k "], %[ry], s44 offen\n"
#define RY_EPC1(i) RY_EPK(i, 0)
#define RY_EPC2(i) RY_EPC1(i) RY_EPK(i, 1)
#define RY_EPC3(i) RY_EPC2(i) RY_EPK(i, 2)
#define RY_EPC4(i) RY_EPC3(i) RY_EPK(i, 3)
#define RY_EPC5(i) RY_EPC4(i) RY_EPK(i, 4)
#define RY_EPC6(i) RY_EPC5(i) RY_EPK(i, 5)
#define RY_EPROW(EPC, i)                       \
    "s_cmp_lt_i32 s[48+" #i "], 0\n"           \
    "s_cbranch_scc1 EP" #i "_%=\n"             \
    "s_mul_i32 s44, s[48+" #i "], %[hw4]\n"    \
    EPC(i)                                     \
    "EP" #i "_%=:\n"
#define RY_EPL(k, OFF) "ds_read_b32 v[%[xa0]+" #k "], v[%[t]+1] offset:" #OFF "\n"
#define RY_EACH1(M) M(0, 0)
#define RY_EACH2(M) RY_EACH1(M) M(1, 256)
#define RY_EACH3(M) RY_EACH2(M) M(2, 512)
#define RY_EACH4(M) RY_EACH3(M) M(3, 768)
#define RY_EACH5(M) RY_EACH4(M) M(4, 1024)
#define RY_EACH6(M) RY_EACH5(M) M(5, 1280)
#define RY_EPILOGUE(EACH, EPC)                                     \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_load_dwordx16 s[48:63], %[rows], 0\n"                       \
    "s_load_dwordx16 s[64:79], %[bias], 0\n"                       \
    "v_subrev_u32 v[%[t]+1], %[base], %[vl]\n"                     \
    "v_add_u32 v[%[t]+1], %[yo], v[%[t]+1]\n"                      \
    EACH(RY_EPL)                                                   \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    RY_EPROW(EPC, 0) RY_EPROW(EPC, 1) RY_EPROW(EPC, 2) RY_EPROW(EPC, 3)      \
    RY_EPROW(EPC, 4) RY_EPROW(EPC, 5) RY_EPROW(EPC, 6) RY_EPROW(EPC, 7)      \
    RY_EPROW(EPC, 8) RY_EPROW(EPC, 9) RY_EPROW(EPC, 10) RY_EPROW(EPC, 11)    \
    RY_EPROW(EPC, 12) RY_EPROW(EPC, 13) RY_EPROW(EPC, 14) RY_EPROW(EPC, 15)

#define RY_IDX_ON "s_set_gpr_idx_on 0, gpr_idx(SRC2,DST)\n"

// Batch J of the six-batch loop: records in buffer RC (record 1 at RC1), the
// next batch's at RN, loads into RNN; activations in set XC, the next
// batch's into XN.  Falls through to batch J + 1; a chunk's last batch goes
// to its out-of-line transition TR<J>.
#define RY_BODY(J, REC, COLS, XL, F, RC, RC1, RN, RNN, XC0, XC1, XN0, XN1)   \
    "LB" #J "_%=:\n"                                                         \
    "s_waitcnt lgkmcnt(0)\n"                                                 \
    "s_load_dwordx16 s[" #RNN ":" #RNN "+15], %[ptr], s35\n"                \
    "s_add_u32 s35, s35, 64\n"                                               \
    "s_bitcmp1_b32 s[" #RC "+" #F "], 0\n"                                   \
    "s_cbranch_scc1 TR" #J "_%=\n"                                           \
    "s_set_gpr_idx_idx 0\n"                                                  \
    RY_PREF(XL, RN, XN0, XN1)                                                \
    REC(COLS, XC0, RC, "B" #J "a") REC(COLS, XC1, RC1, "B" #J "b")
// The transition after batch J's wait and record load: at the stream's last
// batch compute it, release its chunk and finish; else enter the next chunk,
// prefetch, compute, release this chunk and go on with batch J + 1.
#define RY_TRANS(J, JN, REC, COLS, XL, F, CPW, RC, RC1, RN, XC0, XC1, XN0, XN1)   \
    "TR" #J "_%=:\n"                                                         \
    "s_set_gpr_idx_off\n"                                                    \
    "s_bitcmp1_b32 s[" #RC "+" #F "], 1\n"                                   \
    "s_cbranch_scc1 TE" #J "_%=\n"                                           \
    RY_ENTER("E" #J)                                                         \
    RY_IDX_ON                                                                \
    RY_PREF(XL, RN, XN0, XN1)                                                \
    REC(COLS, XC0, RC, "T" #J "a") REC(COLS, XC1, RC1, "T" #J "b")           \
    "s_set_gpr_idx_off\n"                                                    \
    RY_LEAVE("L" #J, CPW)                                                    \
    "s_add_u32 s34, s34, 1\n"                                                \
    "s_mov_b32 s40, s46\n"                                                   \
    "s_mov_b32 s41, s47\n"                                                   \
    RY_IDX_ON                                                                \
    "s_branch LB" #JN "_%=\n"                                                \
    "TE" #J "_%=:\n"                                                         \
    RY_IDX_ON                                                                \
    REC(COLS, XC0, RC, "U" #J "a") REC(COLS, XC1, RC1, "U" #J "b")           \
    "s_set_gpr_idx_off\n"                                                    \
    RY_LEAVE("M" #J, CPW)                                                    \
    "s_branch DN_%=\n"

#define RY_ZV(k) \
    "v_mov_b32 v[%[a]+16*" #k "+0], 0\n v_mov_b32 v[%[a]+16*" #k "+1], 0\n v_mov_b32 v[%[a]+16*" #k "+2], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+3], 0\n v_mov_b32 v[%[a]+16*" #k "+4], 0\n v_mov_b32 v[%[a]+16*" #k "+5], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+6], 0\n v_mov_b32 v[%[a]+16*" #k "+7], 0\n v_mov_b32 v[%[a]+16*" #k "+8], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+9], 0\n v_mov_b32 v[%[a]+16*" #k "+10], 0\n v_mov_b32 v[%[a]+16*" #k "+11], 0\n"    \
    "v_mov_b32 v[%[a]+16*" #k "+12], 0\n v_mov_b32 v[%[a]+16*" #k "+13], 0\n v_mov_b32 v[%[a]+16*" #k "+14], 0\n"   \
    "v_mov_b32 v[%[a]+16*" #k "+15], 0\n"
#define RY_Z1 RY_ZV(0)
#define RY_Z2 RY_Z1 RY_ZV(1)
#define RY_Z3 RY_Z2 RY_ZV(2)
#define RY_Z4 RY_Z3 RY_ZV(3)
#define RY_Z5 RY_Z4 RY_ZV(4)
#define RY_Z6 RY_Z5 RY_ZV(5)

// The whole statement.
#define RY_STREAM(REC, F, COLS, XL, ZC, CPW, EACH, EPC, CLOBV)                                     \
    asm volatile(ZC                                                                                     \
                 "s_mov_b32 s34, 0\n"                                                                   \
                 "s_mov_b32 s38, %[pend]\n"                                                             \
                 "s_load_dwordx16 s[48:63], %[ptr], 0\n"                                                \
                 "s_load_dwordx16 s[64:79], %[ptr], 64\n"                                               \
                 "s_mov_b32 s35, 128\n"                                                                 \
                 "s_mov_b32 s40, 0\n"                                                                   \
                 "s_mov_b32 s41, 0\n"                                                                   \
                 "s_mov_b32 s46, 0\n"                                                                   \
                 "s_mov_b32 s47, 0\n"                                                                   \
                 RY_WAITFILL("E")                                                                       \
                 "s_waitcnt lgkmcnt(0)\n"                                                               \
                 RY_IDX_ON                                                                              \
                 RY_PREF(XL, 48, xa0, xa1)                                                              \
                 RY_BODY(0, REC, COLS, XL, F, 48, 56, 64, 80, xa0, xa1, xb0, xb1)                       \
                 RY_BODY(1, REC, COLS, XL, F, 64, 72, 80, 48, xb0, xb1, xa0, xa1)                       \
                 RY_BODY(2, REC, COLS, XL, F, 80, 88, 48, 64, xa0, xa1, xb0, xb1)                       \
                 RY_BODY(3, REC, COLS, XL, F, 48, 56, 64, 80, xb0, xb1, xa0, xa1)                       \
                 RY_BODY(4, REC, COLS, XL, F, 64, 72, 80, 48, xa0, xa1, xb0, xb1)                       \
                 RY_BODY(5, REC, COLS, XL, F, 80, 88, 48, 64, xb0, xb1, xa0, xa1)                       \
                 "s_branch LB0_%=\n"                                                                    \
                 RY_TRANS(0, 1, REC, COLS, XL, F, CPW, 48, 56, 64, xa0, xa1, xb0, xb1)             \
                 RY_TRANS(1, 2, REC, COLS, XL, F, CPW, 64, 72, 80, xb0, xb1, xa0, xa1)             \
                 RY_TRANS(2, 3, REC, COLS, XL, F, CPW, 80, 88, 48, xa0, xa1, xb0, xb1)             \
                 RY_TRANS(3, 4, REC, COLS, XL, F, CPW, 48, 56, 64, xb0, xb1, xa0, xa1)             \
                 RY_TRANS(4, 5, REC, COLS, XL, F, CPW, 64, 72, 80, xa0, xa1, xb0, xb1)             \
                 RY_TRANS(5, 0, REC, COLS, XL, F, CPW, 80, 88, 48, xb0, xb1, xa0, xa1)             \
                 "DN_%=:\n"                                                                             \
                 "s_setprio 0\n"                                                                        \
                 RY_PUBLISH("FP")                                                                       \
                 RY_EPILOGUE(EACH, EPC)                                                                 \
                 :                                                                                      \
                 : [a] "i"(L::A), [xa0] "i"(L::XA0), [xa1] "i"(L::XA1), [xb0] "i"(L::XB0),              \
                   [xb1] "i"(L::XB1), [t] "i"(L::T), [cbytes] "i"(kChunk * kRingRowBytes), [spin] "s"(spin),  \
                   [ptr] "s"(ptr), [nch] "s"(nch), [ctl] "s"(ctl), [nw] "s"(nw), [rs] "s"(rs),          \
                   [xo] "s"(xo), [yo] "s"(yo), [pat] "s"(pat), [cin] "s"(cin), [hw4] "s"(hw4),          \
                   [base] "s"(base), [flag] "s"(flag), [rows] "s"(rows), [bias] "s"(bias),              \
                   [ry] "s"(ry), [v4] "s"(v4), [nws] "s"(nws), [pend] "s"(pend), [vl] "v"(vl),          \
                   [lo] "v"(lo), [hi] "v"(hi)                                                           \
                 : "memory", "m0", "scc", "vcc", CLOBV, IY_CLOBS)

template <int K, int C>
__device__ __forceinline__ void stream_asm(const uint32_t *ptr, int32_t nch, uint32_t ctl, int32_t nw, i4 rs,
                                           uint32_t xo, uint32_t yo, uint32_t pat, int32_t cin, int32_t hw4,
                                           uint32_t base, int32_t *flag, const int32_t *rows, const float *bias,
                                           i4 ry, int32_t v4, int32_t nws, int32_t pend, int32_t spin, int32_t vl,
                                           float lo, float hi) {
    using L = Lay<C>;
#define RY_BY_C(REC, F)                                                                                \
    if constexpr (C == 1) {                                                                            \
        RY_STREAM(REC, F, RY_C1, RY_XL1, RY_Z1, RY_CPW1, RY_EACH1, RY_EPC1, IY_CLOBV1);       \
    } else if constexpr (C == 2) {                                                                     \
        RY_STREAM(REC, F, RY_C2, RY_XL2, RY_Z2, RY_CPW2, RY_EACH2, RY_EPC2, IY_CLOBV2);       \
    } else if constexpr (C == 3) {                                                                     \
        RY_STREAM(REC, F, RY_C3, RY_XL3, RY_Z3, RY_CPW3, RY_EACH3, RY_EPC3, IY_CLOBV3);       \
    } else if constexpr (C == 4) {                                                                     \
        RY_STREAM(REC, F, RY_C4, RY_XL4, RY_Z4, RY_CPW4, RY_EACH4, RY_EPC4, IY_CLOBV4);       \
    } else if constexpr (C == 5) {                                                                     \
        RY_STREAM(REC, F, RY_C5, RY_XL5, RY_Z5, RY_CPW5, RY_EACH5, RY_EPC5, IY_CLOBV5);       \
    } else {                                                                                           \
        RY_STREAM(REC, F, RY_C6, RY_XL6, RY_Z6, RY_CPW6, RY_EACH6, RY_EPC6, IY_CLOBV6);       \
    }
    if constexpr (K == 1) {
        RY_BY_C(RY_REC_K1, 7)
    } else if constexpr (K == 2) {
        RY_BY_C(RY_REC_K2, 3)
    } else {
        RY_BY_C(RY_REC_K4, 3)
    }
#undef RY_BY_C
}

// ---------------------------------------------------------------------------
// Per-task control
// ---------------------------------------------------------------------------

// The column offsets of column j: x / y byte offsets relative to image n0,
// kOOR past the end.
__device__ __forceinline__ void col_offsets(KArgs &a, int32_t j, int32_t n0, int32_t &xo, int32_t &yo) {
    if (j < a.m) {
        const int32_t n = j / a.hw;
        const int32_t p = j - n * a.hw;
        xo = ((n - n0) * a.cin * a.hw + p) * 4;
        yo = ((n - n0) * a.cout * a.hw + p) * 4;
    } else {
        xo = kOOR;
        yo = kOOR;
    }
}

// Where a task's pieces live: its tile, slot group, this wave's slot, the
// wavefronts with a slot, the tile's first column and image.
struct TaskPos {
    int32_t tile, group, slot, nw, col0, n0;
};

template <int C>
__device__ __forceinline__ TaskPos task_pos(KArgs &a, int32_t task, int wave) {
    TaskPos t;
    t.tile = task / a.groups;
    t.group = task - t.tile * a.groups;
    t.slot = t.group * a.waves + wave;
    t.nw = imin(a.waves, a.slots - t.group * a.waves);
    t.col0 = t.tile * 64 * C;
    t.n0 = t.col0 / a.hw;
    return t;
}

// Copy pattern j (0, 1, 2) of a lane for 16-byte ring copies: two ring rows
// are 3 KiB, filled by three 1 KiB loads; the x offset of the four columns
// load j brings into bytes 1024 j + 16 lane of them, kOOR where those bytes
// are a column slot past C or past the last column.
template <int C>
__device__ __forceinline__ int32_t copy_pattern(KArgs &a, const TaskPos &t, int lane, int j) {
    const int32_t o = 1024 * j + 16 * lane;
    const int32_t r = o >= kRingRowBytes ? 1 : 0;          // second row of the pair
    const int32_t within = o - r * kRingRowBytes;
    const int32_t k = within >> 8;                          // column slot
    const int32_t lc = (within & 255) >> 2;                 // first of four lane columns
    if (k >= C)
        return kOOR;
    int32_t xo, yo;
    col_offsets(a, t.col0 + 64 * k + lc, t.n0, xo, yo);
    return xo == kOOR ? kOOR : xo + r * a.hw * 4;
}

// Set-up of a task: lane column tables, copy patterns and counters into LDS,
// then the first ring's worth of channels copied by every wavefront: its
// share of chunk 0 first, waited for and published at once, then its shares
// of chunks 1 .. 5, published later (in the stream at the wavefront's first
// chunk release, or here by a wavefront without a slot).  Returns the
// bit set of ring chunks this wavefront still has to publish.
__device__ __forceinline__ void publish_fill(unsigned char *lds, int32_t ctl_off, int32_t bits, int lane) {
    if (lane < kRingChunks && ((bits >> lane) & 1))
        __hip_atomic_fetch_add(reinterpret_cast<int32_t *>(lds + ctl_off) + 8 + lane, 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int C>
__device__ __forceinline__ int32_t task_setup(int32_t task, unsigned char *lds, uint32_t lds_base, int wave,
                                              int nwaves, int lane) {
    const auto &a = kargs();
    const TaskPos t = task_pos<C>(a, task, wave);
    const int64_t xbase = static_cast<int64_t>(t.n0) * a.cin * a.hw;
    const i4 rs = rsrc_words(a.x + xbase, a.x_bytes - xbase * 4);
    int32_t *xo_lds = reinterpret_cast<int32_t *>(lds + a.xo_off);
    int32_t *yo_lds = xo_lds + 64 * C;
    int32_t *pat_lds = reinterpret_cast<int32_t *>(lds + a.pat_off);
    int32_t *freec = reinterpret_cast<int32_t *>(lds + a.ctl_off);
    const uint32_t base = lds_base;  // the ring starts at LDS byte 0
    __syncthreads();  // the previous user of LDS is done
    if (wave == 0) {
#pragma unroll 1
        for (int k = 0; k < C; ++k) {
            int32_t xo, yo;
            col_offsets(a, t.col0 + 64 * k + lane, t.n0, xo, yo);
            xo_lds[k * 64 + lane] = xo;
            yo_lds[k * 64 + lane] = yo;
        }
        pat_lds[lane] = copy_pattern<C>(a, t, lane, 0);
        pat_lds[64 + lane] = copy_pattern<C>(a, t, lane, 1);
        pat_lds[128 + lane] = copy_pattern<C>(a, t, lane, 2);
        if (lane < kRingChunks) {
            freec[lane] = 0;
            freec[8 + lane] = 0;
        }
    }
    __syncthreads();
    const int32_t hw4 = a.hw * 4;
    const int32_t nq = imin(kRingChunks, a.nch);   // chunks of the first ring
    int32_t bits = 0;
#pragma unroll 1
    for (int32_t q = 0; q < nq; ++q) {
        const int32_t c0 = q * kChunk;
        const int32_t rows = imin(kChunk, a.cin - c0);
        const uint32_t dst = base + static_cast<uint32_t>(q * kChunk * kRingRowBytes);
        if (a.v4) {
            const int32_t p0 = pat_lds[lane], p1 = pat_lds[64 + lane], p2 = pat_lds[128 + lane];
            const int32_t loads = 3 * ((rows + 1) / 2);
#pragma unroll 1
            for (int32_t u = wave; u < loads; u += nwaves) {
                const int32_t rp = u / 3, j = u - 3 * rp;
                dma_x4(dst + static_cast<uint32_t>(rp * 2 * kRingRowBytes + 1024 * j), j == 0 ? p0 : j == 1 ? p1 : p2,
                       rs, (c0 + 2 * rp) * hw4);
            }
        } else {
#pragma unroll 1
            for (int32_t u = wave; u < rows * C; u += nwaves) {
                const int32_t r = u / C, k = u - r * C;
                dma_dword(dst + static_cast<uint32_t>(r * kRingRowBytes + 256 * k), xo_lds[k * 64 + lane], rs,
                          (c0 + r) * hw4);
            }
        }
        if (q == 0) {
            wait_vm0();
            publish_fill(lds, a.ctl_off, 1, lane);
        } else {
            bits |= 1 << q;
        }
    }
    return bits;
}

// The wavefront's slot over the task's tile (the stream statement).
template <int K, int C>
__device__ __forceinline__ void task_stream(int32_t task, uint32_t lds_base, int wave, int lane, int32_t nws,
                                            int32_t pend) {
    const auto &a = kargs();
    const TaskPos t = task_pos<C>(a, task, wave);
    const int64_t xbase = static_cast<int64_t>(t.n0) * a.cin * a.hw;
    const int64_t ybase = static_cast<int64_t>(t.n0) * a.cout * a.hw;
    const i4 rs = rsrc_words(a.x + xbase, a.x_bytes - xbase * 4);
    const i4 ry = rsrc_words(a.y + ybase, a.y_bytes - ybase * 4);
    const uint32_t *ptr =
        uniform_ptr(a.rec + static_cast<int64_t>(cst(a.slot_batch)[t.slot]) * (kRecWords * kBatchRecs));
    const int32_t *rows = uniform_ptr(a.slot_rows + static_cast<int64_t>(t.slot) * kSlotRows);
    const float *bias = uniform_ptr(a.slot_bias + static_cast<int64_t>(t.slot) * kSlotRows);
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    const uint32_t xo = lds_base + static_cast<uint32_t>(a.xo_off);
    stream_asm<K, C>(ptr, __builtin_amdgcn_readfirstlane(a.nch),
                     __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(a.ctl_off)),
                     __builtin_amdgcn_readfirstlane(t.nw), rs, __builtin_amdgcn_readfirstlane(xo),
                     __builtin_amdgcn_readfirstlane(xo + 256u * C),
                     __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(a.pat_off)),
                     __builtin_amdgcn_readfirstlane(a.cin), __builtin_amdgcn_readfirstlane(a.hw * 4),
                     __builtin_amdgcn_readfirstlane(lds_base), uniform_ptr(a.flag), rows, bias, ry,
                     __builtin_amdgcn_readfirstlane(a.v4), __builtin_amdgcn_readfirstlane(nws),
                     __builtin_amdgcn_readfirstlane(pend), __builtin_amdgcn_readfirstlane(a.spin),
                     static_cast<int32_t>(lds_base) + 4 * lane, lo, hi);
}

// Columns [lcol0, m) by row pairs over 64-column groups (see the file comment).
__device__ __forceinline__ void run_pairs(unsigned char *lds, uint32_t lds_base, int wave, int nwaves, int lane) {
    const auto &a = kargs();
    const float *x = a.x;
    float *y = a.y;
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    const int32_t p0 = static_cast<int32_t>(blockIdx.x) * a.lper;
    const int32_t p1 = imin(p0 + a.lper, a.lpieces);
    const i4 re = rsrc_words(a.pair_ent, a.pair_ent_bytes);
    const int32_t hw4 = a.hw * 4;
    const int32_t epw = a.epw;
    const int32_t ent = a.ent_off + wave * epw * 16;   // this wavefront's entry area
    const auto *pp = cst(a.pair_ptr);
    // entries [e, e + n) of the pair stream into the wavefront's area, 64 per load
    auto stage = [&](int32_t e, int32_t n) {
        for (int32_t i = 0; i * 64 < n; ++i)
            dma_x4(lds_base + static_cast<uint32_t>(ent + 1024 * i), 16 * lane, re, (e + 64 * i) * 16);
    };
    int32_t pc = p0;
    while (pc < p1) {
        const int32_t cg = pc / a.pairs;
        const int32_t pe = imin(p1, (cg + 1) * a.pairs);
        const int32_t col0 = a.lcol0 + 64 * cg;
        const int32_t n0 = col0 / a.hw;
        const int64_t xbase = static_cast<int64_t>(n0) * a.cin * a.hw;
        const int64_t ybase = static_cast<int64_t>(n0) * a.cout * a.hw;
        __syncthreads();
        const i4 rs = rsrc_words(x + xbase, a.x_bytes - xbase * 4);
        if (a.v4) {
            // 1 KiB loads of four channel rows: lane l brings four columns of row l / 16
            int32_t xo, yo;
            col_offsets(a, col0 + 4 * (lane & 15), n0, xo, yo);
            const int32_t voff = xo == kOOR ? kOOR : xo + (lane >> 4) * hw4;
            const int32_t nload = (a.cin + 3) / 4;
            for (int32_t u = wave; u < nload; u += nwaves)
                dma_x4(lds_base + static_cast<uint32_t>(u * 1024), voff, rs, u * 4 * hw4);
        } else {
            int32_t xo, yo;
            col_offsets(a, col0 + lane, n0, xo, yo);
            for (int32_t c = wave; c < a.cin; c += nwaves)
                dma_dword(lds_base + static_cast<uint32_t>(c * 256), xo, rs, c * hw4);
        }
        const int32_t t0 = pc + wave;
        if (t0 < pe) {
            const int32_t pr = t0 - cg * a.pairs;
            stage(pp[pr], imin(epw, pp[pr + 1] - pp[pr]));
        }
        wait_vm0();
        __syncthreads();
        int32_t xo, yo;
        col_offsets(a, col0 + lane, n0, xo, yo);
        const Rsrc ry = make_rsrc(y + ybase, a.y_bytes - ybase * 4);
        const float *strip = reinterpret_cast<const float *>(lds);
        const i4 *area = reinterpret_cast<const i4 *>(lds + ent);
        for (int32_t t = t0; t < pe; t += nwaves) {
            const int32_t pr = t - cg * a.pairs;
            const int32_t e0 = pp[pr], e1 = pp[pr + 1];
            float acc0 = 0.0f, acc1 = 0.0f;
            for (int32_t eb = e0; eb < e1; eb += epw) {
                const int32_t n = imin(epw, e1 - eb);
                if (t != t0 || eb != e0) {
                    stage(eb, n);
                    wait_vm0();
                }
                // entries: channel | mask << 24, weight of row 2 pr, of row 2 pr + 1 (0 where absent)
#pragma unroll 4
                for (int32_t j = 0; j < n; ++j) {
                    const i4 w = area[j];
                    const float xv = strip[(w.x & 0xffffff) * 64 + lane];
                    acc0 = __builtin_fmaf(__int_as_float(w.y), xv, acc0);
                    acc1 = __builtin_fmaf(__int_as_float(w.z), xv, acc1);
                }
            }
            const int32_t r0 = 2 * pr;
            const auto *rb = cst(a.row_bias);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fminf(fmaxf(acc0 + rb[r0], lo), hi)), ry,
                                                  yo, r0 * hw4, 0);
            if (r0 + 1 < a.cout)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fminf(fmaxf(acc1 + rb[r0 + 1], lo), hi)), ry,
                                                      yo, (r0 + 1) * hw4, 0);
        }
        pc = pe;
    }
}

template <int K, int C>
__device__ __forceinline__ void indexed_body() {
    extern __shared__ __align__(16) unsigned char lds[];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nwaves = static_cast<int>(blockDim.x >> 6);
    const uint32_t lds_base = static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) unsigned char *)lds));
    // one whole-tile task per workgroup (the grid has a workgroup per task)
    const int32_t task = static_cast<int32_t>(blockIdx.x);
    if (task < kargs().main_tasks) {
        const int32_t pend = task_setup<C>(task, lds, lds_base, wave, nwaves, lane);
        if (wave < task_pos<C>(kargs(), task, wave).nw) {
            task_stream<K, C>(task, lds_base, wave, lane, nwaves, pend);
        } else {
            wait_vm0();
            publish_fill(lds, kargs().ctl_off, pend, lane);
        }
    }
    if (kargs().lpieces > 0)
        run_pairs(lds, lds_base, wave, nwaves, lane);
}

// One kernel per column count C.
#define IY_KERNEL(CC)                                                     \
    template <int K>                                                      \
    __global__ void __launch_bounds__(1024) spmm_indexed_c##CC(IArgs) {  \
        indexed_body<K, CC>();                                            \
    }
IY_KERNEL(1)
IY_KERNEL(2)
IY_KERNEL(3)
IY_KERNEL(4)
IY_KERNEL(5)
IY_KERNEL(6)

using IKernel = void (*)(IArgs);

template <int K>
IKernel pick_c(int c) {
    switch (c) {
    case 1: return spmm_indexed_c1<K>;
    case 2: return spmm_indexed_c2<K>;
    case 3: return spmm_indexed_c3<K>;
    case 4: return spmm_indexed_c4<K>;
    case 5: return spmm_indexed_c5<K>;
    case 6: return spmm_indexed_c6<K>;
    default: return nullptr;
    }
}

IKernel pick_indexed(int k, int c) {
    if (k == 1)
        return pick_c<1>(c);
    if (k == 2)
        return pick_c<2>(c);
    if (k == 4)
        return pick_c<4>(c);
    return nullptr;
}

}  // namespace

IndexedLaunch plan_indexed_launch(const DevicePlan &p, int64_t m) {
    IndexedLaunch best;
    const int64_t W = p.rwaves;
    const int64_t G = p.rgroups;
    // the ring holds min(kRing, cin rounded up to a chunk) rows, so a layer
    // with few input channels leaves LDS for more workgroups per CU
    const int32_t ring_rows = std::min<int32_t>(kRing, p.rnch * kChunk);
    const int64_t main_lds_max = static_cast<int64_t>(ring_rows) * kRingRowBytes + 64 + 2 * 256 * 6 + 3 * 256;
    const int64_t wg_per_cu =
        std::max<int64_t>(1, std::min<int64_t>(kMaxWaves / W, kMaxLdsBytes / main_lds_max));
    const int64_t grid = static_cast<int64_t>(p.num_cus) * wg_per_cu;
    const int64_t pairs = (p.cout + 1) / 2;
    // row pairs: the strip of cin channel rows (256 bytes each, whole 1 KiB
    // loads), then an entry area of epw 16-byte entries per wavefront
    const int64_t strip_bytes = static_cast<int64_t>((p.cin + 3) / 4) * 1024;
    const int64_t epw = std::min<int64_t>(256, (kMaxLdsBytes - strip_bytes) / (W * 16) / 64 * 64);
    const bool pairs_fit = epw >= 64;
    // Cost in wave-work units: a task of c columns per lane costs c per wave
    // plus a fixed start-up of 1; a row-pair piece (2 rows x 64 columns, one
    // LDS read per nonzero) costs a quarter.
    double best_cost = 1e30;
    for (int c = 1; c <= 6; ++c) {
        const int64_t tc = 64 * c;
        // uniform tiles
        {
            const int64_t tiles = (m + tc - 1) / tc;
            const int64_t rounds = (tiles * G + grid - 1) / grid;
            const double cost = rounds * (c + 1.0);
            if (cost < best_cost) {
                best_cost = cost;
                best.c = c;
                best.tiles = tiles;
                best.lcol0 = static_cast<int32_t>(tiles * tc);
                best.lpieces = 0;
            }
        }
        // one round of whole tiles, the rest by row pairs (their LDS strip
        // would leave one workgroup per CU, so only where that is all the
        // ring leaves anyway)
        if (pairs_fit && wg_per_cu == 1 && grid % G == 0) {
            const int64_t tiles = std::min<int64_t>(grid / G, m / tc);
            if (tiles >= 1) {
                const int64_t left = m - tiles * tc;
                const int64_t pieces = (left + 63) / 64 * pairs;
                const int64_t per_wave = (pieces + grid * W - 1) / (grid * W);
                const double cost = (c + 1.0) + 0.25 * per_wave + (pieces ? 0.5 : 0.0);
                if (cost < best_cost) {
                    best_cost = cost;
                    best.c = c;
                    best.tiles = tiles;
                    best.lcol0 = static_cast<int32_t>(tiles * tc);
                    best.lpieces = static_cast<int32_t>(pieces);
                }
            }
        }
    }
    best.grid = static_cast<int32_t>(std::max<int64_t>(best.tiles * G, 1));
    if (best.lpieces > 0)
        best.grid = static_cast<int32_t>(std::max<int64_t>(best.grid, grid));
    best.lper = best.lpieces ? (best.lpieces + best.grid - 1) / best.grid : 0;
    // LDS: the ring, 64 bytes of counters, the lane x and y column tables
    // (256 C bytes each), three copy patterns.
    best.ctl_off = ring_rows * kRingRowBytes;
    best.xo_off = best.ctl_off + 64;
    best.pat_off = best.xo_off + 2 * 256 * best.c;
    const int32_t main_lds = best.pat_off + 3 * 256;
    best.ent_off = static_cast<int32_t>(strip_bytes);
    best.epw = best.lpieces ? static_cast<int32_t>(epw) : 0;
    const int32_t pair_lds = best.lpieces ? static_cast<int32_t>(strip_bytes + W * 16 * epw) : 0;
    best.lds_bytes = std::max(main_lds, pair_lds);
    return best;
}

hipError_t prepare_indexed(const DevicePlan &p) {
    for (int c = 1; c <= 6; ++c) {
        IKernel kern = pick_indexed(p.k, c);
        if (!kern)
            return hipErrorInvalidValue;
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 static_cast<int>(kMaxLdsBytes));
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t launch_indexed(const DevicePlan &p, const float *x, float *y, int32_t m, int32_t hw, int64_t x_bytes,
                          int64_t y_bytes, hipStream_t stream) {
    const IndexedLaunch L = plan_indexed_launch(p, m);
    IKernel kern = pick_indexed(p.k, L.c);
    if (!kern)
        return hipErrorInvalidValue;
    IArgs a;
    a.x = x;
    a.y = y;
    a.cin = p.cin;
    a.cout = p.cout;
    a.hw = hw;
    a.m = m;
    a.act = p.act;
    a.x_bytes = x_bytes;
    a.y_bytes = y_bytes;
    a.nch = p.rnch;
    a.slots = p.rslots;
    a.groups = p.rgroups;
    a.waves = p.rwaves;
    a.main_tasks = static_cast<int32_t>(L.tiles * p.rgroups);
    a.lcol0 = L.lcol0;
    a.lpieces = L.lpieces;
    a.lper = L.lper;
    a.pairs = (p.cout + 1) / 2;
    a.v4 = (hw % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0) ? 1 : 0;
    a.ctl_off = L.ctl_off;
    a.xo_off = L.xo_off;
    a.pat_off = L.pat_off;
    a.ent_off = L.ent_off;
    a.epw = L.epw;
    a.rec = p.rrec;
    a.slot_batch = p.rslot_batch;
    a.slot_rows = p.rslot_rows;
    a.slot_bias = p.rslot_bias;
    a.pair_ptr = p.rpair_ptr;
    a.pair_ent = p.rpair_ent;
    a.pair_ent_bytes = static_cast<int64_t>(p.rpair_ent_words) * 4;
    a.row_bias = p.rrow_bias;
    a.flag = p.flag;
    a.spin = p.spin_limit;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(L.grid)), dim3(p.rwaves * 64), L.lds_bytes, stream, a);
    return hipGetLastError();
}

}  // namespace spconv
