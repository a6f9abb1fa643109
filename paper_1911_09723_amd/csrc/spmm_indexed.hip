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
//     at run time with register-relative addressing: s_set_gpr_idx_on /
//     _idx put the row in M0 and the FMA's accumulator operand (source 2 and
//     destination) is offset by it.  One index change per nonzero (SALU, one
//     per cycle per CU) feeds C FMAs (VALU), so C is as large as the
//     registers allow.
//   * Records (planner.hpp) carry, per channel, the slot rows and weights of
//     up to 3 (1x1), 2 (1x2) or 1 (1x4 block) nonzeros, two records per
//     64-byte batch.  Each batch's records are loaded with one scalar load a
//     batch ahead into two alternating buffers of reserved SGPRs, and each
//     record's activations are read from LDS one record ahead into reserved
//     VGPRs, so every wait finds its data nearly always already there.
//   * X reaches LDS by buffer loads that write LDS directly (one dword per
//     lane and column), into a ring of 64 channel rows in 4 chunks of 16.
//     The last wavefront to finish with a chunk refills its ring rows with the
//     chunk 4 ahead and publishes it at its next chunk boundary; a wavefront
//     waits only for the chunk it is about to read.
//
// Every row sums its products in ascending input channel from zero with fp32
// FMA and adds the bias last, exactly as the other kernels of this library do,
// so the result does not depend on the kernel, the slot assignment or the
// tile split.
//
// Register plan (per C): compiler-managed v0 .. NV-1 and s0 .. 63; reserved
// accumulators v[A + 16 k + r] (column k, slot row r), activation buffers
// X0/X1 (C each, rounded up to even), two LDS addresses VA0/VA1, record
// buffers s64 .. s95.
//
// Columns left over after the last whole tile round are computed by row
// pairs: each wavefront takes two output channels over 64 columns, with a
// plain loop reading the columns' activations from an LDS strip.
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
constexpr int kSB = 64;            // first reserved SGPR (two 16-dword record buffers)
constexpr int32_t kSpinMax = 1 << 22;

template <int C>
struct Lay {
    static constexpr int XS = (C + 1) & ~1;  // an activation buffer, even-aligned for pair reads
    static constexpr int A = 112 - 16 * C;   // accumulators v[A + 16 k + r], up to v111
    static constexpr int X0 = 112;
    static constexpr int X1 = X0 + XS;
    static constexpr int VA0 = X1 + XS;
    static constexpr int VA1 = VA0 + 1;
    static constexpr int T = VA1 + 1;        // two temporaries
    static constexpr int SHIFT = C <= 1 ? 8 : C <= 2 ? 9 : C <= 4 ? 10 : 11;  // log2 of a ring row's bytes
    static_assert(T + 1 <= 127, "register plan must end by v127");
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
    int32_t ring_off;     // LDS byte offsets: ring (0), counters, lane offsets
    int32_t ctl_off, xo_off;
    const uint32_t *rec;
    const int32_t *slot_batch, *slot_chunk, *slot_rows;
    const float *slot_bias;
    const int32_t *pair_ptr;
    const uint32_t *pair_ent;
    const float *row_bias;
    int32_t *flag;        // set when a bounded wait gives up
};

// The launch arguments, read afresh from the kernel-argument segment: the
// pointer passes through an empty asm statement, so the compiler reloads the
// fields where each phase of the kernel uses them instead of holding every
// argument in scalar registers for the whole kernel (the reserved record
// buffers leave it 64).
typedef const __attribute__((address_space(4))) IArgs KArgs;

__device__ __forceinline__ KArgs &kargs() {
    const IArgs *p = (const IArgs *)(__builtin_amdgcn_kernarg_segment_ptr());
    asm volatile("" : "+s"(p));
    return *cst(p);
}

// Clobber lists of the stream statement: every register it uses for itself.
#define IX_CLOBV1 "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119"
#define IX_CLOBV2 "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119"
#define IX_CLOBV3 "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123"
#define IX_CLOBV4 "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123"
#define IX_CLOBV5 "v32", "v33", "v34", "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45", "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IX_CLOBV6 "v16", "v17", "v18", "v19", "v20", "v21", "v22", "v23", "v24", "v25", "v26", "v27", "v28", "v29", "v30", "v31", "v32", "v33", "v34", "v35", "v36", "v37", "v38", "v39", "v40", "v41", "v42", "v43", "v44", "v45", "v46", "v47", "v48", "v49", "v50", "v51", "v52", "v53", "v54", "v55", "v56", "v57", "v58", "v59", "v60", "v61", "v62", "v63", "v64", "v65", "v66", "v67", "v68", "v69", "v70", "v71", "v72", "v73", "v74", "v75", "v76", "v77", "v78", "v79", "v80", "v81", "v82", "v83", "v84", "v85", "v86", "v87", "v88", "v89", "v90", "v91", "v92", "v93", "v94", "v95", "v96", "v97", "v98", "v99", "v100", "v101", "v102", "v103", "v104", "v105", "v106", "v107", "v108", "v109", "v110", "v111", "v112", "v113", "v114", "v115", "v116", "v117", "v118", "v119", "v120", "v121", "v122", "v123", "v124", "v125", "v126", "v127"
#define IX_CLOBS "s40", "s41", "s42", "s43", "s44", "s45", "s46", "s47", "s48", "s49", "s50", "s51", "s52", "s53", "s54", "s55", "s56", "s57", "s58", "s59", "s60", "s61", "s62", "s63", "s64", "s65", "s66", "s67", "s68", "s69", "s70", "s71", "s72", "s73", "s74", "s75", "s76", "s77", "s78", "s79", "s80", "s81", "s82", "s83", "s84", "s85", "s86", "s87", "s88", "s89", "s90", "s91", "s92", "s93", "s94", "s95"

// ---------------------------------------------------------------------------
// The stream statement.  One inline-assembly statement runs a wavefront's
// whole slot over one tile: zero the accumulators, walk the chunks (wait for
// each, run its batches, release it, refill the ring quarter it frees when
// this wavefront is the last to release it), then bias, activation and store.
// Inside it the compiler places nothing, so the accumulators, activation
// buffers and record buffers are simply registers it was told are clobbered.
//
// Scalar registers of the statement: s40 chunk q, s41 batch b, s42 end batch
// of the chunk, s43 "records of the first batch not loaded yet", s44 the
// chunk's record count is odd, s45 ring quarters copied but not yet published,
// s46-s49, s52-s53 temporaries, s50:51 saved exec, s64-s79 / s80-s95 the two
// record buffers.  Vector: accumulators v[a + 16 k + r], activation buffers
// x0 / x1, their LDS addresses va0 / va1, temporaries t, t + 1.
// ---------------------------------------------------------------------------

#define RX_FMA(k, i, X, SB, W) \
    "v_fma_f32 v[%[a]+16*" #k "+" #i "], v[%[" #X "]+" #k "], s[%[" #SB "]+" #W "], v[%[a]+16*" #k "+" #i "]\n"
#define RX_C1(i, X, SB, W) RX_FMA(0, i, X, SB, W)
#define RX_C2(i, X, SB, W) RX_C1(i, X, SB, W) RX_FMA(1, i, X, SB, W)
#define RX_C3(i, X, SB, W) RX_C2(i, X, SB, W) RX_FMA(2, i, X, SB, W)
#define RX_C4(i, X, SB, W) RX_C3(i, X, SB, W) RX_FMA(3, i, X, SB, W)
#define RX_C5(i, X, SB, W) RX_C4(i, X, SB, W) RX_FMA(4, i, X, SB, W)
#define RX_C6(i, X, SB, W) RX_C5(i, X, SB, W) RX_FMA(5, i, X, SB, W)

// The activations of one record: C dwords, ring-row stride apart (256 B).
#define RX_XL1(X, VA) "ds_read_b32 v[%[" #X "]], v[%[" #VA "]]\n"
#define RX_XL2(X, VA) "ds_read2st64_b32 v[%[" #X "]:%[" #X "]+1], v[%[" #VA "]] offset1:1\n"
#define RX_XL3(X, VA) RX_XL2(X, VA) "ds_read_b32 v[%[" #X "]+2], v[%[" #VA "]] offset:512\n"
#define RX_XL4(X, VA) RX_XL2(X, VA) "ds_read2st64_b32 v[%[" #X "]+2:%[" #X "]+3], v[%[" #VA "]] offset0:2 offset1:3\n"
#define RX_XL5(X, VA) RX_XL4(X, VA) "ds_read_b32 v[%[" #X "]+4], v[%[" #VA "]] offset:1024\n"
#define RX_XL6(X, VA) RX_XL4(X, VA) "ds_read2st64_b32 v[%[" #X "]+4:%[" #X "]+5], v[%[" #VA "]] offset0:4 offset1:5\n"

// One record in buffer SB at word W1 - 1: up to 3 rows (1x1), 2 blocks (1x2)
// or 1 block (1x4).  L: a label name unique within the statement.
#define RX_REC_K1(COLS, X, SB, W1, W2, W3, WA, WB, WC, L)       \
    "s_set_gpr_idx_on s[%[" #SB "]+" #W1 "], gpr_idx(SRC2,DST)\n" \
    COLS(0, X, SB, WA)                                           \
    "s_bitcmp1_b32 s[%[" #SB "]+" #W1 "], 8\n"                    \
    "s_cbranch_scc0 " L "_%=\n"                                   \
    "s_set_gpr_idx_idx s[%[" #SB "]+" #W2 "]\n"                   \
    COLS(0, X, SB, WB)                                           \
    "s_bitcmp1_b32 s[%[" #SB "]+" #W1 "], 9\n"                    \
    "s_cbranch_scc0 " L "_%=\n"                                   \
    "s_set_gpr_idx_idx s[%[" #SB "]+" #W3 "]\n"                   \
    COLS(0, X, SB, WC)                                           \
    L "_%=:\n"                                                    \
    "s_set_gpr_idx_off\n"
#define RX_REC_K2(COLS, X, SB, W1, W2, WA, WB, WC, WD, L)        \
    "s_set_gpr_idx_on s[%[" #SB "]+" #W1 "], gpr_idx(SRC2,DST)\n" \
    COLS(0, X, SB, WA) COLS(1, X, SB, WB)                        \
    "s_bitcmp1_b32 s[%[" #SB "]+" #W1 "], 8\n"                    \
    "s_cbranch_scc0 " L "_%=\n"                                   \
    "s_set_gpr_idx_idx s[%[" #SB "]+" #W2 "]\n"                   \
    COLS(0, X, SB, WC) COLS(1, X, SB, WD)                        \
    L "_%=:\n"                                                    \
    "s_set_gpr_idx_off\n"
#define RX_REC_K4(COLS, X, SB, W1, WA, WB, WC, WD, L)            \
    "s_set_gpr_idx_on s[%[" #SB "]+" #W1 "], gpr_idx(SRC2,DST)\n" \
    COLS(0, X, SB, WA) COLS(1, X, SB, WB) COLS(2, X, SB, WC) COLS(3, X, SB, WD) \
    "s_set_gpr_idx_off\n"

#define RX_R0_K1(COLS, SB, L) RX_REC_K1(COLS, x0, SB, 1, 2, 3, 4, 5, 6, L)
#define RX_R1_K1(COLS, SB, L) RX_REC_K1(COLS, x1, SB, 9, 10, 11, 12, 13, 14, L)
#define RX_R0_K2(COLS, SB, L) RX_REC_K2(COLS, x0, SB, 1, 2, 4, 5, 6, 7, L)
#define RX_R1_K2(COLS, SB, L) RX_REC_K2(COLS, x1, SB, 9, 10, 12, 13, 14, 15, L)
#define RX_R0_K4(COLS, SB, L) RX_REC_K4(COLS, x0, SB, 1, 4, 5, 6, 7, L)
#define RX_R1_K4(COLS, SB, L) RX_REC_K4(COLS, x1, SB, 9, 12, 13, 14, 15, L)

// Batches (records in SB; the next batch's records are loaded into SN from
// byte offset s47 of the stream).  A batch inside a chunk also reads the next
// batch's activations; the last batch of a chunk does not (the next chunk
// may not have landed).  XN: LDS instructions of one activation load.
#define RX_HEAD(XN, SN) "s_waitcnt lgkmcnt(" #XN ")\n" "s_load_dwordx16 s[%[" #SN "]:%[" #SN "]+15], %[ptr], s47\n"
#define RX_MID(SN)                                                 \
    "s_waitcnt lgkmcnt(0)\n"                                        \
    "v_lshl_add_u32 v[%[va0]], s[%[" #SN "]], %[sh], %[vl]\n"       \
    "v_lshl_add_u32 v[%[va1]], s[%[" #SN "]+8], %[sh], %[vl]\n"
#define RX_FULL(R0, R1, COLS, XL, XN, SB, SN, L) \
    RX_HEAD(XN, SN) R0(COLS, SB, L "a") RX_MID(SN) XL(x0, va0) R1(COLS, SB, L "b") XL(x1, va1)
#define RX_LAST2(R0, R1, COLS, XL, XN, SB, SN, L) \
    RX_HEAD(XN, SN) R0(COLS, SB, L "a") "s_waitcnt lgkmcnt(0)\n" R1(COLS, SB, L "b")
#define RX_LAST1(R0, R1, COLS, XL, XN, SB, SN, L) RX_HEAD(XN, SN) R0(COLS, SB, L "a")

// The batches [s41, s42) of a chunk whose first records are (or, for the first
// chunk of the stream, are loaded here) in buffer SB.
#define RX_RUN(R0, R1, COLS, XL, XN, SB, SN, L)                                   \
    "s_cmp_eq_u32 s43, 0\n"                                                        \
    "s_cbranch_scc1 " L "nf_%=\n"                                                  \
    "s_lshl_b32 s46, s41, 6\n"                                                     \
    "s_load_dwordx16 s[%[" #SB "]:%[" #SB "]+15], %[ptr], s46\n"                   \
    "s_mov_b32 s43, 0\n"                                                           \
    L "nf_%=:\n"                                                                   \
    "s_waitcnt lgkmcnt(0)\n"                                                       \
    "v_lshl_add_u32 v[%[va0]], s[%[" #SB "]], %[sh], %[vl]\n"                      \
    "v_lshl_add_u32 v[%[va1]], s[%[" #SB "]+8], %[sh], %[vl]\n"                    \
    XL(x0, va0) XL(x1, va1)                                                        \
    L "lp_%=:\n"                                                                   \
    "s_add_u32 s46, s41, 2\n"                                                      \
    "s_cmp_ge_u32 s46, s42\n"                                                      \
    "s_cbranch_scc1 " L "tl_%=\n"                                                  \
    "s_add_u32 s47, s41, 1\n"                                                      \
    "s_lshl_b32 s47, s47, 6\n"                                                     \
    RX_FULL(R0, R1, COLS, XL, XN, SB, SN, L "A")                                   \
    "s_add_u32 s47, s41, 2\n"                                                      \
    "s_lshl_b32 s47, s47, 6\n"                                                     \
    RX_FULL(R0, R1, COLS, XL, XN, SN, SB, L "B")                                   \
    "s_add_u32 s41, s41, 2\n"                                                      \
    "s_branch " L "lp_%=\n"                                                        \
    L "tl_%=:\n"                                                                   \
    "s_add_u32 s46, s41, 1\n"                                                      \
    "s_cmp_ge_u32 s46, s42\n"                                                      \
    "s_cbranch_scc1 " L "on_%=\n"                                                  \
    "s_lshl_b32 s47, s46, 6\n"                                                     \
    RX_FULL(R0, R1, COLS, XL, XN, SB, SN, L "C")                                   \
    "s_add_u32 s47, s41, 2\n"                                                      \
    "s_lshl_b32 s47, s47, 6\n"                                                     \
    "s_cmp_eq_u32 s44, 0\n"                                                        \
    "s_cbranch_scc0 " L "o1_%=\n"                                                  \
    RX_LAST2(R0, R1, COLS, XL, XN, SN, SB, L "D")                                  \
    "s_branch " L "en_%=\n"                                                        \
    L "o1_%=:\n"                                                                   \
    RX_LAST1(R0, R1, COLS, XL, XN, SN, SB, L "E")                                  \
    "s_branch " L "en_%=\n"                                                        \
    L "on_%=:\n"                                                                   \
    "s_lshl_b32 s47, s46, 6\n"                                                     \
    "s_cmp_eq_u32 s44, 0\n"                                                        \
    "s_cbranch_scc0 " L "o2_%=\n"                                                  \
    RX_LAST2(R0, R1, COLS, XL, XN, SB, SN, L "F")                                  \
    "s_branch " L "en_%=\n"                                                        \
    L "o2_%=:\n"                                                                   \
    RX_LAST1(R0, R1, COLS, XL, XN, SB, SN, L "G")                                  \
    L "en_%=:\n"                                                                   \
    "s_waitcnt lgkmcnt(0)\n"

// Wait until chunk s40 has landed in the ring (its quarter's fill count
// reaches s40 / 4 + 1); a bounded wait that sets the plan's flag on giving up.
#define RX_ENTER                                                   \
    "s_lshr_b32 s46, s40, 2\n"                                     \
    "s_add_u32 s46, s46, 1\n"                                      \
    "s_and_b32 s47, s40, 3\n"                                      \
    "s_lshl_b32 s47, s47, 2\n"                                     \
    "s_add_u32 s47, s47, %[ctl]\n"                                 \
    "s_add_u32 s47, s47, 16\n"                                     \
    "v_mov_b32 v[%[t]], s47\n"                                     \
    "s_mov_b32 s52, 0\n"                                           \
    "ENsp_%=:\n"                                                   \
    "ds_read_b32 v[%[t]+1], v[%[t]]\n"                             \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "v_readfirstlane_b32 s48, v[%[t]+1]\n"                         \
    "s_cmp_ge_i32 s48, s46\n"                                      \
    "s_cbranch_scc1 ENok_%=\n"                                     \
    "s_add_u32 s52, s52, 1\n"                                      \
    "s_cmp_gt_u32 s52, %[spin]\n"                                  \
    "s_cbranch_scc1 ENbad_%=\n"                                    \
    "s_sleep 1\n"                                                  \
    "s_branch ENsp_%=\n"                                           \
    "ENbad_%=:\n"                                                  \
    "s_mov_b64 s[50:51], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "v_mov_b32 v[%[t]], 0\n"                                       \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    "global_atomic_or v[%[t]], v[%[t]+1], %[flag]\n"               \
    "s_mov_b64 exec, s[50:51]\n"                                   \
    "ENok_%=:\n"

// Count the landing of every ring quarter copied earlier (after the copies'
// loads are complete), one lane adding to its fill counter.
#define RX_PUB1(j, L)                                                    \
    "s_bitcmp1_b32 s45, " #j "\n"                                        \
    "s_cbranch_scc0 " L #j "_%=\n"                                       \
    "s_add_u32 s47, %[ctl], 16+4*" #j "\n"                               \
    "v_mov_b32 v[%[t]], s47\n"                                           \
    "ds_add_u32 v[%[t]], v[%[t]+1]\n"                                    \
    L #j "_%=:\n"
#define RX_PUBLISH(L)                                              \
    "s_cmp_eq_u32 s45, 0\n"                                        \
    "s_cbranch_scc1 " L "_%=\n"                                    \
    "s_waitcnt vmcnt(0)\n"                                         \
    "s_mov_b64 s[50:51], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    RX_PUB1(0, L) RX_PUB1(1, L) RX_PUB1(2, L) RX_PUB1(3, L)        \
    "s_mov_b64 exec, s[50:51]\n"                                   \
    "s_mov_b32 s45, 0\n"                                           \
    L "_%=:\n"

// Chunk s40 + 4 into the ring quarter of chunk s40: channel c of column slot k
// goes to ring row c % 64 at byte 256 k, one dword per lane straight from X.
#define RX_CP(k, OFF)                                              \
    "ds_read_b32 v[%[t]], v[%[t]+1] offset:" #OFF "\n"             \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b32 s48, s46\n"                                         \
    "CP" #k "_%=:\n"                                               \
    "s_and_b32 s49, s48, 63\n"                                     \
    "s_lshl_b32 s49, s49, %[sh]\n"                                 \
    "s_add_u32 s49, s49, %[base]\n"                                \
    "s_add_u32 m0, s49, " #OFF "\n"                                \
    "s_mul_i32 s53, s48, %[hw4]\n"                                 \
    "s_nop 0\n"                                                    \
    "buffer_load_dword v[%[t]], %[rs], s53 offen lds\n"            \
    "s_add_u32 s48, s48, 1\n"                                      \
    "s_cmp_lt_u32 s48, s47\n"                                      \
    "s_cbranch_scc1 CP" #k "_%=\n"
#define RX_COPY_HEAD                                               \
    "s_add_u32 s46, s40, 4\n"                                      \
    "s_lshl_b32 s46, s46, 4\n"                                     \
    "s_add_u32 s47, s46, 16\n"                                     \
    "s_min_u32 s47, s47, %[cin]\n"                                 \
    "v_subrev_u32 v[%[t]+1], %[base], %[vl]\n"                     \
    "v_add_u32 v[%[t]+1], %[xo], v[%[t]+1]\n"
#define RX_CP1 RX_CP(0, 0)
#define RX_CP2 RX_CP1 RX_CP(1, 256)
#define RX_CP3 RX_CP2 RX_CP(2, 512)
#define RX_CP4 RX_CP3 RX_CP(3, 768)
#define RX_CP5 RX_CP4 RX_CP(4, 1024)
#define RX_CP6 RX_CP5 RX_CP(5, 1280)

// Release chunk s40 (publish earlier copies first); the last wavefront to
// release it copies chunk s40 + 4 into its quarter.
#define RX_LEAVE(CP)                                               \
    RX_PUBLISH("LP")                                               \
    "s_and_b32 s47, s40, 3\n"                                      \
    "s_lshl_b32 s47, s47, 2\n"                                     \
    "s_add_u32 s47, s47, %[ctl]\n"                                 \
    "v_mov_b32 v[%[t]], s47\n"                                     \
    "v_mov_b32 v[%[t]+1], 1\n"                                     \
    "s_mov_b64 s[50:51], exec\n"                                   \
    "s_mov_b64 exec, 1\n"                                          \
    "ds_add_rtn_u32 v[%[t]+1], v[%[t]], v[%[t]+1]\n"               \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b64 exec, s[50:51]\n"                                   \
    "v_readfirstlane_b32 s46, v[%[t]+1]\n"                         \
    "s_add_u32 s46, s46, 1\n"                                      \
    "s_lshr_b32 s47, s40, 2\n"                                     \
    "s_add_u32 s47, s47, 1\n"                                      \
    "s_mul_i32 s47, s47, %[nw]\n"                                  \
    "s_cmp_lg_u32 s46, s47\n"                                      \
    "s_cbranch_scc1 LN_%=\n"                                       \
    "s_add_u32 s47, s40, 4\n"                                      \
    "s_cmp_ge_u32 s47, %[nch]\n"                                   \
    "s_cbranch_scc1 LN_%=\n"                                       \
    RX_COPY_HEAD CP                                                \
    "s_and_b32 s46, s40, 3\n"                                      \
    "s_lshl_b32 s46, 1, s46\n"                                     \
    "s_or_b32 s45, s45, s46\n"                                     \
    "LN_%=:\n"

// Bias, activation and store of the slot's 16 rows: the lane's C column
// offsets from the LDS table into x0, a row's C accumulators into x1.
#define RX_EPK(k, OFF)                                                   \
    "v_add_f32 v[%[x1]+" #k "], s48, v[%[x1]+" #k "]\n"                  \
    "v_max_f32 v[%[x1]+" #k "], v[%[x1]+" #k "], %[lo]\n"               \
    "v_min_f32 v[%[x1]+" #k "], v[%[x1]+" #k "], %[hi]\n"               \
    "buffer_store_dword v[%[x1]+" #k "], v[%[x0]+" #k "], %[ry], s49 offen\n"
#define RX_EPL(k, OFF) "ds_read_b32 v[%[x0]+" #k "], v[%[t]+1] offset:" #OFF "\n"
#define RX_EPR(k, OFF) "v_mov_b32 v[%[x1]+" #k "], v[%[a]+16*" #k "]\n"
#define RX_EACH1(M) M(0, 0)
#define RX_EACH2(M) RX_EACH1(M) M(1, 256)
#define RX_EACH3(M) RX_EACH2(M) M(2, 512)
#define RX_EACH4(M) RX_EACH3(M) M(3, 768)
#define RX_EACH5(M) RX_EACH4(M) M(4, 1024)
#define RX_EACH6(M) RX_EACH5(M) M(5, 1280)
#define RX_EPILOGUE(EACH)                                          \
    "v_subrev_u32 v[%[t]+1], %[base], %[vl]\n"                     \
    "v_add_u32 v[%[t]+1], %[yo], v[%[t]+1]\n"                      \
    EACH(RX_EPL)                                                   \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_mov_b32 s40, 0\n"                                           \
    "EP_%=:\n"                                                     \
    "s_lshl_b32 s46, s40, 2\n"                                     \
    "s_load_dword s47, %[rows], s46\n"                             \
    "s_load_dword s48, %[bias], s46\n"                             \
    "s_waitcnt lgkmcnt(0)\n"                                       \
    "s_cmp_lt_i32 s47, 0\n"                                        \
    "s_cbranch_scc1 EPn_%=\n"                                      \
    "s_mul_i32 s49, s47, %[hw4]\n"                                 \
    "s_set_gpr_idx_on s40, gpr_idx(SRC0)\n"                        \
    EACH(RX_EPR)                                                   \
    "s_set_gpr_idx_off\n"                                          \
    EACH(RX_EPK)                                                   \
    "EPn_%=:\n"                                                    \
    "s_add_u32 s40, s40, 1\n"                                      \
    "s_cmp_lt_u32 s40, 16\n"                                       \
    "s_cbranch_scc1 EP_%=\n"

// The whole statement.
#define RX_STREAM(R0, R1, COLS, XL, XN, ZC, CP, EACH, CLOBV)                                        \
    asm volatile(ZC                                                                                 \
                 "s_mov_b32 s40, 0\n"                                                               \
                 "s_mov_b32 s45, 0\n"                                                               \
                 "s_mov_b32 s43, 1\n"                                                               \
                 "CH_%=:\n"                                                                         \
                 "s_cmp_ge_u32 s40, %[nch]\n"                                                       \
                 "s_cbranch_scc1 DN_%=\n"                                                           \
                 RX_ENTER                                                                           \
                 "s_lshl_b32 s46, s40, 2\n"                                                         \
                 "s_load_dwordx2 s[48:49], %[ch], s46\n"                                            \
                 "s_waitcnt lgkmcnt(0)\n"                                                           \
                 "s_lshr_b32 s41, s48, 1\n"                                                         \
                 "s_lshr_b32 s42, s49, 1\n"                                                         \
                 "s_and_b32 s44, s48, 1\n"                                                          \
                 "s_cmp_ge_u32 s41, s42\n"                                                          \
                 "s_cbranch_scc1 LV_%=\n"                                                           \
                 "s_bitcmp1_b32 s41, 0\n"                                                           \
                 "s_cbranch_scc1 RQ_%=\n"                                                           \
                 RX_RUN(R0, R1, COLS, XL, XN, b0, b1, "P")                                          \
                 "s_branch LV_%=\n"                                                                 \
                 "RQ_%=:\n"                                                                         \
                 RX_RUN(R0, R1, COLS, XL, XN, b1, b0, "Q")                                          \
                 "LV_%=:\n"                                                                         \
                 RX_LEAVE(CP)                                                                       \
                 "s_add_u32 s40, s40, 1\n"                                                          \
                 "s_branch CH_%=\n"                                                                 \
                 "DN_%=:\n"                                                                         \
                 RX_PUBLISH("FP")                                                                   \
                 RX_EPILOGUE(EACH)                                                                  \
                 :                                                                                  \
                 : [a] "i"(L::A), [x0] "i"(L::X0), [x1] "i"(L::X1), [va0] "i"(L::VA0),              \
                   [va1] "i"(L::VA1), [t] "i"(L::T), [sh] "i"(L::SHIFT), [b0] "i"(64), [b1] "i"(80),  \
                   [spin] "i"(kSpinMax), [ch] "s"(ch), [nch] "s"(nch), [ptr] "s"(ptr), [ctl] "s"(ctl), \
                   [nw] "s"(nw), [rs] "s"(rs), [xo] "s"(xo), [yo] "s"(yo), [cin] "s"(cin),           \
                   [hw4] "s"(hw4), [base] "s"(base), [flag] "s"(flag), [rows] "s"(rows),              \
                   [bias] "s"(bias), [ry] "s"(ry), [vl] "v"(vl), [lo] "v"(lo), [hi] "v"(hi)           \
                 : "memory", "m0", "scc", "vcc", CLOBV, IX_CLOBS)

#define RX_ZV(k) \
    "v_mov_b32 v[%[a]+16*" #k "+0], 0\n v_mov_b32 v[%[a]+16*" #k "+1], 0\n v_mov_b32 v[%[a]+16*" #k "+2], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+3], 0\n v_mov_b32 v[%[a]+16*" #k "+4], 0\n v_mov_b32 v[%[a]+16*" #k "+5], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+6], 0\n v_mov_b32 v[%[a]+16*" #k "+7], 0\n v_mov_b32 v[%[a]+16*" #k "+8], 0\n"      \
    "v_mov_b32 v[%[a]+16*" #k "+9], 0\n v_mov_b32 v[%[a]+16*" #k "+10], 0\n v_mov_b32 v[%[a]+16*" #k "+11], 0\n"    \
    "v_mov_b32 v[%[a]+16*" #k "+12], 0\n v_mov_b32 v[%[a]+16*" #k "+13], 0\n v_mov_b32 v[%[a]+16*" #k "+14], 0\n"   \
    "v_mov_b32 v[%[a]+16*" #k "+15], 0\n"
#define RX_Z1 RX_ZV(0)
#define RX_Z2 RX_Z1 RX_ZV(1)
#define RX_Z3 RX_Z2 RX_ZV(2)
#define RX_Z4 RX_Z3 RX_ZV(3)
#define RX_Z5 RX_Z4 RX_ZV(4)
#define RX_Z6 RX_Z5 RX_ZV(5)

template <int K, int C>
__device__ __forceinline__ void stream_asm(const int32_t *ch, int32_t nch, const uint32_t *ptr, uint32_t ctl,
                                           int32_t nw, i4 rs, uint32_t xo, uint32_t yo, int32_t cin, int32_t hw4,
                                           uint32_t base, int32_t *flag, const int32_t *rows, const float *bias,
                                           i4 ry, int32_t vl, float lo, float hi) {
    using L = Lay<C>;
#define RX_BY_C(R0, R1)                                                                  \
    if constexpr (C == 1) {                                                              \
        RX_STREAM(R0, R1, RX_C1, RX_XL1, 1, RX_Z1, RX_CP1, RX_EACH1, IX_CLOBV1);         \
    } else if constexpr (C == 2) {                                                       \
        RX_STREAM(R0, R1, RX_C2, RX_XL2, 1, RX_Z2, RX_CP2, RX_EACH2, IX_CLOBV2);         \
    } else if constexpr (C == 3) {                                                       \
        RX_STREAM(R0, R1, RX_C3, RX_XL3, 2, RX_Z3, RX_CP3, RX_EACH3, IX_CLOBV3);         \
    } else if constexpr (C == 4) {                                                       \
        RX_STREAM(R0, R1, RX_C4, RX_XL4, 2, RX_Z4, RX_CP4, RX_EACH4, IX_CLOBV4);         \
    } else if constexpr (C == 5) {                                                       \
        RX_STREAM(R0, R1, RX_C5, RX_XL5, 3, RX_Z5, RX_CP5, RX_EACH5, IX_CLOBV5);         \
    } else {                                                                             \
        RX_STREAM(R0, R1, RX_C6, RX_XL6, 3, RX_Z6, RX_CP6, RX_EACH6, IX_CLOBV6);         \
    }
    if constexpr (K == 1) {
        RX_BY_C(RX_R0_K1, RX_R1_K1)
    } else if constexpr (K == 2) {
        RX_BY_C(RX_R0_K2, RX_R1_K2)
    } else {
        RX_BY_C(RX_R0_K4, RX_R1_K4)
    }
#undef RX_BY_C
}

// ---------------------------------------------------------------------------
// Per-task control
// ---------------------------------------------------------------------------

// The column offsets of lane `lane`'s k-th column of a tile (column j):
// x / y byte offsets relative to the tile's first image, kOOR past the end.
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

// Set-up of a task: lane column offsets and counters into LDS, the first
// ring's worth of channels copied by every wavefront.
template <int C>
__device__ __forceinline__ void task_setup(int32_t task, unsigned char *lds, uint32_t lds_base, int wave, int nwaves,
                                           int lane) {
    using L = Lay<C>;
    const auto &a = kargs();
    const TaskPos t = task_pos<C>(a, task, wave);
    const int64_t xbase = static_cast<int64_t>(t.n0) * a.cin * a.hw;
    const i4 rs = rsrc_words(a.x + xbase, a.x_bytes - xbase * 4);
    int32_t *xo_lds = reinterpret_cast<int32_t *>(lds + a.xo_off);
    int32_t *yo_lds = xo_lds + 64 * C;
    int32_t *freec = reinterpret_cast<int32_t *>(lds + a.ctl_off);
    const uint32_t base = lds_base + static_cast<uint32_t>(a.ring_off);
    __syncthreads();  // the previous user of LDS is done
    if (wave == 0) {
#pragma unroll 1
        for (int k = 0; k < C; ++k) {
            int32_t xo, yo;
            col_offsets(a, t.col0 + 64 * k + lane, t.n0, xo, yo);
            xo_lds[k * 64 + lane] = xo;
            yo_lds[k * 64 + lane] = yo;
        }
        if (lane < 4) {
            freec[lane] = 0;
            freec[4 + lane] = lane < a.nch ? 1 : 0;
        }
    }
    __syncthreads();
    const int32_t rows0 = imin(kRing, a.cin);
#pragma unroll 1
    for (int k = 0; k < C; ++k) {
        const int32_t xo = xo_lds[k * 64 + lane];
#pragma unroll 1
        for (int32_t c = wave; c < rows0; c += nwaves)
            dma_dword(base + static_cast<uint32_t>(c << L::SHIFT) + 256u * k, xo, rs, c * a.hw * 4);
    }
    wait_vm0();
    __syncthreads();
}

// The wavefront's slot over the task's tile (the stream statement).
template <int K, int C>
__device__ __forceinline__ void task_stream(int32_t task, uint32_t lds_base, int wave, int lane) {
    const auto &a = kargs();
    const TaskPos t = task_pos<C>(a, task, wave);
    const int64_t xbase = static_cast<int64_t>(t.n0) * a.cin * a.hw;
    const int64_t ybase = static_cast<int64_t>(t.n0) * a.cout * a.hw;
    const i4 rs = rsrc_words(a.x + xbase, a.x_bytes - xbase * 4);
    const i4 ry = rsrc_words(a.y + ybase, a.y_bytes - ybase * 4);
    const uint32_t base = lds_base + static_cast<uint32_t>(a.ring_off);
    const int32_t nch = a.nch;
    const int32_t *ch = uniform_ptr(a.slot_chunk + static_cast<int64_t>(t.slot) * (nch + 1));
    const uint32_t *ptr =
        uniform_ptr(a.rec + static_cast<int64_t>(cst(a.slot_batch)[t.slot]) * (kRecWords * kBatchRecs));
    const int32_t *rows = uniform_ptr(a.slot_rows + static_cast<int64_t>(t.slot) * kSlotRows);
    const float *bias = uniform_ptr(a.slot_bias + static_cast<int64_t>(t.slot) * kSlotRows);
    const float lo = a.act == 0 ? -__builtin_huge_valf() : 0.0f;
    const float hi = a.act == 2 ? 6.0f : __builtin_huge_valf();
    stream_asm<K, C>(ch, __builtin_amdgcn_readfirstlane(nch), ptr,
                     __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(a.ctl_off)),
                     __builtin_amdgcn_readfirstlane(t.nw), rs,
                     __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(a.xo_off)),
                     __builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(a.xo_off) + 256u * C),
                     __builtin_amdgcn_readfirstlane(a.cin), __builtin_amdgcn_readfirstlane(a.hw * 4),
                     __builtin_amdgcn_readfirstlane(base), uniform_ptr(a.flag), rows, bias, ry,
                     static_cast<int32_t>(base) + 4 * lane, lo, hi);
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
    int32_t pc = p0;
    while (pc < p1) {
        const int32_t cg = pc / a.pairs;
        const int32_t pe = std::min(p1, (cg + 1) * a.pairs);
        const int32_t j = a.lcol0 + 64 * cg + lane;
        const int32_t col0 = a.lcol0 + 64 * cg;
        const int32_t n0 = col0 / a.hw;
        const int64_t xbase = static_cast<int64_t>(n0) * a.cin * a.hw;
        const int64_t ybase = static_cast<int64_t>(n0) * a.cout * a.hw;
        int32_t xo, yo;
        col_offsets(a, j, n0, xo, yo);
        __syncthreads();
        const i4 rs = rsrc_words(x + xbase, a.x_bytes - xbase * 4);
        for (int32_t c = wave; c < a.cin; c += nwaves)
            dma_dword(__builtin_amdgcn_readfirstlane(lds_base + static_cast<uint32_t>(c * 256)), xo, rs,
                      c * a.hw * 4);
        wait_vm0();
        __syncthreads();
        const Rsrc ry = make_rsrc(y + ybase, a.y_bytes - ybase * 4);
        const float *strip = reinterpret_cast<const float *>(lds);
        for (int32_t t = pc + wave; t < pe; t += nwaves) {
            const int32_t pr = t - cg * a.pairs;
            const auto *pp = cst(a.pair_ptr);
            const auto *pe_ = cst(a.pair_ent);
            const int32_t e0 = pp[pr], e1 = pp[pr + 1];
            float acc0 = 0.0f, acc1 = 0.0f;
            for (int32_t e = e0; e < e1; ++e) {
                const uint32_t w0 = pe_[4 * e];
                const float wa = __uint_as_float(pe_[4 * e + 1]);
                const float wb = __uint_as_float(pe_[4 * e + 2]);
                const float xv = strip[(w0 & 0xffffffu) * 64 + lane];
                if (w0 & (1u << 24))
                    acc0 = __builtin_fmaf(wa, xv, acc0);
                if (w0 & (2u << 24))
                    acc1 = __builtin_fmaf(wb, xv, acc1);
            }
            const int32_t r0 = 2 * pr;
            const auto *rb = cst(a.row_bias);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(fminf(fmaxf(acc0 + rb[r0], lo), hi)), ry,
                                                  yo, r0 * a.hw * 4, 0);
            if (r0 + 1 < a.cout)
                __builtin_amdgcn_raw_buffer_store_b32(
                    __float_as_uint(fminf(fmaxf(acc1 + rb[r0 + 1], lo), hi)), ry, yo, (r0 + 1) * a.hw * 4,
                    0);
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
        task_setup<C>(task, lds, lds_base, wave, nwaves, lane);
        if (wave < task_pos<C>(kargs(), task, wave).nw)
            task_stream<K, C>(task, lds_base, wave, lane);
    }
    if (kargs().lpieces > 0)
        run_pairs(lds, lds_base, wave, nwaves, lane);
}

// One kernel per column count C.
#define IX_KERNEL(CC)                                                     \
    template <int K>                                                      \
    __global__ void __launch_bounds__(1024) spmm_indexed_c##CC(IArgs) {  \
        indexed_body<K, CC>();                                            \
    }
IX_KERNEL(1)
IX_KERNEL(2)
IX_KERNEL(3)
IX_KERNEL(4)
IX_KERNEL(5)
IX_KERNEL(6)
static_assert(kSB == 64, "record buffers are pinned at s64 .. s95");

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

int32_t ring_row_bytes(int c) { return c <= 1 ? 256 : c <= 2 ? 512 : c <= 4 ? 1024 : 2048; }

}  // namespace

IndexedLaunch plan_indexed_launch(const DevicePlan &p, int64_t m) {
    IndexedLaunch best;
    const int64_t W = p.rwaves;
    const int64_t G = p.rgroups;
    const int64_t wg_per_cu = std::max<int64_t>(1, kMaxWaves / W);
    const int64_t grid = static_cast<int64_t>(p.num_cus) * wg_per_cu;
    const int64_t pairs = (p.cout + 1) / 2;
    const bool pairs_fit = static_cast<int64_t>(p.cin) * 256 <= kMaxLdsBytes - 4096;
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
        // one round of whole tiles, the rest by row pairs
        if (pairs_fit && grid % G == 0) {
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
    const int32_t rowb = ring_row_bytes(best.c);
    best.ctl_off = kRing * rowb;
    best.xo_off = best.ctl_off + 64;
    const int32_t main_lds = best.xo_off + 2 * 64 * 4 * best.c;
    const int32_t pair_lds = best.lpieces ? p.cin * 256 : 0;
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
    a.ring_off = 0;
    a.ctl_off = L.ctl_off;
    a.xo_off = L.xo_off;
    a.rec = p.rrec;
    a.slot_batch = p.rslot_batch;
    a.slot_chunk = p.rslot_chunk;
    a.slot_rows = p.rslot_rows;
    a.slot_bias = p.rslot_bias;
    a.pair_ptr = p.rpair_ptr;
    a.pair_ent = p.rpair_ent;
    a.row_bias = p.rrow_bias;
    a.flag = p.flag;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(L.grid)), dim3(p.rwaves * 64), L.lds_bytes, stream, a);
    return hipGetLastError();
}

}  // namespace spconv
