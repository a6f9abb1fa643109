// Internal interface between the C ABI and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "planner.hpp"

namespace spconv {

// Device-resident copy of a PackedPlan (see planner.hpp for the layout) plus
// the launch facts fixed at plan creation.
struct DevicePlan {
    int32_t kernel = KERNEL_STRIP;
    int32_t group_lanes = 4;
    int32_t tile_cols = 64;
    int32_t waves = 1;
    int32_t lds_bytes = 0;
    int32_t k = 1;
    int32_t storage = 0;
    int32_t act = 0;
    int32_t cin = 0, cout = 0;
    int32_t strip_rows = 0;     // channels of the LDS strip (cin rounded up to 4); 0 for the direct kernel
    int32_t pipe_sets = 1;      // bundles a wavefront interleaves in the pipelined kernel
    int32_t regions = 1;        // strip parts refilled independently
    int32_t region_rows = 0;    // channels per part
    int32_t busy_waves = 0;     // wavefronts with at least one bundle
    int32_t idx_bytes = 0;      // size of the channel stream (bounds of its buffer resource)
    int32_t val_bytes = 0;      // size of the weight stream
    int32_t num_cus = 0;        // compute units of the plan's device
    int32_t blocks_per_cu = 0;  // resident workgroups per CU
    int32_t nbundles = 0;
    int32_t max_parts = 1;      // most workgroups that may share one tile
    int32_t dw_stride = 0;      // fused depthwise 3x3 stage: 0 none, else its stride
    int32_t dw_act = 0;
    int32_t stage_off = 0;      // LDS staging area of the depthwise stage's input windows
    int32_t stage_bytes = 0;
    const int32_t *idx = nullptr;
    const float *val = nullptr;
    const int32_t *hdr = nullptr;       // (first step, steps) per bundle
    const int32_t *table = nullptr;     // rows, then biases (fp32 bits), per (bundle, group)
    const int32_t *rank = nullptr;      // longest-first rank of each bundle
    const int32_t *wave_ptr = nullptr;  // bundles of each wave
    const int32_t *pidx = nullptr;      // interleaved streams and their per-wave tables
    const float *pval = nullptr;
    const uint32_t *psel = nullptr;
    const int32_t *sel_ptr = nullptr;
    const int32_t *wave_ev = nullptr;
    const float *dw = nullptr;          // depthwise taps and biases, kDwParams per strip channel
    // register-indexed kernel (planner.hpp)
    int32_t use_indexed = 0;
    int32_t rslots = 0, rgroups = 0, rwaves = 0, rnch = 0, rlane_cols = 0;
    const uint32_t *rrec = nullptr;
    const int32_t *rslot_batch = nullptr;
    const int32_t *rslot_chunk = nullptr;
    const int32_t *rslot_rows = nullptr;
    const float *rslot_bias = nullptr;
    const int32_t *rpair_ptr = nullptr;
    const uint32_t *rpair_ent = nullptr;
    int64_t rpair_ent_words = 0;
    const float *rrow_bias = nullptr;   // bias of every output channel
    int32_t *flag = nullptr;            // device word: bit 0 set when a bounded wait of a kernel gave up
    int32_t spin_limit = 1 << 22;       // bound of those waits, in sleeps
    int64_t indexed_min_cols = 0;       // automatic choice: runs of at least this many columns take the
                                        // register-indexed kernel (0: never)
    // outer-product kernel (planner.hpp)
    int32_t use_outer = 0, omode = 0, otw = 32, oocts = 0, owaves = 0, ozrow = 0;
    const uint32_t *orec = nullptr;
    const uint32_t *ooff = nullptr;
    int32_t ooff_bytes = 0;             // the offset table including its read-ahead quads
    const int32_t *ooct = nullptr;
    const int32_t *owave_ptr = nullptr;
    const int32_t *owave_oct = nullptr;
    int64_t outer_min_cols = 0;         // automatic choice: runs of at least this many columns take it (0: never)
    // a pass over one channel range of a wider input (spconv_api.cpp): X's
    // channels per image (0: cin), and whether the pass adds to the partial
    // sums already in Y (every pass but the first)
    int32_t xc = 0;
    int32_t accum = 0;
    int32_t splits = 0;  // the plan has split rows (row-table entries kRowPiece)
};

// How one launch of the register-indexed kernel covers m columns: `tiles`
// whole tiles of 64 c columns (times the plan's slot groups), then columns
// [lcol0, m) as `lpieces` (64-column group, row pair) pieces, `lper` per
// workgroup; `grid` workgroups; LDS offsets of the counters, the lane column
// tables and the copy patterns, and the LDS bytes per workgroup.
struct IndexedLaunch {
    int32_t c = 1;
    int64_t tiles = 0;
    int32_t lcol0 = 0, lpieces = 0, lper = 0;
    int32_t grid = 1;
    int32_t ctl_off = 0, xo_off = 0, pat_off = 0, lds_bytes = 0;
    int32_t ent_off = 0, epw = 0;  // row pairs: LDS entry areas and entries per wavefront area
};

IndexedLaunch plan_indexed_launch(const DevicePlan &p, int64_t m);
// Once per plan: allow the indexed kernels their LDS.
hipError_t prepare_indexed(const DevicePlan &p);
// One launch of the register-indexed kernel over all m = N * hw columns.
hipError_t launch_indexed(const DevicePlan &p, const float *x, float *y, int32_t m, int32_t hw, int64_t x_bytes,
                          int64_t y_bytes, hipStream_t stream);

// Once per plan: allow the outer-product kernel its LDS.
hipError_t prepare_outer(const DevicePlan &p);
// LDS bytes of one outer-product workgroup.
int32_t outer_lds_bytes(const DevicePlan &p);
// One launch of the outer-product kernel over all m = N * hw columns (fp32 or
// fp16 x and y as the plan's storage).  `vec` != 0 promises hw a multiple of
// 4 and 16-byte aligned x and y (whole 4-column vectors per image).
hipError_t launch_outer(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                        int64_t x_bytes, hipStream_t stream);

// Once per plan, on its device: raise the kernel's dynamic-LDS limit when
// needed and record num_cus and blocks_per_cu.
hipError_t prepare_launch(DevicePlan &p);

// Queue one launch computing all m = N * hw output columns.  `vec` != 0
// promises that hw is a multiple of the columns in one 16-byte vector and
// that x and y are 16-byte aligned, enabling 16-byte loads and stores.
// `x_bytes` and `y_bytes` are the sizes of x and y.  With a depthwise stage,
// x is N x cin x in_h x in_w and hw = out_h * out_w (out_w given); otherwise
// in_h, in_w and out_w are ignored.
hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                       int64_t x_bytes, int64_t y_bytes, int32_t in_h, int32_t in_w, int32_t out_w,
                       hipStream_t stream);

}  // namespace spconv
