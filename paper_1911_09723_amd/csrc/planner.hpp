// Host-side format planner for the sparse 1x1 convolution.
//
// Pure C++17: no HIP dependency, so everything here runs and is tested on a
// machine without a GPU.  Input is the block-CSR weight format of the paper's
// library (Sec. 3.3: dense masked weights are converted to a block compressed
// sparse row form for inference; Sec. 3.2: a block is k consecutive output
// channels sharing one input channel).  Output is the packed image the GPU
// kernels stream.
//
// Packed layout (all int32 / fp32, little-endian, every array 16-byte aligned):
//
//   A *bundle* is `groups` (= 64 / lanes_per_row) block rows that one
//   wavefront processes at the same time, one row per lane group.  Bundles
//   are made of consecutive rows in processing order (descending nonzero
//   count unless reordering is off), so the rows of a bundle have similar
//   lengths.  Its length L is the longest of its rows rounded up to a multiple
//   of 4 (at least 4); shorter rows are padded with (channel 0, weight 0)
//   slots, which add an exact zero.  A *step* is 4 slots of every row.
//
//   hdr[4*b + 0]  first slot of bundle b (a multiple of 4)
//   hdr[4*b + 1]  L / 4: steps of bundle b
//   rows[groups*b + g]         block row handled by lane group g, or -1 (padding group)
//   bundle_bias[(groups*b + g)*k + i]  bias of row rows[..]*k + i (0 for padding)
//
//   Slot numbering inside bundle b (base S = hdr[4*b]):
//     slot S + (t4 * groups + g) * 4 + u   for step t4 < L/4, u < 4
//   so one 16-byte load fetches the next 4 channel indices of a row.
//   idx[slot]        input channel c; the first slot of a bundle's last step
//                    also carries kLastStepFlag
//   val[slot*k + i]  weight of block row element i (fp16-rounded for fp16 storage)
//
//   Bundles are assigned to the `waves` wavefronts of a workgroup by longest
//   processing time first; wave_ptr[w] .. wave_ptr[w+1] are wave w's bundles,
//   which are stored contiguously in that order, so each wavefront reads one
//   continuous stream of steps.
//
// The per-row summation order is ascending input channel (the CSR order), with
// padding zeros in between; it does not depend on the bundle grouping, so the
// result is bitwise independent of reordering and wave assignment.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace spconv {

enum Status { OK = 0, E_ARG = 1, E_FORMAT = 2, E_SHAPE = 3, E_UNSUPPORTED = 4, E_NOMEM = 5, E_HIP = 6 };

enum Kernel { KERNEL_STRIP = 0, KERNEL_DIRECT = 1 };

// Largest LDS footprint of one workgroup on gfx950 (160 KiB per CU).
constexpr int64_t kMaxLdsBytes = 160 * 1024;
// Every X read of a lane is one 16-byte vector: 4 fp32 or 8 fp16 columns.
constexpr int kLaneBytes = 16;
// Wavefronts per workgroup (1024 threads).
constexpr int32_t kMaxWaves = 16;
// Bit set in the channel index of the first slot of a bundle's last step.  It
// lies above any valid channel and above the bits that survive the kernels'
// scaling of the channel to a byte offset, so the kernels read it without
// masking it out.
constexpr int32_t kLastStepFlag = 1 << 30;
// Main-loop steps the kernels may fetch past the end of a bundle.
constexpr int64_t kLookaheadSteps = 4;
// Strip bytes one loader wavefront holds in registers: 64 lanes x 16 vectors.
constexpr int64_t kLoaderBytesPerWave = 64 * 16 * 16;

struct Input {
    int32_t cout = 0, cin = 0, block_rows = 1;
    const int32_t *row_ptr = nullptr;
    const int32_t *col_idx = nullptr;
    const float *values = nullptr;
    const float *bias = nullptr;
    int32_t act = 0;      // 0 none, 1 relu, 2 relu6
    int32_t storage = 0;  // 0 fp32, 1 fp16
};

struct Options {
    int32_t reorder = 1;
    int32_t host_only = 0;
    int32_t lanes_per_row = 0;
    int32_t waves = 0;
    int32_t vecs_per_lane = 0;
    int32_t prefetch = 1;
};

struct PackedPlan {
    // shape and epilogue
    int32_t cout = 0, cin = 0, k = 1, act = 0, storage = 0;
    // launch geometry
    int32_t kernel = KERNEL_STRIP;
    int32_t lanes_per_row = 16;  // G
    int32_t vecs_per_lane = 1;   // 16-byte X vectors each lane reads per nonzero
    int32_t groups = 4;          // 64 / G
    int32_t cols_per_lane = 4;   // vecs_per_lane * 16 bytes / element size
    int32_t tile_cols = 64;      // G * cols_per_lane
    int32_t waves = 1;           // compute wavefronts (each owns a list of bundles)
    int32_t loader_waves = 0;    // wavefronts that prefetch the next strip (strip kernel)
    int32_t lds_bytes = 0;       // strip + bundle table (strip kernel)
    int32_t strip_bytes = 0;
    // packed streams
    std::vector<int32_t> idx;
    std::vector<float> val;
    std::vector<int32_t> hdr;
    std::vector<int32_t> rows;
    std::vector<int32_t> wave_ptr;
    std::vector<float> bias;
    std::vector<float> bundle_bias;  // bias of the row of each (bundle, group, block element)
    int32_t meta_bytes = 0;          // rows + bundle_bias, copied into LDS by the strip kernel
    std::vector<int32_t> perm;     // block rows in processing order
    std::vector<int32_t> row_nnz;  // stored blocks per block row (host only; for unpacking)
    // statistics
    int64_t nnzb = 0;
    int64_t slots = 0;
    int64_t max_wave_cost = 0;
    int64_t sum_wave_cost = 0;
};

// Round an fp32 value to the nearest IEEE binary16 value, ties to even, and
// return the binary16 bit pattern (overflow gives infinity, NaN stays NaN).
uint16_t float_to_half_rne(float v);
// Exact binary16 -> fp32 conversion.
float half_to_float(uint16_t h);

// Check the block-CSR arrays; on failure return the status and set `err`.
Status validate(const Input &in, std::string &err);

// Validate, order, bundle, balance and pack.  Returns OK or an error with `err` set.
Status build_plan(const Input &in, const Options &opt, PackedPlan &out, std::string &err);

// Rebuild block-CSR arrays (and the processing order) from a packed plan.
// Any output pointer may be null.
void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm);

}  // namespace spconv
