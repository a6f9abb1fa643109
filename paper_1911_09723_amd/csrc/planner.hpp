// Host-side format planner for the sparse 1x1 convolution.
//
// Pure C++17: no HIP dependency, so everything here runs and is tested on a
// machine without a GPU.  Input is the block-CSR weight format of the paper's
// library (Sec. 3.3: dense masked weights are converted to a block compressed
// sparse row form for inference; Sec. 3.2: a block is k consecutive output
// channels sharing one input channel).  Output is the packed image the GPU
// kernels stream.
//
// Packed layout (all int32 / fp32, little-endian):
//
//   A *bundle* is 4 block rows that one wavefront processes at the same time,
//   one row per group of 16 lanes.  Bundles are made of consecutive rows in
//   processing order (descending nonzero count unless reordering is off), so
//   the rows of a bundle have similar lengths.  Its length is the longest of
//   its rows rounded up to a whole number of *steps* of 4 slots (at least one
//   step); shorter rows are padded with (channel 0, weight 0) slots, which add
//   an exact zero.
//
//   Bundles are assigned to the `waves` wavefronts of a workgroup by longest
//   processing time first; wave_ptr[w] .. wave_ptr[w+1] are wave w's bundles.
//   A wavefront's bundles, in that order, form one continuous stream of steps,
//   stored as *chunks* of 4 steps: chunk q holds, for lane group g and slot
//   u < 16 of that group's 16 slots in the chunk (steps 4q .. 4q+3, 4 slots
//   each), entry
//       e = 64 * (wave_chunk[w] + q) + 16 * g + u
//   so lane L of a wavefront loads entry 64 * chunk + L: one coalesced load
//   per chunk.
//   idx[e]           input channel * row_scale (row_scale = bytes of one LDS
//                    strip row for the strip kernel, 1 for the direct kernel)
//   val[e*k + i]     weight of block row element i (fp16-rounded for fp16 storage)
//
//   hdr[2*b + 0]     first step of bundle b within its wavefront's stream
//   hdr[2*b + 1]     steps of bundle b
//   meta: the table the strip kernel copies into LDS, in three arrays
//     rows[4*b + g]              block row of lane group g, or -1 (padding group)
//     bias[(4*b + g)*k + i]      bias of output channel rows[..]*k + i (0 for padding), fp32 bits
//     steps[b]                   = hdr[2*b + 1]
//   split[65*w + i]  first bundle of part i of 64 of wave w's stream (parts cut
//                    at bundle boundaries, each about 1/64 of the steps);
//                    split[65*w + 64] = wave_ptr[w + 1].  A tile shared by P
//                    workgroups (P a power of two up to 64) gives part p the
//                    bundles split[65*w + p*64/P] .. split[65*w + (p+1)*64/P].
//
// The per-row summation order is ascending input channel (the CSR order), with
// padding zeros in between; it does not depend on the bundle grouping, so the
// result is bitwise independent of reordering, wave assignment and splitting.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace spconv {

enum Status { OK = 0, E_ARG = 1, E_FORMAT = 2, E_SHAPE = 3, E_UNSUPPORTED = 4, E_NOMEM = 5, E_HIP = 6 };

enum Kernel { KERNEL_STRIP = 0, KERNEL_DIRECT = 1 };

// Largest LDS footprint of one workgroup on gfx950 (160 KiB per CU).
constexpr int64_t kMaxLdsBytes = 160 * 1024;
// Lanes sharing one block row: one 16-lane DPP row of a wavefront.
constexpr int32_t kLanesPerRow = 16;
// Block rows per bundle (lane groups per wavefront).
constexpr int32_t kGroups = 64 / kLanesPerRow;
// Slots per lane group in one chunk (one per lane) and steps per chunk.
constexpr int32_t kChunkSlots = kLanesPerRow;
constexpr int32_t kChunkSteps = kChunkSlots / 4;
// Finest split of a wavefront's stream.
constexpr int32_t kMaxParts = 64;
// Wavefronts per workgroup (1024 threads).
constexpr int32_t kMaxWaves = 16;
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
    int32_t kernel = 0;     // 0 automatic, 1 strip, 2 direct
    int32_t vec_bytes = 0;  // 0 automatic, else 8 or 16 bytes of X per lane and nonzero
    int32_t waves = 0;
    int32_t prefetch = 1;
};

struct PackedPlan {
    // shape and epilogue
    int32_t cout = 0, cin = 0, k = 1, act = 0, storage = 0;
    // launch geometry
    int32_t kernel = KERNEL_STRIP;
    int32_t vec_bytes = 16;      // bytes of X each lane reads per nonzero
    int32_t cols_per_lane = 4;   // vec_bytes / element size
    int32_t tile_cols = 64;      // kLanesPerRow * cols_per_lane
    int32_t row_scale = 256;     // idx = channel * row_scale
    int32_t waves = 1;           // compute wavefronts (each owns a list of bundles)
    int32_t loader_waves = 0;    // wavefronts that prefetch the next strip (strip kernel)
    int32_t lds_bytes = 0;       // strip + bundle table (strip kernel)
    int32_t strip_bytes = 0;
    int32_t max_parts = 1;       // most workgroups that may share one tile
    // packed streams
    std::vector<int32_t> idx;
    std::vector<float> val;
    std::vector<int32_t> hdr;
    std::vector<int32_t> rows;
    std::vector<float> bundle_bias;  // bias of each (bundle, group, block element)
    std::vector<int32_t> wave_ptr;
    std::vector<int32_t> wave_chunk;
    std::vector<int32_t> split;
    std::vector<int32_t> perm;     // block rows in processing order
    std::vector<int32_t> row_nnz;  // stored blocks per block row (host only; for unpacking)
    // statistics
    int64_t nnzb = 0;
    int64_t slots = 0;  // packed entries including padding (64 per chunk)
    int64_t max_wave_cost = 0;
    int64_t sum_wave_cost = 0;

    int32_t nbundles() const { return static_cast<int32_t>(hdr.size() / 2); }
    // 32-bit words of the LDS bundle table: rows, biases, steps
    int32_t meta_words() const { return nbundles() * (kGroups * (1 + k) + 1); }
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
