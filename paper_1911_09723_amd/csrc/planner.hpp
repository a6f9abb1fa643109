// Host-side format planner for the sparse 1x1 convolution.
//
// Pure C++17: no HIP dependency, so everything here runs and is tested on a
// machine without a GPU.  Input is the block-CSR weight format of the paper's
// library (Sec. 3.3: dense masked weights are converted to a block compressed
// sparse row form for inference; Sec. 3.2: a block is k consecutive output
// channels sharing one input channel).  Output is the packed image the GPU
// kernels stream.
//
// Lane groups.  A wavefront's 64 lanes form 64 / G groups of G lanes; each
// group works on one block row and each lane accumulates 16 / G vectors of 16
// bytes of output columns (the group together covers the 256-byte tile row).
// A lane needs the channel and the weights of every stored block of its row,
// so the G lanes of a group load the same 16-byte records: one vector load
// per lane per step of 4 slots, with no cross-lane broadcast instruction.
//
// Packed layout (all int32 / fp32, little-endian):
//
//   A *bundle* is NB = 64 / G block rows that one wavefront processes at the
//   same time, one row per lane group.  Bundles are made of consecutive rows
//   in processing order (descending nonzero count unless reordering is off),
//   so the rows of a bundle have similar lengths.  Its length is the longest
//   of its rows rounded up to a whole number of *steps* of 4 slots (at least
//   one step); shorter rows are padded with (channel 0, weight 0) slots, which
//   add an exact zero.
//
//   Bundles are assigned to the `waves` wavefronts of a workgroup by longest
//   processing time first; wave_ptr[w] .. wave_ptr[w+1] are wave w's bundles,
//   stored in that order as one continuous stream of steps.  Step s (a global
//   step index) holds, for group q < NB and slot u < 4, entry
//       e = (s * NB + q) * 4 + u
//   idx[e]           input channel * row_scale (row_scale = 256, the bytes of
//                    one LDS strip row, for the strip kernel; 1 for the direct
//                    kernel)
//   val[e*k + i]     weight of block-row element i (fp16-rounded for fp16 storage)
//   so the lanes of group q read idx bytes (s*NB + q)*16 .. +15 and val bytes
//   (s*NB + q)*16k .. +16k-1: the 4 slots of their row in step s.
//
//   Padding slots read strip row strip_rows - 1 (channel 0 for the direct
//   kernel): a row of the strip's upper part (below).
//
//   hdr[2*b + 0]     first (global) step of bundle b
//   hdr[2*b + 1]     steps of bundle b
//   rows[NB*b + q]   block row of group q of bundle b, or -1 (padding group)
//   bias[(NB*b + q)*k + i]  bias of output channel rows[..]*k + i (0 for padding)
//   rank[b]          position of bundle b in the longest-first order; a tile
//                    shared by P workgroups (P a power of two up to max_parts)
//                    gives part p the bundles with rank % P == p.
//
//   Strip halves.  The strip's rows are split at split_rows (a multiple of 4):
//   the lower part holds channels [0, split_rows), the upper part the rest.
//   Since every row reads its channels in ascending order, a bundle stops
//   reading the lower part after a few steps and starts reading the upper part
//   after a few steps; per wave (stream offsets from its first step):
//   wave_meta[2*w + 0]  steps after which the wave no longer reads the lower part
//   wave_meta[2*w + 1]  first step that reads the upper part (stream length if none)
//   A kernel can then refill the lower part with the next tile's channels while
//   the wavefronts finish the current tile in the upper part, and the other way
//   round.
//
// The per-row summation order is ascending input channel (the CSR order), with
// padding zeros after the last stored block; it does not depend on the bundle
// grouping, so the result is bitwise independent of reordering, lane-group
// width, wave assignment and splitting.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace spconv {

enum Status { OK = 0, E_ARG = 1, E_FORMAT = 2, E_SHAPE = 3, E_UNSUPPORTED = 4, E_NOMEM = 5, E_HIP = 6 };

enum Kernel { KERNEL_STRIP = 0, KERNEL_DIRECT = 1 };

// Largest LDS footprint of one workgroup on gfx950 (160 KiB per CU).
constexpr int64_t kMaxLdsBytes = 160 * 1024;
// Bytes of one strip row in LDS (one input channel over one tile of columns).
constexpr int32_t kRowBytes = 256;
// Slots per step (one 16-byte record of channels per lane group).
constexpr int32_t kStepSlots = 4;
// Wavefronts per workgroup (1024 threads).
constexpr int32_t kMaxWaves = 16;
// Finest split of a tile over workgroups.
constexpr int32_t kMaxParts = 64;
// LDS bytes of the strip-refill counters at the end of a workgroup's LDS.
constexpr int32_t kCtlBytes = 16;

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
    int32_t kernel = 0;       // 0 automatic, 1 strip, 2 direct
    int32_t group_lanes = 0;  // 0 automatic, else 4, 8 or 16 lanes per block row
    int32_t waves = 0;        // 0 automatic, else 1 .. 16 wavefronts per workgroup
};

struct PackedPlan {
    // shape and epilogue
    int32_t cout = 0, cin = 0, k = 1, act = 0, storage = 0;
    // launch geometry
    int32_t kernel = KERNEL_STRIP;
    int32_t group_lanes = 4;     // G: lanes per block row
    int32_t bundle_rows = 16;    // NB = 64 / G block rows per bundle
    int32_t cols_per_lane = 16;  // (16 / G) vectors of 16 bytes
    int32_t tile_cols = 64;      // 256 bytes of columns
    int32_t row_scale = kRowBytes;
    int32_t waves = 1;           // wavefronts per workgroup (each owns a list of bundles)
    int32_t strip_rows = 0;      // cin rounded up to a multiple of 4 (strip kernel)
    int32_t split_rows = 0;      // rows of the strip's lower part (a multiple of 4)
    int32_t busy_waves = 0;      // wavefronts with at least one bundle
    int32_t lds_bytes = 0;       // strip + bundle table (strip kernel)
    int32_t max_parts = 1;       // most workgroups that may share one tile
    // packed streams
    std::vector<int32_t> idx;
    std::vector<float> val;
    std::vector<int32_t> hdr;
    std::vector<int32_t> rows;
    std::vector<float> bundle_bias;
    std::vector<int32_t> rank;
    std::vector<int32_t> wave_ptr;
    std::vector<int32_t> wave_meta;
    std::vector<int32_t> perm;     // block rows in processing order
    std::vector<int32_t> row_nnz;  // stored blocks per block row (host only; for unpacking)
    // statistics
    int64_t nnzb = 0;
    int64_t slots = 0;  // packed slots of all groups including padding
    int64_t max_wave_cost = 0;
    int64_t sum_wave_cost = 0;

    int32_t nbundles() const { return static_cast<int32_t>(hdr.size() / 2); }
    int64_t steps() const { return static_cast<int64_t>(idx.size()) / (4 * bundle_rows); }
    // 32-bit words of the LDS bundle table: rows, biases
    int32_t table_words() const { return nbundles() * bundle_rows * (1 + k); }
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
