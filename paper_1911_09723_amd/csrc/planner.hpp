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
//   one step); shorter rows are padded with weight-0 slots (below).
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
//   Padding slots read channel strip_rows (strip kernel: an LDS row of zeros
//   after the strip, so they add an exact zero whatever X holds) or channel 0
//   (direct kernel).
//
//   hdr[2*b + 0]     first (global) step of bundle b
//   hdr[2*b + 1]     steps of bundle b
//   rows[NB*b + q]   block row of group q of bundle b, or -1 (padding group)
//   bias[(NB*b + q)*k + i]  bias of output channel rows[..]*k + i (0 for padding)
//   rank[b]          position of bundle b in the longest-first order; a tile
//                    shared by P workgroups (P a power of two up to max_parts)
//                    gives part p the bundles with rank % P == p.
//
// Interleaved streams (strip kernel).  The pipelined kernel keeps the strip as
// `regions` parts of region_rows channels (the last may be shorter) and
// refills each part with the next tile's channels as soon as every wavefront
// is done with it.  That only overlaps copying with computing when each
// wavefront reads the channels of a tile roughly in ascending order once, so
// its stream interleaves the steps of `pipe_sets` bundles at a time (one
// accumulator set each): the bundles wave_ptr[w] + j*S .. + S - 1 (S =
// pipe_sets) form its j-th set group, bundle wave_ptr[w] + j*S + i uses set
// i, and the group's steps are merged by the mean of the lowest and highest
// channel each step reads, keeping every bundle's own step order (so every
// row still sums in ascending channel order).  pidx / pval hold the same
// records as idx / val, with each wave's steps (same global step range) in
// that order.  Per wave:
//   psel[sel_ptr[w] + i / 16] bits 2*(i % 16), +1   set of the wave's i-th step,
//                    and whether it is its bundle's last step
//   wave_ev[8*w + 0 .. 3]   (pos << 4) | region for each region the wave reads,
//                    sorted by pos: the first step that reads it ("need")
//   wave_ev[8*w + 4 .. 7]   the same for the last step that reads it
//                    ("release"; step 0 for a region it never reads)
//   unused entries hold INT32_MAX.
//
// The per-row summation order is ascending input channel (the CSR order), with
// padding zeros after the last stored block; it does not depend on the bundle
// grouping, so the result is bitwise independent of reordering, lane-group
// width, wave assignment, interleaving and splitting.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace spconv {

enum Status { OK = 0, E_ARG = 1, E_FORMAT = 2, E_SHAPE = 3, E_UNSUPPORTED = 4, E_NOMEM = 5, E_HIP = 6 };

enum Kernel { KERNEL_STRIP = 0, KERNEL_DIRECT = 1, KERNEL_INDEXED = 2 };

// Largest LDS footprint of one workgroup on gfx950 (160 KiB per CU).
constexpr int64_t kMaxLdsBytes = 160 * 1024;
// Bytes of one strip row in LDS (one input channel over one tile of columns).
constexpr int32_t kRowBytes = 256;
// Slots per step (one 16-byte record of channels per lane group).
constexpr int32_t kStepSlots = 4;
// A bundle's row-table entry for the second piece of a split row (its lane
// group's partial sums are added into the previous group's before the
// epilogue); and the shortest row that may be split.
constexpr int32_t kRowPiece = -2;
constexpr int32_t kSplitMinNnz = 32;
// Wavefronts per workgroup (1024 threads).
constexpr int32_t kMaxWaves = 16;
// Finest split of a tile over workgroups.
constexpr int32_t kMaxParts = 64;
// Most parts of the strip the pipelined kernel refills independently.
constexpr int32_t kMaxRegions = 4;
constexpr int32_t kAutoRegionRows = 192;  // channels per strip part of the automatic choice
// LDS bytes of the strip-refill counters at the end of a workgroup's LDS
// (per region: wavefronts done with it, copies of it landed).
constexpr int32_t kCtlBytes = 8 * kMaxRegions;
// Steps per selector word of the interleaved streams (2 bits each).
constexpr int32_t kSelSteps = 16;
// Events per wavefront in wave_ev.
constexpr int32_t kWaveEvents = 2 * kMaxRegions;
// Floats per channel of a fused depthwise stage's parameters (9 taps, bias, padding to 64 bytes).
constexpr int32_t kDwParams = 16;
// Smallest depthwise staging area worth a second workgroup per CU.
constexpr int64_t kMinStageBytes = 16 * 1024;

// Register-indexed kernel (KERNEL_INDEXED): rows are grouped into slots of
// kSlotRows output channels, one slot per wavefront; the wavefront walks its
// slot's nonzeros by ascending input channel, reads each channel's X values
// once per record from an LDS ring, and adds them into the accumulator of the
// record's row, chosen at run time by register-relative addressing.
//
//   Slots.  Block rows (1 x k blocks) are assigned to slots of at most
//   kSlotRows / k block rows, longest processing time first (heaviest rows
//   first, each to the least loaded slot with room), so every slot carries
//   about the same number of stored blocks.  Slot row i is output channel
//   rslot_rows[s * kSlotRows + i] (-1: unused), with bias rslot_bias[...].
//   A block at slot position b occupies slot rows b*k .. b*k + k - 1.
//
//   Records (kRecWords 32-bit words each): the stored blocks of one slot at one
//   input channel c, at most kRecSlots(k) = 3, 2, 1 blocks for k = 1, 2, 4:
//     w[0]  (c % kRing) * kRingRowBytes (LDS byte offset of the ring row holding c)
//     w[1]  first block's slot row | (more than 1 block) << 8 | (more than 2) << 9
//     w[2]  second block's slot row (k <= 2), w[3] third (k == 1)
//     w[4..7]  weights: k == 1: one per block; k == 2: 2 per block; k == 4: the 4
//   A slot's records ascend by channel.  Channels come in chunks of kChunk;
//   each chunk's records fill whole batches (kBatchRecs records, kRecWords *
//   kBatchRecs words), padded with records of weight 0, and a chunk without
//   stored blocks in the slot still gets one batch of such records, so a
//   wavefront passes every chunk.  The first record of every batch carries
//   the batch's flags in word flag_word(k) (7 for k == 1, else 3): bit 0 the
//   batch is its chunk's last, bit 1 it is the stream's last.  Padding records
//   name the chunk's first channel and slot row 0.  Slot s's stream starts at
//   batch rslot_batch[s]; chunk q of it starts at batch rslot_chunk[s * (nch +
//   1) + q] of the stream (q = nch: the stream's length) and holds
//   rslot_nrec[s * nch + q] stored records.  The record array ends with
//   kBatchRecs * 2 zero records (read ahead, unused).
//
//   Row pairs (columns left over after the kernel's whole tiles): pair j is
//   output channels 2j and 2j + 1; rpair_ptr[j] .. rpair_ptr[j + 1] index its
//   entries in rpair_ent, 4 words each: channel | (mask << 24) (bit 0: channel
//   2j has a weight at c, bit 1: 2j + 1 has one), the two weights, 0.  Entries
//   ascend by channel.
//
// Every row still sums its products in ascending input channel from zero,
// then adds the bias, so results do not depend on the slot assignment.
constexpr int32_t kSlotRows = 16;
constexpr int32_t kRecWords = 8;
constexpr int32_t kBatchRecs = 2;
constexpr int32_t kRing = 96;        // LDS ring rows (channels) of the register-indexed kernel
constexpr int32_t kRingRowBytes = 1536;  // one ring row: 6 column slots of 64 fp32
constexpr int32_t kChunk = 16;
static_assert(kRing % kChunk == 0, "a chunk never wraps around the ring");
constexpr int32_t kSlotsPerGroup = 16;
inline int32_t rec_slots(int32_t k) { return k == 1 ? 3 : k == 2 ? 2 : 1; }
inline int32_t flag_word(int32_t k) { return k == 1 ? 7 : 3; }
constexpr uint32_t kLastOfChunk = 1u;
constexpr uint32_t kLastOfStream = 2u;

// Lockstep kernel (kernel = 4): a wavefront steps the block rows of one
// "group set" in lockstep, one stored block each per step, over a tile of
// output columns whose X rows sit in one of two LDS buffers.  Two modes:
//   matrix (1 x 4 blocks): a stored block times a 4-column X vector is a
//     4 x 4 outer product, and the matrix cores' fp32 4x4x1 instruction
//     computes 16 of them at once, each from its own block of 4 lanes
//     (register r of lane 4b + t gets A[4b + r] * B[4b + t] + C, one
//     rounding, like a fused multiply-add);
//   vector (unstructured, 1 x 1): each lane adds weight * X for its row and 4
//     columns with fused multiply-adds.
//
//   Tiles.  otw = 32 consecutive output columns (16 in vector mode when cin
//   exceeds kOuterMaxCin32); the tile's X rows (4 * otw bytes each: channel c
//   at byte 4 * otw * c, then unused rows up to ozrow = cin rounded up to the
//   rows one 1 KB copy moves, then one row of zeros) fill one of two LDS
//   buffers.  A lane covers 4 columns, so a lane group of otw / 4 lanes
//   covers the tile and a wavefront has ogroups = 256 / otw groups.
//   Group sets.  Block rows sorted by stored blocks (descending, ties by row
//   index) are taken ogroups at a time; group g works on block row g of its
//   set, all in lockstep, in ascending channel, for 4 * nquads steps (the
//   longest row rounded up to whole quads of 4 steps, at least one); a row
//   past its last block reads the zero row with weight 0.
//   Records, per set and quad j of steps 4j .. 4j + 3:
//     orec  per weight slot u (matrix: u = 4g + t, 32 slots, element t of
//           group g's block; vector: u = g), four words: the slot's weight at
//           each of the 4 steps (fp32 bits, rounded to fp16 first for fp16
//           storage; 0 for padding).  Matrix lanes 8g + t and 8g + 4 + t read
//           slot 4g + t; vector lanes of group g read slot g.
//     ooff  per group g, four words: the LDS byte offset of the channel row
//           each of the 4 steps reads (channel * 4 * otw; padding
//           ozrow * 4 * otw).
//   Set o's quads start at quad ooct_tab[kOctWords * o] of both arrays and run
//   ooct_tab[.. + 1] quads; words 2 .. 2 + ogroups - 1 hold its block rows
//   (-1: none).  Both arrays end with kOuterAhead zero quads (read ahead).
//   Waves.  The sets are dealt to owaves wavefronts twice, longest first to
//   the least loaded: once for even tiles, then again for odd tiles starting
//   from the even loads, so each wavefront's two-tile total is balanced.  Wave
//   w's sets for tiles of parity q are owave_oct[owave_ptr[q * owaves + w] ..
//   owave_ptr[q * owaves + w + 1]).
constexpr int32_t kOuterCols = 32;   // the widest tile
constexpr int32_t kOctWords = 32;
constexpr int32_t kOuterAhead = 4;   // quads of records read ahead
constexpr int32_t kOuterQuadSteps = 4;
// Widest input with two buffers of 32-column tiles (and their control words)
// in one workgroup's LDS; with 16-column tiles (vector mode only).
constexpr int32_t kOuterMaxCin32 = 632;
constexpr int32_t kOuterMaxCin16 = 1264;

struct Input {
    int32_t cout = 0, cin = 0, block_rows = 1;
    // input channels per block (Fig. 5: 4x1 and 2x2 blocks beside 1x4): block t
    // covers channels col_idx[t] .. col_idx[t] + block_cols - 1 and holds
    // values[(t * block_rows + i) * block_cols + j]; the planner expands it into
    // block_cols consecutive entries of the kernels' 1 x block_rows format
    int32_t block_cols = 1;
    const int32_t *row_ptr = nullptr;
    const int32_t *col_idx = nullptr;
    const float *values = nullptr;
    const float *bias = nullptr;
    int32_t act = 0;      // 0 none, 1 relu, 2 relu6
    int32_t storage = 0;  // 0 fp32, 1 fp16
    // Optional depthwise 3x3 stage run on the input first (the MobileNet block
    // order, Sec. 2; the library's CHW depthwise kernels, Sec. 3.3):
    //   D[n, c, oy, ox] = dw_act(dw_bias[c] + sum_{dy, dx} dw_weights[c][dy][dx]
    //                               * X[n, c, s*oy + dy - 1, s*ox + dx - 1])
    // with zero padding 1 and stride s = dw_stride; the 1x1 then reads D.
    int32_t dw_stride = 0;               // 0: no depthwise stage; else 1 or 2
    const float *dw_weights = nullptr;   // [cin][3][3]
    const float *dw_bias = nullptr;      // [cin] or null for zeros
    int32_t dw_act = 0;
};

struct Options {
    int32_t reorder = 1;
    int32_t host_only = 0;
    int32_t kernel = 0;       // 0 automatic, 1 strip, 2 direct, 3 register-indexed, 4 outer-product
    int32_t group_lanes = 0;  // 0 automatic, else 4, 8 or 16 lanes per block row
    int32_t waves = 0;        // 0 automatic, else 1 .. 16 wavefronts per workgroup
    int32_t pipe_sets = 0;    // 0 automatic, else 1 or 2 bundles interleaved per wavefront
    int32_t regions = 0;      // 0 automatic, else 1 .. kMaxRegions strip parts
    int32_t lane_cols = 0;    // register-indexed kernel: 0 automatic, else 1 .. 6 columns per lane
    int32_t split = 1;        // heavy rows may be packed as two pieces (off for channel-range passes,
                              // whose rows must be summed in one ascending pass)
};

// One lane group of a bundle as the row table describes it (group_row).
struct GroupRow {
    int32_t row;    // the output (block) row, -1 for none
    int32_t piece;  // -1 the whole row; 0 / 1 the even / odd nonzeros of a split row
    int32_t n;      // real entries of the group
};

struct PackedPlan {
    // shape and epilogue
    int32_t cout = 0, cin = 0, k = 1, act = 0, storage = 0;
    int32_t kc = 1;  // input channels per block of the caller's format (the packed streams hold the expansion)
    // launch geometry
    int32_t kernel = KERNEL_STRIP;
    int32_t group_lanes = 4;     // G: lanes per block row
    int32_t bundle_rows = 16;    // NB = 64 / G block rows per bundle
    int32_t cols_per_lane = 16;  // (16 / G) vectors of 16 bytes
    int32_t tile_cols = 64;      // 256 bytes of columns
    int32_t row_scale = kRowBytes;
    int32_t waves = 1;           // wavefronts per workgroup (each owns a list of bundles)
    int32_t strip_rows = 0;      // cin rounded up to a multiple of 4 (strip kernel)
    int32_t busy_waves = 0;      // wavefronts with at least one bundle
    int32_t split_rows = 0;      // rows packed as two pieces (heavy rows)
    int32_t lds_bytes = 0;       // strip, zero row, bundle table, counters (strip kernel)
    int32_t pipe_sets = 1;       // bundles a wavefront interleaves (strip kernel)
    int32_t regions = 1;         // strip parts refilled independently (strip kernel)
    int32_t region_rows = 0;     // channels per part, a multiple of 4
    int32_t max_parts = 1;       // most workgroups that may share one tile
    // fused depthwise 3x3 stage (Input::dw_stride); such a plan runs the simple
    // strip loop, which computes each strip from the input instead of copying it
    int32_t dw_stride = 0, dw_act = 0;
    int32_t stage_off = 0;    // LDS [stage_off, stage_off + stage_bytes): the depthwise input windows
    int32_t stage_bytes = 0;  // (all LDS left after the strip and the bundle table)
    std::vector<float> dw;  // [strip_rows][kDwParams]: the 9 taps (dy-major), then the bias; 0 past cin
    // packed streams
    std::vector<int32_t> idx;
    std::vector<float> val;
    std::vector<int32_t> hdr;
    std::vector<int32_t> rows;
    std::vector<float> bundle_bias;
    std::vector<int32_t> rank;
    std::vector<int32_t> wave_ptr;
    std::vector<int32_t> pidx;     // interleaved streams (strip kernel)
    std::vector<float> pval;
    std::vector<uint32_t> psel;
    std::vector<int32_t> sel_ptr;
    std::vector<int32_t> wave_ev;
    // register-indexed kernel (planner.hpp, "Register-indexed kernel"); empty
    // when the plan cannot use it
    int32_t use_indexed = 0;     // spconv_run launches the register-indexed kernel
    int32_t rslots = 0;          // slots of kSlotRows output channels
    int32_t rgroups = 0;         // groups of slots sharing one LDS ring (one workgroup each)
    int32_t rwaves = 0;          // wavefronts per workgroup = slots per group (the last may have fewer)
    int32_t rnch = 0;            // chunks of kChunk input channels
    int32_t rlane_cols = 0;      // columns per lane fixed by the caller (0: chosen per run)
    int32_t auto_kernel = 0;     // the caller left the kernel to the library (options.kernel = 0)
    std::vector<uint32_t> rrec;
    std::vector<int32_t> rslot_batch;
    std::vector<int32_t> rslot_chunk;
    std::vector<int32_t> rslot_nrec;
    std::vector<int32_t> rslot_rows;
    std::vector<float> rslot_bias;
    std::vector<int32_t> rpair_ptr;
    std::vector<uint32_t> rpair_ent;
    std::vector<float> rrow_bias;  // bias of every output channel (the row-pair phase)
    // outer-product kernel (planner.hpp, "Outer-product kernel"); empty when
    // the plan cannot use it
    int32_t use_outer = 0;   // spconv_run launches the lockstep kernel
    int32_t omode = 0;       // 0 matrix (1 x 4 blocks), 1 vector (unstructured)
    int32_t otw = 32;        // tile columns
    int32_t ogroups = 8;     // lane groups (block rows of a set) per wavefront
    int32_t oocts = 0;       // group sets
    int32_t owaves = 0;      // wavefronts per workgroup
    int32_t ozrow = 0;       // LDS row of zeros
    std::vector<uint32_t> orec;
    std::vector<uint32_t> ooff;
    std::vector<int32_t> ooct_tab;
    std::vector<int32_t> owave_ptr;
    std::vector<int32_t> owave_oct;
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

// Dense weights (Sec. 3.3: dense masked weights are converted to a block
// compressed sparse row form for inference).  `dense` is row-major
// [cout][cin]; a weight is stored when it is not zero (-0.0 counts as zero).
//
// The largest k in {4, 2, 1} dividing cout for which every aligned group of k
// rows has a single zero / nonzero pattern in every column (Sec. 3.2: output
// channel blocks of 2 and 4), so a 1 x k block-CSR stores no zero.
Status detect_block_rows(int32_t cout, int32_t cin, const float *dense, int32_t &k, std::string &err);
// The 1 x k block-CSR of a dense weight: a block (aligned group of k rows,
// one column) is stored when any of its k weights is nonzero, with its k
// weights in block-major order (zeros included).  Sets nnzb and, when not
// null, row_ptr[cout/k + 1]; with col_idx not null also writes col_idx[nnzb]
// and values[nnzb * k] (E_ARG when nnzb exceeds `capacity` blocks).
Status dense_to_bcsr(int32_t cout, int32_t cin, const float *dense, int32_t k, int32_t *row_ptr,
                     int32_t *col_idx, float *values, int64_t capacity, int64_t &nnzb, std::string &err);

// The same for blocks of kr output x kc input channels (Fig. 5: 4x1 and 2x2
// beside 1x4): the (kr, kc) in {1, 2, 4}^2 with the most weights per block
// (output blocks first on a tie) for which every aligned block is all zero or
// all nonzero; and the conversion to that block-CSR (col_idx = first input
// channel of a block, values[(t * kr + i) * kc + j]).  kc = 1 is
// dense_to_bcsr.
Status detect_blocks(int32_t cout, int32_t cin, const float *dense, int32_t &kr, int32_t &kc, std::string &err);
Status dense_to_blocks(int32_t cout, int32_t cin, const float *dense, int32_t kr, int32_t kc, int32_t *row_ptr,
                       int32_t *col_idx, float *values, int64_t capacity, int64_t &nnzb, std::string &err);

// Check the block-CSR arrays; on failure return the status and set `err`.
Status validate(const Input &in, std::string &err);

// Validate, order, bundle, balance and pack.  Returns OK or an error with `err` set.
Status build_plan(const Input &in, const Options &opt, PackedPlan &out, std::string &err);

// Rebuild block-CSR arrays (and the processing order) from a packed plan.
// Any output pointer may be null.
GroupRow group_row(const PackedPlan &p, int32_t b, int32_t q);
void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm);

// Build the register-indexed kernel's slots, records and row pairs (fields
// r* of PackedPlan) from 1 x k block-CSR arrays; `order` lists the block rows
// in processing order.
void build_indexed(const Input &in, const std::vector<int32_t> &order, PackedPlan &p);

// Whether the lockstep kernel can run this layer: 1 x 4 blocks (matrix
// mode) with cin <= kOuterMaxCin32, or unstructured fp32 (vector mode) with
// cin <= kOuterMaxCin16; no depthwise stage.
bool outer_supported(const Input &in);
// Build its group sets, records and wave lists (fields o* of PackedPlan).
void build_outer(const Input &in, PackedPlan &p);
// Rebuild block-CSR arrays from the lockstep kernel's records, checking their
// structure (lockstep padding, ascending channels, offsets, wave lists).
// E_FORMAT with `err` set when inconsistent or absent.
Status unpack_outer(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, std::string &err);

// Rebuild block-CSR arrays from the register-indexed records (and separately
// from the row pairs), checking the stream structure: batch alignment of
// chunks, ascending channels, ring rows, slot-row ranges.  E_FORMAT with `err`
// set when inconsistent or absent.
Status unpack_indexed(const PackedPlan &p, bool from_pairs, int32_t *row_ptr, int32_t *col_idx, float *values,
                      std::string &err);

// The same from the interleaved streams, walking them as the pipelined kernel
// does (selector bits, set groups) and checking that every strip read lies
// between its region's need and release events.  Returns OK, or E_FORMAT with
// `err` set when the streams are inconsistent or the plan has none.
Status unpack_interleaved(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values,
                          std::string &err);

}  // namespace spconv
