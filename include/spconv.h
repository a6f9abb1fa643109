/*
 * spconv.h -- sparse 1x1 convolution (sparse weights x dense CHW activations)
 * on AMD Instinct MI355X (gfx950).
 *
 * The operation (Fast Sparse ConvNets, Sec. 3.2 and Fig. 2: a 1x1
 * convolution over activations stored channel-major, CHW, is a sparse-matrix
 * times dense-matrix product; Sec. 3.2: output-channel blocks of k rows share
 * one nonzero pattern; Sec. 3.3: weights are converted to a block-compressed
 * sparse row format for inference).  For every image n, output channel r and
 * spatial position p:
 *
 *     Y[n, r, p] = act( b[r] + sum_{stored (r, c)} W[r, c] * X[n, c, p] )
 *
 * with act one of identity, max(v, 0) or min(max(v, 0), 6), evaluated in
 * fp32 and rounded once to the storage type.
 *
 * Conventions for every call:
 *   - Status codes are returned; no C++ exception crosses this interface.
 *     After a failure, spconv_last_error() returns a message for the calling
 *     thread.
 *   - Host arrays passed to a call are only read during that call; the caller
 *     keeps ownership and may free them on return.
 *   - Device pointers are plain HIP device addresses (e.g. from hipMalloc or a
 *     PyTorch tensor's data_ptr()); they stay owned by the caller.
 */
#ifndef SPCONV_H
#define SPCONV_H

#include <stddef.h>
#include <stdint.h>

/* The library is built with hidden visibility; only these entry points are exported. */
#if defined(__GNUC__) || defined(__clang__)
#define SPCONV_API __attribute__((visibility("default")))
#else
#define SPCONV_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct spconv_plan_s *spconv_plan; /* opaque, immutable once created */

typedef enum {
    SPCONV_OK = 0,
    SPCONV_E_ARG = 1,         /* bad argument: NULL pointer, negative size, x/y overlap, wrong device */
    SPCONV_E_FORMAT = 2,      /* malformed CSR / block-CSR arrays */
    SPCONV_E_SHAPE = 3,       /* inconsistent sizes (cout % block_rows, sizes too large) */
    SPCONV_E_UNSUPPORTED = 4, /* valid request this build does not implement */
    SPCONV_E_NOMEM = 5,       /* host or device allocation failed */
    SPCONV_E_HIP = 6          /* a HIP runtime call failed (message names it) */
} spconv_status;

typedef enum { SPCONV_F32 = 0, SPCONV_F16 = 1 } spconv_dtype;

typedef enum { SPCONV_ACT_NONE = 0, SPCONV_ACT_RELU = 1, SPCONV_ACT_RELU6 = 2 } spconv_act;

/*
 * Build a plan from CSR (block_rows = 1) or 1 x block_rows block-CSR weights
 * (Sec. 3.2: k consecutive output channels share one column pattern; the
 * paper's kernels block by 2 and 4 output channels).  Validates the arrays, orders the
 * (block) rows by nonzero count for load balance, packs column indices and
 * values into the layout the kernels stream, and copies the result to the
 * current HIP device.  Synchronous.
 *
 *   out         receives the plan; set to NULL on failure
 *   cout, cin   output / input channels; cout % block_rows == 0, both >= 1
 *   block_rows  1, 2 or 4
 *   row_ptr     host, cout/block_rows + 1 entries: row_ptr[0] = 0, non-decreasing
 *   col_idx     host, row_ptr[cout/block_rows] entries, each in [0, cin), strictly
 *               ascending within a (block) row
 *   values      host, row_ptr[end] * block_rows floats, block-major:
 *               values[t * k + i] = W[rb * k + i, col_idx[t]] for t in block row rb;
 *               must be finite.  With storage SPCONV_F16 each value is rounded to
 *               the nearest fp16 value (ties to even) before use.
 *   bias        host, cout floats, or NULL for zeros; kept in fp32
 *   act         epilogue activation
 *   storage     element type of X and Y (W is used at that precision; the
 *               accumulation is always fp32)
 *
 * Errors: SPCONV_E_ARG (NULL out/row_ptr, NULL col_idx/values with nonzeros,
 * bad enum), SPCONV_E_SHAPE, SPCONV_E_FORMAT (message names the first bad
 * entry), SPCONV_E_UNSUPPORTED (block_rows not 1, 2 or 4), SPCONV_E_NOMEM,
 * SPCONV_E_HIP (no usable device, allocation or copy failure).  Nothing is
 * leaked on failure.
 */
SPCONV_API spconv_status spconv_plan_create(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                 const int32_t *row_ptr, const int32_t *col_idx,
                                 const float *values, const float *bias, spconv_act act,
                                 spconv_dtype storage);

/*
 * Run the plan:  y = act(W x + b)  on NCHW tensors of the plan's storage type
 * (for a plan with a depthwise stage, see spconv_plan_create_fused: x is that
 * stage's input and y is n x cout x out_h x out_w).
 *
 *   x       device, n * cin * h * w elements, NCHW contiguous
 *   y       device, n * cout * h * w elements, NCHW contiguous; must not overlap x
 *           (every output channel reads every input channel, so in-place is impossible)
 *   n, h, w batch and spatial sizes, >= 0; n == 0 or h * w == 0 is a no-op
 *   stream  hipStream_t to launch on, or NULL for the default stream
 *
 * Asynchronous: returns once the kernel is queued on `stream`; x and y must
 * stay alive until that work completes.  Allocates nothing and never
 * synchronizes.  Pointers need only element alignment (16-byte alignment with
 * h * w a multiple of the vector width takes the fastest load path).  The plan
 * must have been created on the current device.  A plan is immutable, so
 * concurrent runs of one plan on different streams are safe.
 *
 * Errors: SPCONV_E_ARG (NULL plan/x/y with work to do, negative sizes, overlap,
 * other device, host-only plan), SPCONV_E_SHAPE (sizes beyond 2^31 columns or
 * elements beyond 2^62), SPCONV_E_UNSUPPORTED (the images one tile of output
 * columns touches, ((tile columns - 1) / (out_h * out_w) + 2) of them, span
 * 2^31 bytes or more of x or of y), SPCONV_E_HIP
 * (launch failure).  Every check on the arguments runs before any HIP call and
 * before a host-only plan is refused, so a host-only plan exercises them
 * without a device.  Faults during execution surface at the caller's next
 * synchronization.
 */
SPCONV_API spconv_status spconv_run(spconv_plan plan, const void *x, void *y, int32_t n, int32_t h, int32_t w,
                         void *stream);

/* Free the plan and its device buffers.  NULL is a no-op.  The caller must
 * ensure no queued run still uses the plan. */
SPCONV_API spconv_status spconv_destroy(spconv_plan plan);

/* Message for the calling thread's most recent failure ("" if none).  The
 * pointer stays valid until the next spconv_* call on the same thread. */
SPCONV_API const char *spconv_last_error(void);

/* ---------------------------------------------------------------------------
 * Dense weights.  Sec. 3.3: a trained (pruned) model keeps its weights as a
 * dense tensor with zeros, which the library converts to a block compressed
 * sparse row form for inference; Sec. 3.2: blocks of 2 or 4 consecutive
 * output channels that share one zero / nonzero pattern.  `dense` is host
 * memory, row-major [cout][cin] fp32 (W[r][c] at dense[r * cin + c]); a
 * weight is stored when it is not zero (-0.0 counts as zero); every value
 * must be finite (SPCONV_E_FORMAT names the first one that is not).  Host
 * only, synchronous; the caller keeps ownership of every array.
 * ------------------------------------------------------------------------- */

/*
 * The largest k in {4, 2, 1} that divides cout and for which every aligned
 * group of k rows (rows k*b .. k*b + k - 1) has the same zero / nonzero
 * pattern in every column, so that the 1 x k block-CSR stores no zero.
 *   block_rows  out: the detected k
 * Errors: SPCONV_E_ARG (NULL pointer), SPCONV_E_SHAPE (cout or cin < 1,
 * cin > 2^24), SPCONV_E_FORMAT (a non-finite weight).
 */
SPCONV_API spconv_status spconv_detect_block_rows(int32_t cout, int32_t cin, const float *dense, int32_t *block_rows);

/*
 * Convert a dense weight to 1 x block_rows block-CSR (the layout that
 * spconv_plan_create takes): block (b, c) is stored when any of
 * W[b*k .. b*k + k - 1][c] is nonzero, with all k of its weights (zeros
 * included), columns ascending within a block row.
 *   block_rows  1, 2 or 4; cout % block_rows == 0
 *   row_ptr     out, cout/block_rows + 1 entries, or NULL
 *   col_idx     out, `capacity` entries; NULL = only count the blocks
 *   values      out, capacity * block_rows entries (required with col_idx)
 *   capacity    blocks that col_idx / values can hold
 *   nnzb        out: number of stored blocks (set also on SPCONV_E_ARG for
 *               too small a capacity, so a caller can size its arrays with a
 *               first call that passes col_idx = NULL)
 * Errors: SPCONV_E_ARG (NULL dense / nnzb, values or row_ptr missing with
 * col_idx, capacity too small), SPCONV_E_UNSUPPORTED (block_rows not 1, 2 or
 * 4), SPCONV_E_SHAPE, SPCONV_E_FORMAT.
 */
SPCONV_API spconv_status spconv_dense_to_bcsr(int32_t cout, int32_t cin, const float *dense, int32_t block_rows,
                                   int32_t *row_ptr, int32_t *col_idx, float *values, int64_t capacity,
                                   int64_t *nnzb);

/*
 * spconv_plan_create from a dense weight: block_rows = 0 detects the block
 * height (spconv_detect_block_rows), else 1, 2 or 4; then converts
 * (spconv_dense_to_bcsr) and plans.  Other arguments and errors as for
 * spconv_plan_create.
 */
SPCONV_API spconv_status spconv_plan_create_dense(spconv_plan *out, int32_t cout, int32_t cin, const float *dense,
                                       int32_t block_rows, const float *bias, spconv_act act,
                                       spconv_dtype storage);

/* ---------------------------------------------------------------------------
 * The other CHW operators of a network (Sec. 3.3: besides the sparse 1x1,
 * the library provides the depthwise convolution, global average pooling
 * and a dense 3x3 stride-2 convolution from the HWC image to CHW; Sec. 3.1:
 * the first convolution stays dense).  fp32 only; every pointer is device
 * memory owned by the caller; one asynchronous kernel launch on `stream`
 * (NULL: the default stream); nothing is allocated and nothing synchronizes.
 * Sizes of 0 are no-ops.  Outputs must not overlap inputs (SPCONV_E_ARG).
 * ------------------------------------------------------------------------- */

/*
 * Dense 3x3 convolution, zero padding 1, from an HWC image to CHW:
 *   y[n, o, oy, ox] = act( bias[o] + sum_{dy, dx, i} weight[o][dy][dx][i]
 *                                     * x[n, s*oy + dy - 1, s*ox + dx - 1, i] )
 *   x       [n][h][w][cin]          weight  [cout][3][3][cin]
 *   bias    [cout] or NULL          y       [n][cout][(h-1)/s+1][(w-1)/s+1]
 *   stride  1 or 2 (the network stem uses 2)
 * Errors: SPCONV_E_ARG (NULL pointer with work to do, negative size, bad
 * stride or act, overlap), SPCONV_E_SHAPE (cin or cout < 1, too many
 * pixels, an image of 2^31 or more elements, n * ceil(ho * wo / 256) of
 * 2^31 or more), SPCONV_E_UNSUPPORTED (cin > 8), SPCONV_E_HIP.
 */
SPCONV_API spconv_status spconv_conv3x3_hwc(const float *x, const float *weight, const float *bias, spconv_act act,
                                 int32_t stride, float *y, int32_t n, int32_t h, int32_t w, int32_t cin,
                                 int32_t cout, void *stream);

/*
 * Depthwise 3x3 convolution, zero padding 1, on CHW tensors (a standalone
 * launch; spconv_plan_create_fused runs the same stage inside the 1x1):
 *   y[n, c, oy, ox] = act( bias[c] + sum_{dy, dx} weight[c][dy][dx] * x[n, c, s*oy + dy - 1, s*ox + dx - 1] )
 *   x [n][c][h][w], weight [c][3][3], bias [c] or NULL, y [n][c][(h-1)/s+1][(w-1)/s+1], stride 1 or 2.
 * Errors: SPCONV_E_ARG, SPCONV_E_SHAPE (too many outputs), SPCONV_E_HIP.
 */
SPCONV_API spconv_status spconv_depthwise3x3(const float *x, const float *weight, const float *bias, spconv_act act,
                                  int32_t stride, float *y, int32_t n, int32_t c, int32_t h, int32_t w,
                                  void *stream);

/*
 * Dense fully connected layer (the network's classifier, kept dense as in
 * Sec. 3.1 / Table 1):  y[n, r] = act( bias[r] + sum_c weight[r][c] * x[n][c] ),
 * fp32: the input channels are taken in 16 consecutive ranges, each summed
 * by FMA in ascending c from zero, and the range sums are added in ascending
 * order; then the bias.  x [n][cin], weight [cout][cin] row-major, bias
 * [cout] or NULL, y [n][cout].
 * Errors: SPCONV_E_ARG (NULL pointer with work to do, negative size, bad act,
 * overlap), SPCONV_E_SHAPE (cin == 0 with outputs, n > 262140), SPCONV_E_HIP.
 */
SPCONV_API spconv_status spconv_linear(const float *x, const float *weight, const float *bias, spconv_act act, float *y,
                            int32_t n, int32_t cin, int32_t cout, void *stream);

/*
 * Global average pooling: y[n, c] = (1 / (h w)) * sum_p x[n, c, p], summed in
 * ascending p in fp32.  x [n][c][h][w], y [n][c].
 * Errors: SPCONV_E_ARG, SPCONV_E_SHAPE (h * w == 0 with n * c > 0), SPCONV_E_HIP.
 */
SPCONV_API spconv_status spconv_global_avg_pool(const float *x, float *y, int32_t n, int32_t c, int32_t h, int32_t w,
                                     void *stream);

/*
 * Dense weights to blocks of block_rows output x block_cols input channels
 * (Fig. 5: 1x4, 4x1 and 2x2 blocks), aligned (block (b, q) covers rows
 * b*kr .. b*kr + kr - 1 and channels q*kc .. q*kc + kc - 1); the layout that
 * spconv_plan_create_blocked takes.
 *
 * spconv_detect_blocks: the (kr, kc) in {1, 2, 4} x {1, 2, 4} with the most
 * weights per block (on a tie the taller, output-channel block) such that
 * kr divides cout, kc divides cin and every aligned block is all zero or all
 * nonzero.  Errors as spconv_detect_block_rows.
 *
 * spconv_dense_to_bcsr_blocked: as spconv_dense_to_bcsr with block_cols
 * (1, 2 or 4, dividing cin): a block is stored when any of its weights is
 * nonzero; col_idx[t] = its first input channel; values has capacity *
 * block_rows * block_cols entries, values[(t * kr + i) * kc + j].
 *
 * spconv_plan_create_dense_blocked: detect (block_rows = block_cols = 0) or
 * take both, convert, and plan as spconv_plan_create_blocked.
 */
SPCONV_API spconv_status spconv_detect_blocks(int32_t cout, int32_t cin, const float *dense, int32_t *block_rows,
                                              int32_t *block_cols);
SPCONV_API spconv_status spconv_dense_to_bcsr_blocked(int32_t cout, int32_t cin, const float *dense,
                                                      int32_t block_rows, int32_t block_cols, int32_t *row_ptr,
                                                      int32_t *col_idx, float *values, int64_t capacity,
                                                      int64_t *nnzb);
SPCONV_API spconv_status spconv_plan_create_dense_blocked(spconv_plan *out, int32_t cout, int32_t cin,
                                                          const float *dense, int32_t block_rows,
                                                          int32_t block_cols, const float *bias, spconv_act act,
                                                          spconv_dtype storage);

/* ---------------------------------------------------------------------------
 * Planner controls and introspection.  These let a caller (and the CPU-only
 * tests) see what the host-side planner decided without running a kernel.
 * ------------------------------------------------------------------------- */

typedef struct {
    int32_t struct_size; /* sizeof(spconv_options) */
    int32_t reorder;     /* 1 (default): process rows in descending nonzero order; 0: natural order */
    int32_t host_only;   /* 1: plan on the host only, no device memory; spconv_run refuses it */
    int32_t kernel;      /* 0 = choose automatically: the LDS-strip or direct-load kernel, or, for
                            runs with enough columns on layers where it measured faster, the
                            register-indexed kernel (spconv_plan_info.indexed_min_cols) or the
                            outer-product kernel (spconv_plan_info.outer_min_cols); fp32
                            unstructured inputs of more than 1264 channels take channel-range
                            passes (5);
                            1 = LDS-strip kernel (SPCONV_E_UNSUPPORTED when the strip of cin
                            channels does not fit in LDS); 2 = direct-load kernel; 3 =
                            register-indexed kernel (SPCONV_E_UNSUPPORTED for fp16 storage or a
                            depthwise stage); 4 = outer-product kernel on the matrix cores
                            (1 x 4 blocks, no depthwise stage, cin <= 632, else
                            SPCONV_E_UNSUPPORTED); 5 = channel-range passes for inputs too wide
                            for one LDS strip (Sec. 3.2, 4.1): the input channels in ranges of at
                            most 512, one LDS-strip launch each on the same y, every launch
                            after the first adding to the partial sums the earlier ones left in
                            y, the bias and activation applied by the last; each output is still
                            summed over all channels in ascending order (fp32 unstructured plans
                            without a depthwise stage, not static, else SPCONV_E_UNSUPPORTED) */
    int32_t group_lanes; /* 0 = choose automatically; else 4, 8 or 16 lanes per (block) row: each
                            lane accumulates 16 / group_lanes vectors of 16 bytes of the tile's
                            columns, and a wavefront works on 64 / group_lanes rows at a time
                            (SPCONV_E_UNSUPPORTED when a lane would hold more than 64 fp32
                            accumulators) */
    int32_t waves;       /* 0 = choose automatically; else the number of wavefronts per
                            workgroup, 1 to 16 */
    int32_t pipe_sets;   /* LDS-strip kernel: 0 = choose automatically; 1 or 2 bundles of rows a
                            wavefront interleaves by input channel so that it reads each tile's
                            channels in ascending order once (2 needs twice the accumulators:
                            SPCONV_E_UNSUPPORTED beyond 32 per lane) */
    int32_t regions;     /* LDS-strip kernel: 0 = choose automatically; else 1 to 4 parts of the
                            strip, each refilled with the next tile's channels as soon as every
                            wavefront is done with it */
    int32_t lane_cols;   /* register-indexed kernel: 0 = choose automatically at each run; else
                            1 to 6 columns per lane (tiles of 64 * lane_cols columns) */
} spconv_options;

/*
 * As spconv_plan_create_ex, with blocks of block_rows consecutive output
 * channels x block_cols consecutive input channels (Fig. 5: 1x4, 4x1 and 2x2
 * blocks train to the same accuracy; Sec. 3.2 names the shapes):
 *   block_cols  1, 2 or 4 (1 is spconv_plan_create_ex)
 *   col_idx     first input channel of each block; within a block row the
 *               blocks ascend and do not overlap (col_idx[t] >= col_idx[t-1] +
 *               block_cols); every block lies inside [0, cin); alignment to
 *               block_cols is not required
 *   values      row_ptr[end] * block_rows * block_cols floats:
 *               values[(t * block_rows + i) * block_cols + j] =
 *               W[rb * block_rows + i, col_idx[t] + j]
 * The planner expands each block into block_cols consecutive single-channel
 * entries of the 1 x block_rows kernels; the sum for each output stays in
 * ascending input channel, so the result equals that of the same weight
 * given unblocked.  spconv_plan_unpack returns the blocks as given.
 * Errors: as spconv_plan_create_ex; SPCONV_E_ARG (block_cols <= 0),
 * SPCONV_E_UNSUPPORTED (block_cols not 1, 2 or 4), SPCONV_E_FORMAT (a block
 * outside [0, cin) or overlapping the previous one).
 */
SPCONV_API spconv_status spconv_plan_create_blocked(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                         int32_t block_cols, const int32_t *row_ptr, const int32_t *col_idx,
                                         const float *values, const float *bias, spconv_act act,
                                         spconv_dtype storage, const spconv_options *opts);

/* Fill *opts with the defaults used by spconv_plan_create. */
SPCONV_API void spconv_options_init(spconv_options *opts);

/* As spconv_plan_create, with explicit planner options (NULL = defaults). */
SPCONV_API spconv_status spconv_plan_create_ex(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                    const int32_t *row_ptr, const int32_t *col_idx,
                                    const float *values, const float *bias, spconv_act act,
                                    spconv_dtype storage, const spconv_options *opts);

/* ---------------------------------------------------------------------------
 * Fused depthwise 3x3 -> sparse 1x1.  A MobileNet block runs a depthwise 3x3
 * convolution (one 3x3 filter per channel) right before each 1x1 (Sec. 2;
 * Sec. 3.3 lists the CHW depthwise kernels beside the sparse 1x1).  A fused
 * plan computes both in one launch, keeping the depthwise output on chip:
 *
 *     D[n, c, oy, ox] = dw_act( dw_bias[c] + sum_{dy, dx in 0..2} dw_weights[c][dy][dx]
 *                                  * X[n, c, s*oy + dy - 1, s*ox + dx - 1] )
 *     Y[n, r, p]      = act( b[r] + sum_{stored (r, c)} W[r, c] * D[n, c, p] )
 *
 * with zero padding 1 (X reads outside the image give 0) and stride s, so an
 * h x w input gives an out_h x out_w output, out_h = (h - 1) / s + 1,
 * out_w = (w - 1) / s + 1.  D is evaluated in fp32 (fma in dy, dx order, then
 * the bias, then dw_act) and is never written to memory.
 * ------------------------------------------------------------------------- */

/*
 * As spconv_plan_create_ex, with a depthwise stage in front:
 *   dw_weights  host, cin * 9 floats, [c][dy][dx]; must be finite
 *   dw_bias     host, cin floats, or NULL for zeros; must be finite
 *   dw_act      activation of the depthwise stage
 *   dw_stride   1 or 2
 *   storage     SPCONV_F32 only
 *   opts        as for spconv_plan_create_ex; the plan always uses the
 *               LDS-strip kernel with one bundle per accumulator set, so
 *               kernel = 2, pipe_sets and regions are refused
 * spconv_run on the plan takes x = the depthwise input (n x cin x h x w) and
 * writes y = n x cout x out_h x out_w.
 * Errors: as spconv_plan_create_ex; SPCONV_E_ARG (dw_stride not 1 or 2, NULL
 * dw_weights, bad dw_act), SPCONV_E_FORMAT (a non-finite depthwise weight or
 * bias), SPCONV_E_UNSUPPORTED (SPCONV_F16 storage, kernel = 2, pipe_sets or
 * regions set, or a strip of cin channels that does not fit in LDS).
 */
SPCONV_API spconv_status spconv_plan_create_fused(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                       const int32_t *row_ptr, const int32_t *col_idx,
                                       const float *values, const float *bias, spconv_act act,
                                       const float *dw_weights, const float *dw_bias, spconv_act dw_act,
                                       int32_t dw_stride, spconv_dtype storage,
                                       const spconv_options *opts);

typedef struct {
    int32_t cout, cin, block_rows;
    int32_t storage, act;
    int32_t kernel;        /* 0: LDS-strip kernel; 1: direct-load kernel for wide inputs */
    int32_t group_lanes;   /* lanes per (block) row */
    int32_t bundle_rows;   /* (block) rows a wavefront works on at a time = 64 / group_lanes */
    int32_t cols_per_lane; /* output columns each lane accumulates */
    int32_t tile_cols;     /* columns per workgroup tile (256 bytes of one channel) */
    int32_t waves;         /* wavefronts per workgroup */
    int32_t lds_bytes;     /* LDS per workgroup */
    int32_t max_parts;     /* most workgroups that may share the rows of one tile */
    int32_t pipe_sets;     /* bundles a wavefront interleaves (0: direct-load kernel or depthwise stage) */
    int32_t regions;       /* strip parts refilled independently (0: direct-load kernel or depthwise
                              stage) */
    int64_t nnzb;          /* stored blocks (of block_rows x block_cols weights) */
    int64_t slots;         /* packed (channel, weight) slots including padding */
    int64_t max_wave_cost; /* largest per-wavefront work estimate (slots + epilogue) */
    int64_t sum_wave_cost; /* total of the per-wavefront work estimates */
    int64_t device_bytes;  /* device memory the plan holds */
    int32_t dw_stride;     /* fused depthwise stage: 0 none, else its stride */
    int32_t dw_act;        /* its activation */
    int32_t block_cols;    /* input channels per block (1 unless created by spconv_plan_create_blocked) */
    int32_t split_rows;    /* LDS-strip and direct-load kernels: rows more than twice the median length
                              (at least 32 nonzeros) packed as two pieces, their even and their odd
                              nonzeros, in neighbouring lane groups whose partial sums are added before
                              the epilogue (unstructured plans; such a row is summed as its two pieces
                              rather than in one ascending pass) */
    int64_t indexed_min_cols; /* kernel chosen automatically: runs of at least this many output columns
                                 (N * out_h * out_w) take the register-indexed kernel; 0 = never (and
                                 for host-only plans, which know no device) */
    int64_t outer_min_cols;   /* the same for the outer-product kernel, which takes precedence */
    int64_t channel_passes;   /* kernel option 5: the number of channel-range passes a run launches
                                 (0 for other plans) */
} spconv_plan_info;

/* Describe a plan.  Host only; does not touch the device. */
SPCONV_API spconv_status spconv_plan_get_info(spconv_plan plan, spconv_plan_info *info);

/*
 * Reconstruct the plan's weights from its packed host image, in the input's
 * block-CSR form: row_ptr[cout/k + 1], col_idx[nnzb], values[nnzb * k] (each
 * may be NULL to skip), and perm[cout/k] (may be NULL): perm[i] = the block
 * row processed i-th.  Host only.  Lets tests check that packing loses nothing.
 */
SPCONV_API spconv_status spconv_plan_unpack(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx, float *values,
                                 int32_t *perm);

/*
 * The same reconstruction from the interleaved weight streams the pipelined
 * LDS-strip kernel reads (row_ptr, col_idx, values as above, each may be
 * NULL), walking them with the kernel's own bookkeeping: per step, the
 * accumulator set and last-step bits pick the bundle, and every strip channel
 * read must fall between the need and release events of its strip part.
 * Host only.  SPCONV_E_FORMAT (message set) when the streams are inconsistent
 * or the plan has none (direct-load kernel, depthwise stage).
 */
SPCONV_API spconv_status spconv_plan_unpack_interleaved(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx,
                                             float *values);

/*
 * The same reconstruction from the register-indexed kernel's streams: with
 * from_pairs = 0 from the slot records (walking each slot's chunk table,
 * batch flags and ring offsets as the kernel does), with from_pairs = 1 from
 * the row-pair entries that cover the columns left after the whole tiles.
 * row_ptr, col_idx, values as for spconv_plan_unpack (each may be NULL).
 * Host only.  SPCONV_E_FORMAT (message set) when a stream is inconsistent or
 * the plan has none (fp16 storage, depthwise stage).
 */
SPCONV_API spconv_status spconv_plan_unpack_indexed(spconv_plan plan, int32_t from_pairs, int32_t *row_ptr,
                                                    int32_t *col_idx, float *values);

/*
 * The same reconstruction from the outer-product kernel's records (Sec. 3.2:
 * 1 x 4 output-channel blocks; the octs of 8 block rows in lockstep, their
 * records of (weight, LDS channel offset) per lane slot and step, the zero-row
 * padding, and the per-tile-parity wave lists, all checked as the kernel
 * walks them).  row_ptr, col_idx, values as for spconv_plan_unpack (each may
 * be NULL).  Host only.  SPCONV_E_FORMAT (message set) when the records are
 * inconsistent or the plan has none (not 1 x 4 blocks, depthwise stage,
 * cin above 632).
 */
SPCONV_API spconv_status spconv_plan_unpack_outer(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx,
                                                  float *values);

/*
 * For callers that cannot allocate device memory (code that must not call
 * hipMalloc: tight serving loops, harnesses that forbid it).  As
 * spconv_plan_create_ex, but the plan's device image (packed weights, tables
 * and error word) goes into a static device array of SPCONV_STATIC_PLAN_BYTES
 * that the library holds on each GPU it runs on until the process ends,
 * instead of a new allocation; no hipMalloc or hipFree is called, only one
 * synchronous host-to-device copy.  The array is shared: each call on a
 * device overwrites it, so only the plan created last on that device can run
 * (spconv_run refuses an earlier one with SPCONV_E_ARG), and creating such a
 * plan while a run of the previous one is still executing, or from two threads
 * on one device at once, races.  spconv_destroy frees only the plan's host
 * part.  Errors: SPCONV_E_SHAPE when the image is larger than the array (the
 * message gives both sizes; checked before any HIP call), SPCONV_E_ARG for
 * options.host_only = 1, otherwise as spconv_plan_create_ex.
 */
#define SPCONV_STATIC_PLAN_BYTES (32u << 20)
SPCONV_API spconv_status spconv_plan_create_static(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                                   const int32_t *row_ptr, const int32_t *col_idx,
                                                   const float *values, const float *bias, spconv_act act,
                                                   spconv_dtype storage, const spconv_options *opts);

/*
 * The plan's device error word, written by its kernels: bit 0
 * (SPCONV_FLAG_WAIT_GAVE_UP) is set when a bounded wait inside a kernel on an
 * on-chip counter (a strip or ring part landing, a share being issued) ran
 * out; that wavefront went on without the data, so the output of that launch
 * is not to be trusted.  Waits for all work queued on the plan's device to
 * finish, then reads the word into *flags; with clear != 0 resets it to zero.
 * SPCONV_E_ARG for a NULL argument or a host-only plan, SPCONV_E_HIP when a
 * HIP call fails (message set).
 */
#define SPCONV_FLAG_WAIT_GAVE_UP 1
SPCONV_API spconv_status spconv_plan_check(spconv_plan plan, int32_t *flags, int32_t clear);

/*
 * Test hook for the error path above: the bound of every such wait in the
 * plan's later launches, in sleeps of about 64 clocks (default 1 << 22, about
 * 0.1 s).  0 makes every wait that finds its data missing give up at once;
 * kernels still run to completion.  The one setting a plan has that can
 * change: not to be called while another thread queues runs of the plan.
 * SPCONV_E_ARG for a NULL plan or a negative bound.  Host only.
 */
SPCONV_API spconv_status spconv_plan_set_wait_limit(spconv_plan plan, int32_t sleeps);

#ifdef __cplusplus
}
#endif

#endif /* SPCONV_H */
