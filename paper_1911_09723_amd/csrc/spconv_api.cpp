// C ABI of libspconv (declared in include/spconv.h).
//
// spconv_plan_create: validate + plan on the host (planner.cpp), then one
// device allocation holding every packed array, filled with one synchronous
// copy.  spconv_run: argument checks, then one asynchronous kernel launch on
// the caller's stream (spmm_kernels.hip); it allocates nothing and never
// synchronizes.
#include "spconv.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <new>
#include <mutex>
#include <string>
#include <vector>

#include "launch.hpp"
#include "net_kernels.hpp"
#include "planner.hpp"

struct spconv_plan_s {
    spconv::PackedPlan host;
    spconv::DevicePlan dev;
    int device = -1;
    void *dmem = nullptr;
    size_t dbytes = 0;
    bool host_only = false;
    uint64_t static_gen = 0;  // plans in the static device array: the generation they wrote (0: not one)
    // channel-range passes (kernel option 5): one plan per range of input
    // channels starting at pass_c0[i], run in order; empty for other plans
    std::vector<spconv_plan_s *> passes;
    std::vector<int32_t> pass_c0;
};

namespace {

thread_local std::string g_err;

constexpr int32_t kKernelPasses = 5;    // kernel option: channel-range passes
constexpr int32_t kPassChannels = 512;  // most input channels per pass (its LDS strip fits)

// The static device array of spconv_plan_create_static: one per GPU (each
// device holds its own copy of this file-scope array), found once per device
// with hipGetSymbolAddress; host code uses only that address.  Each creation
// on a device bumps the device's generation; runs of a plan whose generation
// is no longer the device's are refused.
constexpr size_t kStaticPlanBytes = size_t(32) << 20;
static_assert(kStaticPlanBytes == SPCONV_STATIC_PLAN_BYTES, "header and library agree on the array's size");
__device__ __align__(256) unsigned char scratch[kStaticPlanBytes];

struct StaticArray {
    void *ptr = nullptr;  // device address of scratch on this device
    uint64_t gen = 0;     // generation of the plan whose image it holds
};
constexpr int kMaxStaticDevices = 64;
std::mutex g_static_mu;
StaticArray g_static[kMaxStaticDevices];

spconv_status fail(spconv_status st, const std::string &msg) {
    g_err = msg;
    return st;
}

spconv_status hip_fail(const char *what, hipError_t e) {
    g_err = std::string(what) + " failed: " + hipGetErrorName(e) + " (" + hipGetErrorString(e) + ")";
    return SPCONV_E_HIP;
}

// Test hook: SPCONV_FAULT=alloc makes the device allocation in plan creation
// report failure, to exercise the no-leak error path.
bool fault_alloc() {
    const char *f = std::getenv("SPCONV_FAULT");
    return f && std::strcmp(f, "alloc") == 0;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

spconv::Input make_input(int32_t cout, int32_t cin, int32_t block_rows, const int32_t *row_ptr,
                         const int32_t *col_idx, const float *values, const float *bias, spconv_act act,
                         spconv_dtype storage) {
    spconv::Input in;
    in.cout = cout;
    in.cin = cin;
    in.block_rows = block_rows;
    in.row_ptr = row_ptr;
    in.col_idx = col_idx;
    in.values = values;
    in.bias = bias;
    in.act = static_cast<int32_t>(act);
    in.storage = static_cast<int32_t>(storage);
    return in;
}

// Pack the plan's device image and copy it to the device: into a new
// allocation, or (use_static) into the device's static array, which needs no
// allocation.
spconv_status upload(spconv_plan_s *pl, bool use_static) {
    const spconv::PackedPlan &h = pl->host;
    // bundle table: rows, then the biases of those rows as fp32 bit patterns
    std::vector<int32_t> table(static_cast<size_t>(h.table_words()));
    std::copy(h.rows.begin(), h.rows.end(), table.begin());
    if (!h.bundle_bias.empty())
        std::memcpy(table.data() + h.rows.size(), h.bundle_bias.data(), h.bundle_bias.size() * sizeof(float));
    struct Part {
        const void *src;
        size_t bytes;
        size_t off;
    } parts[26] = {
        {h.idx.data(), h.idx.size() * sizeof(int32_t), 0},
        {h.val.data(), h.val.size() * sizeof(float), 0},
        {h.hdr.data(), h.hdr.size() * sizeof(int32_t), 0},
        {table.data(), table.size() * sizeof(int32_t), 0},
        {h.rank.data(), h.rank.size() * sizeof(int32_t), 0},
        {h.wave_ptr.data(), h.wave_ptr.size() * sizeof(int32_t), 0},
        {h.pidx.data(), h.pidx.size() * sizeof(int32_t), 0},
        {h.pval.data(), h.pval.size() * sizeof(float), 0},
        {h.psel.data(), h.psel.size() * sizeof(uint32_t), 0},
        {h.sel_ptr.data(), h.sel_ptr.size() * sizeof(int32_t), 0},
        {h.wave_ev.data(), h.wave_ev.size() * sizeof(int32_t), 0},
        {h.dw.data(), h.dw.size() * sizeof(float), 0},
        {h.rrec.data(), h.rrec.size() * sizeof(uint32_t), 0},
        {h.rslot_batch.data(), h.rslot_batch.size() * sizeof(int32_t), 0},
        {h.rslot_chunk.data(), h.rslot_chunk.size() * sizeof(int32_t), 0},
        {h.rslot_rows.data(), h.rslot_rows.size() * sizeof(int32_t), 0},
        {h.rslot_bias.data(), h.rslot_bias.size() * sizeof(float), 0},
        {h.rpair_ptr.data(), h.rpair_ptr.size() * sizeof(int32_t), 0},
        {h.rpair_ent.data(), h.rpair_ent.size() * sizeof(uint32_t), 0},
        {h.rrow_bias.data(), h.rrow_bias.size() * sizeof(float), 0},
        {nullptr, 0, 0},  // the error flag word (zeroed)
        {h.orec.data(), h.orec.size() * sizeof(uint32_t), 0},
        {h.ooct_tab.data(), h.ooct_tab.size() * sizeof(int32_t), 0},
        {h.owave_ptr.data(), h.owave_ptr.size() * sizeof(int32_t), 0},
        {h.owave_oct.data(), h.owave_oct.size() * sizeof(int32_t), 0},
        {h.ooff.data(), h.ooff.size() * sizeof(uint32_t), 0},
    };
    size_t total = 0;
    for (Part &p : parts) {
        p.off = total;
        total = align_up(total + std::max<size_t>(p.bytes, 16), 256);
    }
    if (use_static && total > kStaticPlanBytes)  // before any HIP call
        return fail(SPCONV_E_SHAPE, "the plan's device image needs " + std::to_string(total) +
                                        " bytes; the static array holds " + std::to_string(kStaticPlanBytes));
    if (!use_static && fault_alloc())
        return fail(SPCONV_E_NOMEM, "device allocation failed (SPCONV_FAULT=alloc)");
    hipError_t e = hipGetDevice(&pl->device);
    if (e != hipSuccess)
        return hip_fail("hipGetDevice", e);
    void *dest = nullptr;
    if (use_static) {
        if (pl->device < 0 || pl->device >= kMaxStaticDevices)
            return fail(SPCONV_E_UNSUPPORTED, "device " + std::to_string(pl->device) + " is beyond the static arrays");
        std::lock_guard<std::mutex> lock(g_static_mu);
        StaticArray &sa = g_static[pl->device];
        if (!sa.ptr) {
            // once per device, with it current: the device address of its copy of the array
            void *ptr = nullptr;
            e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
            if (e != hipSuccess)
                return hip_fail("hipGetSymbolAddress (static plan array)", e);
            sa.ptr = ptr;
        }
        dest = sa.ptr;
        pl->static_gen = ++sa.gen;
    } else {
        e = hipMalloc(&pl->dmem, total);
        if (e == hipErrorOutOfMemory) {
            pl->dmem = nullptr;
            return fail(SPCONV_E_NOMEM, "hipMalloc of " + std::to_string(total) + " bytes: out of memory");
        }
        if (e != hipSuccess) {
            pl->dmem = nullptr;
            return hip_fail("hipMalloc", e);
        }
        dest = pl->dmem;
    }
    pl->dbytes = total;
    std::string image(total, '\0');  // the error word (and every padding byte) starts at zero
    for (const Part &p : parts)
        if (p.bytes)
            std::memcpy(&image[p.off], p.src, p.bytes);
    e = hipMemcpy(dest, image.data(), total, hipMemcpyHostToDevice);
    if (e != hipSuccess)
        return hip_fail("hipMemcpy (plan upload)", e);
    char *base = static_cast<char *>(dest);
    spconv::DevicePlan &d = pl->dev;
    d.idx = reinterpret_cast<const int32_t *>(base + parts[0].off);
    d.val = reinterpret_cast<const float *>(base + parts[1].off);
    d.hdr = reinterpret_cast<const int32_t *>(base + parts[2].off);
    d.table = reinterpret_cast<const int32_t *>(base + parts[3].off);
    d.rank = reinterpret_cast<const int32_t *>(base + parts[4].off);
    d.wave_ptr = reinterpret_cast<const int32_t *>(base + parts[5].off);
    d.pidx = reinterpret_cast<const int32_t *>(base + parts[6].off);
    d.pval = reinterpret_cast<const float *>(base + parts[7].off);
    d.psel = reinterpret_cast<const uint32_t *>(base + parts[8].off);
    d.sel_ptr = reinterpret_cast<const int32_t *>(base + parts[9].off);
    d.wave_ev = reinterpret_cast<const int32_t *>(base + parts[10].off);
    d.dw = reinterpret_cast<const float *>(base + parts[11].off);
    d.rrec = reinterpret_cast<const uint32_t *>(base + parts[12].off);
    d.rslot_batch = reinterpret_cast<const int32_t *>(base + parts[13].off);
    d.rslot_chunk = reinterpret_cast<const int32_t *>(base + parts[14].off);
    d.rslot_rows = reinterpret_cast<const int32_t *>(base + parts[15].off);
    d.rslot_bias = reinterpret_cast<const float *>(base + parts[16].off);
    d.rpair_ptr = reinterpret_cast<const int32_t *>(base + parts[17].off);
    d.rpair_ent = reinterpret_cast<const uint32_t *>(base + parts[18].off);
    d.rpair_ent_words = static_cast<int64_t>(h.rpair_ent.size());
    d.rrow_bias = reinterpret_cast<const float *>(base + parts[19].off);
    d.flag = reinterpret_cast<int32_t *>(base + parts[20].off);
    d.orec = reinterpret_cast<const uint32_t *>(base + parts[21].off);
    d.ooct = reinterpret_cast<const int32_t *>(base + parts[22].off);
    d.owave_ptr = reinterpret_cast<const int32_t *>(base + parts[23].off);
    d.owave_oct = reinterpret_cast<const int32_t *>(base + parts[24].off);
    d.ooff = reinterpret_cast<const uint32_t *>(base + parts[25].off);
    return SPCONV_OK;
}

// The automatic kernel choice between the LDS-strip / direct-load kernels and
// the register-indexed one, from their measured times on MI355X over the
// workload layers: the register-indexed kernel wins where the direct-load
// kernel would run (inputs too wide for an LDS strip) and, once a run has at
// least one whole round of its 384-column tiles, on layers with few input
// channels or denser weights; elsewhere (small batches, few output channels,
// 90-95% sparse wide layers) the strip kernels are faster.
int64_t indexed_min_cols(const spconv::PackedPlan &h, const spconv::DevicePlan &d) {
    if (!h.auto_kernel || d.rslots == 0 || d.num_cus <= 0)
        return 0;
    if (h.kernel == spconv::KERNEL_DIRECT)
        return 1024;
    const double density = static_cast<double>(h.nnzb) * h.k / (static_cast<double>(h.cout) * h.cin);
    if (d.rslots >= 4 && (h.cin <= 64 || density >= 0.15))
        return int64_t(64) * 6 * ((d.num_cus + d.rgroups - 1) / d.rgroups);
    return 0;
}

// The automatic choice of the lockstep kernel, from its measured times on
// MI355X over the workload layers.  Matrix mode (1 x 4 blocks): it wins at
// every batch measured (runs with fewer tiles than compute units share each
// tile among workgroups by set) when the sets average at least two quads (8
// steps); with shorter rows (few input channels) its per-tile costs
// dominate.  Vector mode (unstructured): it wins only on inputs too wide for
// an LDS strip (where the others read X from L2 per nonzero).
int64_t outer_min_cols(const spconv::PackedPlan &h, const spconv::DevicePlan &d) {
    if (!h.auto_kernel || d.oocts == 0 || d.num_cus <= 0)
        return 0;
    if (h.omode == 1)
        return h.kernel == spconv::KERNEL_DIRECT ? 1 : 0;
    int64_t quads = 0;
    for (int32_t o = 0; o < h.oocts; ++o)
        quads += h.ooct_tab[static_cast<size_t>(o) * spconv::kOctWords + 1];
    return quads >= 2 * static_cast<int64_t>(h.oocts) ? 1 : 0;
}

void fill_device_geometry(spconv_plan_s *pl) {
    const spconv::PackedPlan &h = pl->host;
    spconv::DevicePlan &d = pl->dev;
    d.kernel = h.kernel;
    d.group_lanes = h.group_lanes;
    d.tile_cols = h.tile_cols;
    d.waves = h.waves;
    d.lds_bytes = h.lds_bytes;
    d.k = h.k;
    d.storage = h.storage;
    d.act = h.act;
    d.cin = h.cin;
    d.cout = h.cout;
    d.strip_rows = h.strip_rows;
    d.pipe_sets = h.pipe_sets;
    d.regions = h.regions;
    d.region_rows = h.region_rows;
    d.busy_waves = h.busy_waves;
    d.idx_bytes = static_cast<int32_t>(h.idx.size() * sizeof(int32_t));
    d.val_bytes = static_cast<int32_t>(h.val.size() * sizeof(float));
    d.nbundles = h.nbundles();
    d.splits = h.split_rows > 0 ? 1 : 0;
    d.max_parts = h.max_parts;
    d.dw_stride = h.dw_stride;
    d.dw_act = h.dw_act;
    d.stage_off = h.stage_off;
    d.stage_bytes = h.stage_bytes;
    d.use_indexed = h.use_indexed;
    d.rslots = h.rslots;
    d.rgroups = h.rgroups;
    d.rwaves = h.rwaves;
    d.rnch = h.rnch;
    d.rlane_cols = h.rlane_cols;
    d.use_outer = h.use_outer;
    d.omode = h.omode;
    d.otw = h.otw;
    d.oocts = h.oocts;
    d.owaves = h.owaves;
    d.ozrow = h.ozrow;
    d.ooff_bytes = static_cast<int32_t>(h.ooff.size() * sizeof(uint32_t));
}

bool ranges_overlap(const void *a, size_t abytes, const void *b, size_t bbytes) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// Plan creation shared by every entry point: options, planning, upload.
spconv_status create_passes(spconv_plan_s *pl, const spconv::Input &in, const spconv_options &o);

// Free a plan, its passes and its device image without touching the error
// message (create_plan's failure paths keep theirs); the first HIP error.
hipError_t free_plan(spconv_plan_s *pl) {
    hipError_t st = hipSuccess;
    for (spconv_plan_s *q : pl->passes) {
        const hipError_t e = free_plan(q);
        if (st == hipSuccess)
            st = e;
    }
    if (pl->dmem) {
        const hipError_t e = hipFree(pl->dmem);
        if (st == hipSuccess)
            st = e;
    }
    delete pl;
    return st;
}

// xc, accum: set for the passes of a channel-range plan (see create_passes)
spconv_status create_plan(spconv_plan *out, const spconv::Input &in, const spconv_options *opts,
                          bool use_static = false, int32_t xc = 0, int32_t accum = 0) {
    if (!out)
        return fail(SPCONV_E_ARG, "out is NULL");
    *out = nullptr;
    spconv_options o;
    spconv_options_init(&o);
    if (opts) {
        if (opts->struct_size != static_cast<int32_t>(sizeof(spconv_options)))
            return fail(SPCONV_E_ARG, "spconv_options.struct_size does not match this library");
        o = *opts;
    }
    if (o.host_only != 0 && o.host_only != 1)
        return fail(SPCONV_E_ARG, "host_only must be 0 or 1");
    if (use_static && o.host_only)
        return fail(SPCONV_E_ARG, "a plan in the static device array cannot be host-only");
    spconv::Options po;
    po.reorder = o.reorder;
    po.host_only = o.host_only;
    po.kernel = o.kernel;
    po.group_lanes = o.group_lanes;
    po.waves = o.waves;
    po.pipe_sets = o.pipe_sets;
    po.regions = o.regions;
    po.lane_cols = o.lane_cols;
    po.split = xc == 0 && accum == 0 ? 1 : 0;  // a pass's rows are summed in one ascending pass
    // automatic choice: fp32 unstructured inputs too wide for the lockstep
    // kernel's strips (measured: passes over the LDS-strip kernel beat the
    // direct-load kernel there, 124 against 197 us for 1280 -> 320 @ 7x7,
    // batch 128; below that width the lockstep kernel is faster)
    const bool auto_passes = o.kernel == 0 && in.cin > spconv::kOuterMaxCin16 && in.block_rows == 1 &&
                             in.block_cols <= 1 && in.storage == 0 && !in.dw_stride && !use_static && xc == 0;
    const bool passes = o.kernel == kKernelPasses || auto_passes;
    if (passes) {
        if (in.block_rows != 1 || in.block_cols > 1 || in.storage != 0 || in.dw_stride || use_static) {
            *out = nullptr;
            return fail(SPCONV_E_UNSUPPORTED, "channel-range passes (kernel 5) run fp32 unstructured plans without "
                                              "a depthwise stage, not in the static device array");
        }
        po.kernel = 0;  // the plan itself: the automatic choice (its image serves unpacking and info)
    }

    spconv_plan_s *pl = new (std::nothrow) spconv_plan_s();
    if (!pl)
        return fail(SPCONV_E_NOMEM, "host allocation of the plan failed");
    std::string err;
    spconv::Status st;
    try {
        st = spconv::build_plan(in, po, pl->host, err);
    } catch (const std::bad_alloc &) {
        delete pl;
        return fail(SPCONV_E_NOMEM, "host allocation failed while packing the plan");
    }
    if (st != spconv::OK) {
        delete pl;
        return fail(static_cast<spconv_status>(st), err);
    }
    fill_device_geometry(pl);
    pl->dev.xc = xc;
    pl->dev.accum = accum;
    pl->host_only = o.host_only == 1;
    if (!pl->host_only) {
        spconv_status us = upload(pl, use_static);
        if (us == SPCONV_OK) {
            hipError_t pe = spconv::prepare_launch(pl->dev);
            if (pe == hipSuccess && pl->dev.rslots > 0)
                pe = spconv::prepare_indexed(pl->dev);
            if (pe == hipSuccess && pl->dev.oocts > 0)
                pe = spconv::prepare_outer(pl->dev);
            pl->dev.indexed_min_cols = indexed_min_cols(pl->host, pl->dev);
            pl->dev.outer_min_cols = outer_min_cols(pl->host, pl->dev);
            if (pe != hipSuccess)
                us = hip_fail("kernel launch set-up", pe);
        }
        if (us != SPCONV_OK) {
            (void)free_plan(pl);
            return us;
        }
    }
    if (passes) {
        const spconv_status us = create_passes(pl, in, o);
        if (us != SPCONV_OK) {
            (void)free_plan(pl);
            return us;
        }
    }
    *out = pl;
    return SPCONV_OK;
}

// Kernel option 5: the input channels in ranges of at most kPassChannels
// (equal sizes, multiples of 4), each a plan of the LDS-strip kernel over its
// columns of W (shifted to start at 0) that reads X with the full input's
// image stride.  The passes run in order on the same Y: every pass after the
// first starts each row's accumulators from Y (the sums over the earlier
// ranges), so each output is summed over all channels in ascending order from
// zero, as in the other kernels; only the last adds the bias and applies the
// activation.  The passes share the plan's error word.
spconv_status create_passes(spconv_plan_s *pl, const spconv::Input &in, const spconv_options &o) {
    const int32_t np = (in.cin + kPassChannels - 1) / kPassChannels;
    const int32_t per = ((in.cin + np - 1) / np + 3) & ~3;
    for (int32_t c0 = 0; c0 < in.cin; c0 += per) {
        const int32_t c1 = std::min(in.cin, c0 + per);
        const bool last = c1 == in.cin;
        std::vector<int32_t> rp(static_cast<size_t>(in.cout) + 1, 0), ci;
        std::vector<float> va;
        for (int32_t r = 0; r < in.cout; ++r) {
            for (int32_t t = in.row_ptr[r]; t < in.row_ptr[r + 1]; ++t) {
                if (in.col_idx[t] >= c0 && in.col_idx[t] < c1) {
                    ci.push_back(in.col_idx[t] - c0);
                    va.push_back(in.values[t]);
                }
            }
            rp[static_cast<size_t>(r) + 1] = static_cast<int32_t>(ci.size());
        }
        spconv::Input sub = in;
        sub.cin = c1 - c0;
        sub.row_ptr = rp.data();
        sub.col_idx = ci.data();
        sub.values = va.data();
        sub.bias = last ? in.bias : nullptr;
        sub.act = last ? in.act : static_cast<int32_t>(SPCONV_ACT_NONE);
        spconv_options so = o;
        so.kernel = 1;  // the LDS-strip kernel
        spconv_plan q = nullptr;
        const spconv_status st = create_plan(&q, sub, &so, false, in.cin, c0 > 0 ? 1 : 0);
        if (st != SPCONV_OK)
            return st;
        q->dev.flag = pl->dev.flag;
        q->dev.spin_limit = pl->dev.spin_limit;
        pl->passes.push_back(q);
        pl->pass_c0.push_back(c0);
    }
    return SPCONV_OK;
}

}  // namespace

extern "C" {

void spconv_options_init(spconv_options *opts) {
    if (!opts)
        return;
    std::memset(opts, 0, sizeof(*opts));
    opts->struct_size = static_cast<int32_t>(sizeof(spconv_options));
    opts->reorder = 1;
}

spconv_status spconv_plan_create_ex(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                    const int32_t *row_ptr, const int32_t *col_idx, const float *values,
                                    const float *bias, spconv_act act, spconv_dtype storage,
                                    const spconv_options *opts) {
    g_err.clear();
    return create_plan(out, make_input(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage), opts);
}

spconv_status spconv_plan_create_static(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                        const int32_t *row_ptr, const int32_t *col_idx, const float *values,
                                        const float *bias, spconv_act act, spconv_dtype storage,
                                        const spconv_options *opts) {
    g_err.clear();
    return create_plan(out, make_input(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage), opts,
                       true);
}

spconv_status spconv_plan_create_fused(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                       const int32_t *row_ptr, const int32_t *col_idx, const float *values,
                                       const float *bias, spconv_act act, const float *dw_weights,
                                       const float *dw_bias, spconv_act dw_act, int32_t dw_stride,
                                       spconv_dtype storage, const spconv_options *opts) {
    g_err.clear();
    spconv::Input in = make_input(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage);
    if (dw_stride != 1 && dw_stride != 2) {
        if (out)
            *out = nullptr;
        return fail(SPCONV_E_ARG, "dw_stride must be 1 or 2 (got " + std::to_string(dw_stride) + ")");
    }
    in.dw_stride = dw_stride;
    in.dw_weights = dw_weights;
    in.dw_bias = dw_bias;
    in.dw_act = static_cast<int32_t>(dw_act);
    return create_plan(out, in, opts);
}

spconv_status spconv_plan_create_blocked(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                         int32_t block_cols, const int32_t *row_ptr, const int32_t *col_idx,
                                         const float *values, const float *bias, spconv_act act,
                                         spconv_dtype storage, const spconv_options *opts) {
    g_err.clear();
    spconv::Input in = make_input(cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage);
    in.block_cols = block_cols;
    return create_plan(out, in, opts);
}

spconv_status spconv_plan_create(spconv_plan *out, int32_t cout, int32_t cin, int32_t block_rows,
                                 const int32_t *row_ptr, const int32_t *col_idx, const float *values,
                                 const float *bias, spconv_act act, spconv_dtype storage) {
    return spconv_plan_create_ex(out, cout, cin, block_rows, row_ptr, col_idx, values, bias, act, storage,
                                 nullptr);
}

spconv_status spconv_detect_block_rows(int32_t cout, int32_t cin, const float *dense, int32_t *block_rows) {
    g_err.clear();
    if (!block_rows)
        return fail(SPCONV_E_ARG, "block_rows is NULL");
    std::string err;
    int32_t k = 1;
    const spconv::Status st = spconv::detect_block_rows(cout, cin, dense, k, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    *block_rows = k;
    return SPCONV_OK;
}

spconv_status spconv_dense_to_bcsr(int32_t cout, int32_t cin, const float *dense, int32_t block_rows,
                                   int32_t *row_ptr, int32_t *col_idx, float *values, int64_t capacity,
                                   int64_t *nnzb) {
    g_err.clear();
    if (!nnzb)
        return fail(SPCONV_E_ARG, "nnzb is NULL");
    std::string err;
    int64_t n = 0;
    const spconv::Status st =
        spconv::dense_to_bcsr(cout, cin, dense, block_rows, row_ptr, col_idx, values, capacity, n, err);
    *nnzb = n;
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    return SPCONV_OK;
}

spconv_status spconv_detect_blocks(int32_t cout, int32_t cin, const float *dense, int32_t *block_rows,
                                   int32_t *block_cols) {
    g_err.clear();
    if (!block_rows || !block_cols)
        return fail(SPCONV_E_ARG, "block_rows or block_cols is NULL");
    std::string err;
    int32_t kr = 1, kc = 1;
    const spconv::Status st = spconv::detect_blocks(cout, cin, dense, kr, kc, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    *block_rows = kr;
    *block_cols = kc;
    return SPCONV_OK;
}

spconv_status spconv_dense_to_bcsr_blocked(int32_t cout, int32_t cin, const float *dense, int32_t block_rows,
                                           int32_t block_cols, int32_t *row_ptr, int32_t *col_idx, float *values,
                                           int64_t capacity, int64_t *nnzb) {
    g_err.clear();
    if (!nnzb)
        return fail(SPCONV_E_ARG, "nnzb is NULL");
    std::string err;
    int64_t n = 0;
    const spconv::Status st = spconv::dense_to_blocks(cout, cin, dense, block_rows, block_cols, row_ptr, col_idx,
                                                      values, capacity, n, err);
    *nnzb = n;
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    return SPCONV_OK;
}

spconv_status spconv_plan_create_dense_blocked(spconv_plan *out, int32_t cout, int32_t cin, const float *dense,
                                               int32_t block_rows, int32_t block_cols, const float *bias,
                                               spconv_act act, spconv_dtype storage) {
    g_err.clear();
    if (!out)
        return fail(SPCONV_E_ARG, "out is NULL");
    *out = nullptr;
    if ((block_rows == 0) != (block_cols == 0))
        return fail(SPCONV_E_ARG, "block_rows and block_cols must both be 0 (detect) or both be given");
    std::string err;
    int32_t kr = block_rows, kc = block_cols;
    spconv::Status st = spconv::OK;
    if (kr == 0)
        st = spconv::detect_blocks(cout, cin, dense, kr, kc, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    int64_t nnzb = 0;
    st = spconv::dense_to_blocks(cout, cin, dense, kr, kc, nullptr, nullptr, nullptr, 0, nnzb, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    std::vector<int32_t> row_ptr, col_idx;
    std::vector<float> values;
    try {
        row_ptr.resize(static_cast<size_t>(cout / kr) + 1);
        col_idx.resize(static_cast<size_t>(std::max<int64_t>(nnzb, 1)));
        values.resize(static_cast<size_t>(std::max<int64_t>(nnzb, 1) * kr * kc));
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while converting the dense weight");
    }
    st = spconv::dense_to_blocks(cout, cin, dense, kr, kc, row_ptr.data(), col_idx.data(), values.data(), nnzb,
                                 nnzb, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    return spconv_plan_create_blocked(out, cout, cin, kr, kc, row_ptr.data(), col_idx.data(), values.data(), bias,
                                      act, storage, nullptr);
}

spconv_status spconv_plan_create_dense(spconv_plan *out, int32_t cout, int32_t cin, const float *dense,
                                       int32_t block_rows, const float *bias, spconv_act act,
                                       spconv_dtype storage) {
    g_err.clear();
    if (!out)
        return fail(SPCONV_E_ARG, "out is NULL");
    *out = nullptr;
    std::string err;
    int32_t k = block_rows;
    spconv::Status st = spconv::OK;
    if (k == 0)
        st = spconv::detect_block_rows(cout, cin, dense, k, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    int64_t nnzb = 0;
    st = spconv::dense_to_bcsr(cout, cin, dense, k, nullptr, nullptr, nullptr, 0, nnzb, err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    std::vector<int32_t> row_ptr, col_idx;
    std::vector<float> values;
    try {
        row_ptr.resize(static_cast<size_t>(cout / k) + 1);
        col_idx.resize(static_cast<size_t>(std::max<int64_t>(nnzb, 1)));
        values.resize(static_cast<size_t>(std::max<int64_t>(nnzb, 1) * k));
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while converting the dense weight");
    }
    st = spconv::dense_to_bcsr(cout, cin, dense, k, row_ptr.data(), col_idx.data(), values.data(), nnzb, nnzb,
                               err);
    if (st != spconv::OK)
        return fail(static_cast<spconv_status>(st), err);
    return spconv_plan_create(out, cout, cin, k, row_ptr.data(), col_idx.data(), values.data(), bias, act,
                              storage);
}

spconv_status spconv_run(spconv_plan plan, const void *x, void *y, int32_t n, int32_t h, int32_t w,
                         void *stream) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    if (n < 0 || h < 0 || w < 0)
        return fail(SPCONV_E_ARG, "n, h and w must be >= 0");
    // every check below up to the host-only refusal is on the arguments alone
    // (no HIP call), so host-only plans exercise them too
    const char *host_only_msg = "plan was created with host_only = 1 and has no device data";
    const spconv::PackedPlan &p = plan->host;
    // a depthwise stage maps the h x w input to out_h x out_w (zero padding 1)
    const int32_t s = p.dw_stride ? p.dw_stride : 1;
    const int64_t oh = p.dw_stride ? (h > 0 ? (h - 1) / s + 1 : 0) : h;
    const int64_t ow = p.dw_stride ? (w > 0 ? (w - 1) / s + 1 : 0) : w;
    const int64_t hw = oh * ow, ihw = static_cast<int64_t>(h) * w;
    const int64_t m = static_cast<int64_t>(n) * hw;
    if (m == 0)
        return plan->host_only ? fail(SPCONV_E_ARG, host_only_msg) : SPCONV_OK;
    if (!x || !y)
        return fail(SPCONV_E_ARG, "x or y is NULL");
    if (ihw > INT32_MAX || static_cast<int64_t>(n) * ihw > INT32_MAX)
        return fail(SPCONV_E_SHAPE, "n * h * w must be below 2^31 columns");
    const size_t e = p.storage == 1 ? 2 : 4;
    const int64_t xel = static_cast<int64_t>(n) * ihw * p.cin, yel = m * p.cout;
    if (xel > (int64_t(1) << 62) / 4 || yel > (int64_t(1) << 62) / 4)
        return fail(SPCONV_E_SHAPE, "tensor too large");
    if (reinterpret_cast<uintptr_t>(x) % e || reinterpret_cast<uintptr_t>(y) % e)
        return fail(SPCONV_E_ARG, "x and y must be aligned to the element size");
    if (ranges_overlap(x, static_cast<size_t>(xel) * e, y, static_cast<size_t>(yel) * e))
        return fail(SPCONV_E_ARG, "x and y overlap; the operation cannot run in place");
    // the kernels address X and Y relative to the first image of a tile with
    // 32-bit byte offsets: the images one tile's columns touch (at most
    // (tile_cols - 1) / hw + 2 of them) must span less than 2^31 bytes of each
    const bool outer = p.use_outer || (plan->dev.outer_min_cols > 0 && m >= plan->dev.outer_min_cols);
    const bool indexed = !outer && (plan->dev.use_indexed ||
                                    (plan->dev.indexed_min_cols > 0 && m >= plan->dev.indexed_min_cols));
    const int64_t tile_cols = outer ? p.otw : indexed ? 64 * 6 : p.tile_cols;
    const int64_t span = (tile_cols - 1) / hw + 2;
    if (span * std::max(ihw * p.cin, hw * p.cout) * static_cast<int64_t>(e) >= (int64_t(1) << 31) - 16)
        return fail(SPCONV_E_UNSUPPORTED,
                    "h * w * channels too large: the images of one tile must span less than 2^31 bytes");
    if (plan->host_only)
        return fail(SPCONV_E_ARG, host_only_msg);
    if (plan->static_gen) {
        std::lock_guard<std::mutex> lock(g_static_mu);
        if (g_static[plan->device].gen != plan->static_gen)
            return fail(SPCONV_E_ARG, "a later spconv_plan_create_static on this device replaced the plan's "
                                      "device image");
    }
    int dev = -1;
    hipError_t he = hipGetDevice(&dev);
    if (he != hipSuccess)
        return hip_fail("hipGetDevice", he);
    if (dev != plan->device)
        return fail(SPCONV_E_ARG, "plan was created on device " + std::to_string(plan->device) +
                                      " but the current device is " + std::to_string(dev));
    const int64_t qv = 16 / static_cast<int64_t>(e);  // columns in one 16-byte vector
    const int32_t vec = (hw % qv == 0) && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                        reinterpret_cast<uintptr_t>(y) % 16 == 0;
    if (!plan->passes.empty()) {
        // channel-range passes in order: pass i reads X from its first channel
        for (size_t i = 0; i < plan->passes.size() && he == hipSuccess; ++i) {
            const int64_t skip = static_cast<int64_t>(plan->pass_c0[i]) * ihw * static_cast<int64_t>(e);
            he = spconv::launch_spmm(plan->passes[i]->dev, static_cast<const char *>(x) + skip, y,
                                     static_cast<int32_t>(m), static_cast<int32_t>(hw), vec,
                                     xel * static_cast<int64_t>(e) - skip, yel * static_cast<int64_t>(e), h, w,
                                     static_cast<int32_t>(ow), static_cast<hipStream_t>(stream));
        }
    } else if (outer)
        he = spconv::launch_outer(plan->dev, x, y, static_cast<int32_t>(m), static_cast<int32_t>(hw),
                                  hw % 4 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                                      reinterpret_cast<uintptr_t>(y) % 16 == 0,
                                  xel * static_cast<int64_t>(e), static_cast<hipStream_t>(stream));
    else if (indexed)
        he = spconv::launch_indexed(plan->dev, static_cast<const float *>(x), static_cast<float *>(y),
                                    static_cast<int32_t>(m), static_cast<int32_t>(hw), xel * static_cast<int64_t>(e),
                                    yel * static_cast<int64_t>(e), static_cast<hipStream_t>(stream));
    else
        he = spconv::launch_spmm(plan->dev, x, y, static_cast<int32_t>(m), static_cast<int32_t>(hw), vec,
                                 xel * static_cast<int64_t>(e), yel * static_cast<int64_t>(e), h, w,
                                 static_cast<int32_t>(ow), static_cast<hipStream_t>(stream));
    if (he != hipSuccess)
        return hip_fail("kernel launch", he);
    return SPCONV_OK;
}

spconv_status spconv_conv3x3_hwc(const float *x, const float *weight, const float *bias, spconv_act act,
                                 int32_t stride, float *y, int32_t n, int32_t h, int32_t w, int32_t cin,
                                 int32_t cout, void *stream) {
    g_err.clear();
    if (n < 0 || h < 0 || w < 0)
        return fail(SPCONV_E_ARG, "n, h and w must be >= 0");
    if (stride != 1 && stride != 2)
        return fail(SPCONV_E_ARG, "stride must be 1 or 2");
    if (act < SPCONV_ACT_NONE || act > SPCONV_ACT_RELU6)
        return fail(SPCONV_E_ARG, "act must be SPCONV_ACT_NONE, _RELU or _RELU6");
    if (cin < 1 || cout < 1)
        return fail(SPCONV_E_SHAPE, "cin and cout must be >= 1");
    if (cin > 8)
        return fail(SPCONV_E_UNSUPPORTED, "the HWC convolution supports cin <= 8");
    if (static_cast<int64_t>(n) * h * w == 0)
        return SPCONV_OK;
    if (!x || !weight || !y)
        return fail(SPCONV_E_ARG, "x, weight or y is NULL");
    const int64_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t xel = static_cast<int64_t>(n) * h * w * cin, yel = static_cast<int64_t>(n) * cout * ho * wo;
    if (static_cast<int64_t>(n) * ho * wo > (int64_t(1) << 38))
        return fail(SPCONV_E_SHAPE, "too many output pixels");
    if (static_cast<int64_t>(h) * w * cin >= INT32_MAX || static_cast<int64_t>(n) * ((ho * wo + 255) / 256) >= INT32_MAX)
        return fail(SPCONV_E_SHAPE, "an image must hold fewer than 2^31 elements and n * ceil(ho * wo / 256) "
                                    "must stay below 2^31");
    if (ranges_overlap(x, static_cast<size_t>(xel) * 4, y, static_cast<size_t>(yel) * 4))
        return fail(SPCONV_E_ARG, "x and y overlap");
    const hipError_t he = spconv::launch_conv3x3_hwc(x, weight, bias, y, n, h, w, cin, cout, stride,
                                                     static_cast<int32_t>(act), static_cast<hipStream_t>(stream));
    return he == hipSuccess ? SPCONV_OK : hip_fail("kernel launch", he);
}

spconv_status spconv_depthwise3x3(const float *x, const float *weight, const float *bias, spconv_act act,
                                  int32_t stride, float *y, int32_t n, int32_t c, int32_t h, int32_t w,
                                  void *stream) {
    g_err.clear();
    if (n < 0 || c < 0 || h < 0 || w < 0)
        return fail(SPCONV_E_ARG, "n, c, h and w must be >= 0");
    if (stride != 1 && stride != 2)
        return fail(SPCONV_E_ARG, "stride must be 1 or 2");
    if (act < SPCONV_ACT_NONE || act > SPCONV_ACT_RELU6)
        return fail(SPCONV_E_ARG, "act must be SPCONV_ACT_NONE, _RELU or _RELU6");
    if (static_cast<int64_t>(n) * c * h * w == 0)
        return SPCONV_OK;
    if (!x || !weight || !y)
        return fail(SPCONV_E_ARG, "x, weight or y is NULL");
    const int64_t ho = (h - 1) / stride + 1, wo = (w - 1) / stride + 1;
    const int64_t xel = static_cast<int64_t>(n) * c * h * w, yel = static_cast<int64_t>(n) * c * ho * wo;
    if (yel > (int64_t(1) << 38))
        return fail(SPCONV_E_SHAPE, "too many output elements");
    if (ranges_overlap(x, static_cast<size_t>(xel) * 4, y, static_cast<size_t>(yel) * 4))
        return fail(SPCONV_E_ARG, "x and y overlap");
    const hipError_t he = spconv::launch_dw3x3(x, weight, bias, y, n, c, h, w, stride, static_cast<int32_t>(act),
                                               static_cast<hipStream_t>(stream));
    return he == hipSuccess ? SPCONV_OK : hip_fail("kernel launch", he);
}

spconv_status spconv_linear(const float *x, const float *weight, const float *bias, spconv_act act, float *y,
                            int32_t n, int32_t cin, int32_t cout, void *stream) {
    g_err.clear();
    if (n < 0 || cin < 0 || cout < 0)
        return fail(SPCONV_E_ARG, "n, cin and cout must be >= 0");
    if (act < SPCONV_ACT_NONE || act > SPCONV_ACT_RELU6)
        return fail(SPCONV_E_ARG, "act must be SPCONV_ACT_NONE, _RELU or _RELU6");
    if (static_cast<int64_t>(n) * cout == 0)
        return SPCONV_OK;
    if (cin == 0)
        return fail(SPCONV_E_SHAPE, "cin must be >= 1");
    if ((static_cast<int64_t>(n) + 3) / 4 > 65535)
        return fail(SPCONV_E_SHAPE, "n must be at most 262140");
    if (!x || !weight || !y)
        return fail(SPCONV_E_ARG, "x, weight or y is NULL");
    if (ranges_overlap(x, static_cast<size_t>(n) * cin * 4, y, static_cast<size_t>(n) * cout * 4))
        return fail(SPCONV_E_ARG, "x and y overlap");
    const hipError_t he = spconv::launch_linear(x, weight, bias, y, n, cin, cout, static_cast<int32_t>(act),
                                                static_cast<hipStream_t>(stream));
    return he == hipSuccess ? SPCONV_OK : hip_fail("kernel launch", he);
}

spconv_status spconv_global_avg_pool(const float *x, float *y, int32_t n, int32_t c, int32_t h, int32_t w,
                                     void *stream) {
    g_err.clear();
    if (n < 0 || c < 0 || h < 0 || w < 0)
        return fail(SPCONV_E_ARG, "n, c, h and w must be >= 0");
    if (static_cast<int64_t>(n) * c == 0)
        return SPCONV_OK;
    if (static_cast<int64_t>(h) * w == 0)
        return fail(SPCONV_E_SHAPE, "h * w must be >= 1 to average");
    if (!x || !y)
        return fail(SPCONV_E_ARG, "x or y is NULL");
    const int64_t planes = static_cast<int64_t>(n) * c, hw = static_cast<int64_t>(h) * w;
    if (planes > (int64_t(1) << 38))
        return fail(SPCONV_E_SHAPE, "too many planes");
    if (ranges_overlap(x, static_cast<size_t>(planes * hw) * 4, y, static_cast<size_t>(planes) * 4))
        return fail(SPCONV_E_ARG, "x and y overlap");
    const hipError_t he = spconv::launch_gap(x, y, n, c, hw, static_cast<hipStream_t>(stream));
    return he == hipSuccess ? SPCONV_OK : hip_fail("kernel launch", he);
}

spconv_status spconv_destroy(spconv_plan plan) {
    g_err.clear();
    if (!plan)
        return SPCONV_OK;
    const hipError_t e = free_plan(plan);
    return e == hipSuccess ? SPCONV_OK : hip_fail("hipFree", e);
}

const char *spconv_last_error(void) { return g_err.c_str(); }

spconv_status spconv_plan_get_info(spconv_plan plan, spconv_plan_info *info) {
    g_err.clear();
    if (!plan || !info)
        return fail(SPCONV_E_ARG, "plan or info is NULL");
    const spconv::PackedPlan &p = plan->host;
    std::memset(info, 0, sizeof(*info));
    info->cout = p.cout;
    info->cin = p.cin;
    info->block_rows = p.k;
    info->storage = p.storage;
    info->act = p.act;
    info->kernel = p.kernel;
    info->group_lanes = p.group_lanes;
    info->bundle_rows = p.bundle_rows;
    info->cols_per_lane = p.cols_per_lane;
    info->tile_cols = p.tile_cols;
    info->waves = p.waves;
    info->max_parts = p.max_parts;
    info->pipe_sets = p.kernel == spconv::KERNEL_STRIP ? p.pipe_sets : 0;
    info->regions = p.kernel == spconv::KERNEL_STRIP ? p.regions : 0;
    info->lds_bytes = p.lds_bytes;
    info->nnzb = p.nnzb / p.kc;
    info->slots = p.slots;
    info->max_wave_cost = p.max_wave_cost;
    info->sum_wave_cost = p.sum_wave_cost;
    info->device_bytes = static_cast<int64_t>(plan->dbytes);
    info->dw_stride = p.dw_stride;
    info->dw_act = p.dw_act;
    info->block_cols = p.kc;
    info->split_rows = p.split_rows;
    info->indexed_min_cols = plan->host_only ? 0 : plan->dev.indexed_min_cols;
    info->outer_min_cols = plan->host_only ? 0 : plan->dev.outer_min_cols;
    info->channel_passes = static_cast<int64_t>(plan->passes.size());
    return SPCONV_OK;
}

// The packed streams hold input-channel blocks expanded to single channels
// (kc consecutive entries per block, in order): gather them back.
static void reblock(const spconv::PackedPlan &p, const std::vector<int32_t> &rp, const std::vector<int32_t> &ci,
             const std::vector<float> &va, int32_t *row_ptr, int32_t *col_idx, float *values) {
    const int32_t k = p.k, kc = p.kc, rows = p.cout / k;
    if (row_ptr)
        for (int32_t r = 0; r <= rows; ++r)
            row_ptr[r] = rp[r] / kc;
    const int64_t nb = rp[rows] / kc;
    for (int64_t t = 0; t < nb; ++t) {
        if (col_idx)
            col_idx[t] = ci[t * kc];
        if (values)
            for (int32_t i = 0; i < k; ++i)
                for (int32_t j = 0; j < kc; ++j)
                    values[(t * k + i) * kc + j] = va[(t * kc + j) * k + i];
    }
}

spconv_status spconv_plan_unpack(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx, float *values,
                                 int32_t *perm) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    const spconv::PackedPlan &p = plan->host;
    if (p.kc == 1) {
        spconv::unpack_plan(p, row_ptr, col_idx, values, perm);
        return SPCONV_OK;
    }
    try {
        std::vector<int32_t> rp(p.cout / p.k + 1), ci(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1)));
        std::vector<float> va(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1) * p.k));
        spconv::unpack_plan(p, rp.data(), ci.data(), va.data(), perm);
        reblock(p, rp, ci, va, row_ptr, col_idx, values);
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while unpacking");
    }
    return SPCONV_OK;
}

spconv_status spconv_plan_unpack_interleaved(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx,
                                             float *values) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    std::string err;
    const spconv::PackedPlan &p = plan->host;
    if (p.kc == 1) {
        const spconv::Status st = spconv::unpack_interleaved(p, row_ptr, col_idx, values, err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        return SPCONV_OK;
    }
    try {
        std::vector<int32_t> rp(p.cout / p.k + 1), ci(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1)));
        std::vector<float> va(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1) * p.k));
        const spconv::Status st = spconv::unpack_interleaved(p, rp.data(), ci.data(), va.data(), err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        reblock(p, rp, ci, va, row_ptr, col_idx, values);
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while unpacking");
    }
    return SPCONV_OK;
}

spconv_status spconv_plan_unpack_outer(spconv_plan plan, int32_t *row_ptr, int32_t *col_idx, float *values) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    std::string err;
    const spconv::PackedPlan &p = plan->host;
    if (p.kc == 1) {
        const spconv::Status st = spconv::unpack_outer(p, row_ptr, col_idx, values, err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        return SPCONV_OK;
    }
    try {
        std::vector<int32_t> rp(p.cout / p.k + 1), ci(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1)));
        std::vector<float> va(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1) * p.k));
        const spconv::Status st = spconv::unpack_outer(p, rp.data(), ci.data(), va.data(), err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        reblock(p, rp, ci, va, row_ptr, col_idx, values);
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while unpacking");
    }
    return SPCONV_OK;
}

spconv_status spconv_plan_unpack_indexed(spconv_plan plan, int32_t from_pairs, int32_t *row_ptr, int32_t *col_idx,
                                         float *values) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    std::string err;
    const spconv::PackedPlan &p = plan->host;
    if (p.kc == 1) {
        const spconv::Status st = spconv::unpack_indexed(p, from_pairs != 0, row_ptr, col_idx, values, err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        return SPCONV_OK;
    }
    try {
        std::vector<int32_t> rp(p.cout / p.k + 1), ci(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1)));
        std::vector<float> va(static_cast<size_t>(std::max<int64_t>(p.nnzb, 1) * p.k));
        const spconv::Status st = spconv::unpack_indexed(p, from_pairs != 0, rp.data(), ci.data(), va.data(), err);
        if (st != spconv::OK)
            return fail(static_cast<spconv_status>(st), err);
        reblock(p, rp, ci, va, row_ptr, col_idx, values);
    } catch (const std::bad_alloc &) {
        return fail(SPCONV_E_NOMEM, "host allocation failed while unpacking");
    }
    return SPCONV_OK;
}

spconv_status spconv_plan_check(spconv_plan plan, int32_t *flags, int32_t clear) {
    g_err.clear();
    if (!plan || !flags)
        return fail(SPCONV_E_ARG, "plan or flags is NULL");
    if (plan->host_only || !plan->dev.flag)
        return fail(SPCONV_E_ARG, "a host-only plan has no device error word");
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess)
        return hip_fail("hipGetDevice", e);
    if (cur != plan->device && (e = hipSetDevice(plan->device)) != hipSuccess)
        return hip_fail("hipSetDevice", e);
    spconv_status st = SPCONV_OK;
    if ((e = hipDeviceSynchronize()) != hipSuccess) {
        st = hip_fail("hipDeviceSynchronize", e);
    } else if ((e = hipMemcpy(flags, plan->dev.flag, sizeof(int32_t), hipMemcpyDeviceToHost)) != hipSuccess) {
        st = hip_fail("hipMemcpy (error word)", e);
    } else if (clear) {
        const int32_t zero = 0;
        if ((e = hipMemcpy(plan->dev.flag, &zero, sizeof(int32_t), hipMemcpyHostToDevice)) != hipSuccess)
            st = hip_fail("hipMemcpy (clear error word)", e);
    }
    if (cur != plan->device)
        (void)hipSetDevice(cur);
    return st;
}

spconv_status spconv_plan_set_wait_limit(spconv_plan plan, int32_t sleeps) {
    g_err.clear();
    if (!plan)
        return fail(SPCONV_E_ARG, "plan is NULL");
    if (sleeps < 0)
        return fail(SPCONV_E_ARG, "the wait bound must be >= 0");
    plan->dev.spin_limit = sleeps;
    for (spconv_plan_s *q : plan->passes)
        q->dev.spin_limit = sleeps;
    return SPCONV_OK;
}

}  // extern "C"
