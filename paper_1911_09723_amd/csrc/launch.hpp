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
    int32_t vec_bytes = 16;
    int32_t tile_cols = 64;
    int32_t waves = 1;
    int32_t loader_waves = 0;
    int32_t lds_bytes = 0;
    int32_t k = 1;
    int32_t storage = 0;
    int32_t act = 0;
    int32_t cin = 0, cout = 0;
    int32_t idx_bytes = 0;      // size of the index stream (bounds of its buffer resource)
    int32_t val_bytes = 0;      // size of the weight stream
    int32_t num_cus = 0;        // compute units of the plan's device
    int32_t blocks_per_cu = 0;  // resident workgroups per CU of the strip kernel
    int32_t strip_bytes = 0;    // LDS bytes of the X strip (the bundle table follows it)
    int32_t meta_words = 0;     // 32-bit words of the bundle table
    int32_t nbundles = 0;
    int32_t max_parts = 1;      // most workgroups that may share one tile
    const int32_t *idx = nullptr;
    const float *val = nullptr;
    const int32_t *hdr = nullptr;         // (first step, steps) per bundle
    const int32_t *meta = nullptr;        // rows, biases (fp32 bits), steps
    const int32_t *wave_ptr = nullptr;    // bundles of each wave
    const int32_t *wave_chunk = nullptr;  // first chunk of each wave
    const int32_t *split = nullptr;       // 65 part boundaries per wave
};

// Once per plan, on its device: raise the kernel's dynamic-LDS limit when
// needed and record num_cus and blocks_per_cu.
hipError_t prepare_launch(DevicePlan &p);

// Queue one launch computing all m = N * hw columns.  `vec` != 0 promises
// that hw is a multiple of the columns in one 16-byte vector and that x and y
// are 16-byte aligned, enabling 16-byte global loads and stores.
hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int32_t m, int32_t hw, int32_t vec,
                       hipStream_t stream);

}  // namespace spconv
