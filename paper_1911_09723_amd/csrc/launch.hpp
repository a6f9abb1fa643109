// Internal interface between the C ABI and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

#include "planner.hpp"

namespace spconv {

// Device-resident copy of a PackedPlan (see planner.hpp for the layout).
struct DevicePlan {
    int32_t kernel = KERNEL_STRIP;
    int32_t lanes_per_row = 16;
    int32_t tile_cols = 64;
    int32_t waves = 1;
    int32_t lds_bytes = 0;
    int32_t k = 1;
    int32_t storage = 0;
    int32_t act = 0;
    int32_t cin = 0, cout = 0;
    const int32_t *idx = nullptr;
    const float *val = nullptr;
    const int32_t *hdr = nullptr;
    const int32_t *rows = nullptr;
    const int32_t *wave_ptr = nullptr;
    const float *bias = nullptr;
};

// Queue one launch computing all m = N * hw columns.  `vec` != 0 promises
// that hw is a multiple of the per-lane column count and x, y are 16-byte
// aligned, enabling 16-byte global loads and stores.
hipError_t launch_spmm(const DevicePlan &p, const void *x, void *y, int64_t m, int32_t hw, int32_t vec,
                       hipStream_t stream);

}  // namespace spconv
