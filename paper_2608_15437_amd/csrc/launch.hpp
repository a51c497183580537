// Host-side launchers of the voxelisation kernels (one per translation unit).
#pragma once

#include <algorithm>

#include "common.hpp"

namespace mmbev {

hipError_t launch_stage(const Config& c, hipStream_t st);
hipError_t launch_filter(const Config& c, hipStream_t st);
hipError_t launch_segments(const Config& c, hipStream_t st);
hipError_t launch_compact(const Config& c, uint32_t* kout, uint32_t* vout, hipStream_t st);
hipError_t launch_radix_pass(const Config& c, int pass, const uint32_t* kin, const uint32_t* vin, uint32_t* kout,
                             uint32_t* vout, hipStream_t st);
hipError_t launch_unique(const Config& c, const uint32_t* keys, hipStream_t st);
hipError_t launch_finalize(const Config& c, hipStream_t st);
hipError_t launch_cap(const Config& c, const uint32_t* vals, hipStream_t st);
hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);

}  // namespace mmbev
