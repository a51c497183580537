// Host-side launchers of the voxelisation kernels (one per translation unit).
#pragma once

#include "common.hpp"

namespace mmbev {

hipError_t launch_stage(const Config& c, hipStream_t st);
hipError_t launch_filter(const Config& c, hipStream_t st);
// which: 0 = voxel-key sort (Alg. 1 Voxelize), 1 = first-appearance sort of capped frames' voxels
hipError_t launch_radix_pass(const Config& c, int which, int pass, const uint32_t* kin, const uint32_t* vin,
                             uint32_t* kout, uint32_t* vout, bool mark, hipStream_t st);
hipError_t launch_unique(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_finalize(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_cap_prep(const Config& c, const uint32_t* vals, uint32_t* ckeys, uint32_t* cvals,
                           hipStream_t st);
hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);

}  // namespace mmbev
