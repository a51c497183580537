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

// ScatterToBEV: a clear of the whole map, then the voxels' values.
struct BevConfig {
  const int4* coords;    // [rows] (b, iz, iy, ix)
  const float* feats;    // [rows][C]
  const int64_t* voff;   // [B+1]
  float* map;            // [B][C*Dz][Dy][Dx]
  int32_t* fault;        // MMBEV_FAULT_VOXELS is ORed in; null: no contract checks
  int64_t rows;          // rows the voxel arrays hold: B * max_voxels
  uint64_t plane;        // Dx * Dy
  uint32_t Dx, Dy, Dz;
  int32_t B, C, max_voxels;
  int32_t vec;           // the map is 16-byte aligned: the clear uses 16-byte stores
};

hipError_t launch_bev(const BevConfig& c, hipStream_t st);

}  // namespace mmbev
