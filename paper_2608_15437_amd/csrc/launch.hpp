// Host-side launchers of the voxelisation kernels (one per translation unit).
#pragma once

#include <algorithm>

#include "common.hpp"

namespace mmbev {

hipError_t launch_stage(const Config& c, hipStream_t st);
hipError_t launch_filter(const Config& c, hipStream_t st);
hipError_t launch_segments(const Config& c, hipStream_t st);
hipError_t launch_compact(const Config& c, uint32_t* kout, hipStream_t st);
hipError_t launch_radix_pass(const Config& c, int pass, const uint32_t* kin, const uint32_t* vin, uint32_t* kout,
                             uint32_t* vout, hipStream_t st);
hipError_t launch_heads(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_fincap(const Config& c, hipStream_t st);
hipError_t launch_mean(const Config& c, const uint32_t* keys, const uint32_t* vals, hipStream_t st);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st);
hipError_t launch_copy_fault(const WsHeader* h, int32_t* out, hipStream_t st);

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

// Connected-component proposer: workspace header, and what its kernels read.
struct CcHeader {
  int32_t fault;      // byte 0: MMBEV_FAULT_VOXELS
  uint32_t clusters;  // clusters over all frames
};

constexpr uint32_t kCcRowGrid = 8192;     // workgroups of the per-row launches (they loop)
constexpr int64_t kCcMaxCells = (int64_t)1 << 29;  // cells over all frames (single-workgroup block scan)

struct CcConfig {
  const int4* coords;       // [rows]
  const int32_t* counts;    // [rows]
  const int64_t* voff;      // [B+1]
  mmbev_cluster_t* out;     // [rows]
  int64_t* out_off;         // [B+1]
  int32_t* labels;          // [rows]
  CcHeader* hdr;
  uint32_t* occ;            // [nwords] occupied cells; rootbits follows it directly
  uint32_t* rootbits;       // [nwords] roots of kept components
  uint32_t* wpre;           // [nwords] kept roots in the words before
  uint32_t* bsum;           // [nblocks]
  int32_t* parent;          // [cells], valid at occupied cells only
  int32_t* cnt;             // [cells], valid at occupied cells only
  int32_t* rcell;           // [rows] the row's cell (top bit: another row owns it), or -1
  int64_t rows;             // B * max_voxels
  int64_t cells;            // B * ncell
  uint32_t nwords, nblocks;
  uint32_t Dx, Dy, Dz;
  int32_t B, max_voxels, ncell, Wx, Wy, shift, z_min, z_max, conn, min_cells;
};

hipError_t launch_clusters(const CcConfig& c, hipStream_t st);

}  // namespace mmbev
