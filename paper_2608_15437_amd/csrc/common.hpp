// Shared definitions of the gfx950 voxelisation path: the launch
// configuration computed on the host, the workspace layout, and the pinned
// per-point arithmetic (Eq. 6 compensation, the Alg. 1 ROI keep test, grid
// quantisation) that the filter and the mean kernels must evaluate
// identically.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mmbev.h"

namespace mmbev {

constexpr int kBlock = 256;           // threads per workgroup (4 wave64)
constexpr int kWaves = kBlock / 64;
constexpr int kFilterTile = 1024;     // points per filter tile (unit of the per-tile frame/ROI ranges)
constexpr int kWaveQueue = 128;       // candidate ring of one filter wave (power of two, >= 128)
constexpr int kMaxLdsFrames = 64;     // frames of one filter chunk whose offsets are staged in LDS
constexpr int kMaxLdsRois = 256;      // ROI records of one filter chunk staged in LDS
constexpr int kMaxLdsBudgetWords = 256;
constexpr int kMaxSortLdsFrames = 4096;  // frame offsets staged in LDS by the sort and scan kernels
constexpr int kMaxFilterGrid = 4096;     // persistent filter workgroups
constexpr int kMaxFilterChunks = kMaxFilterGrid * kWaves;  // filter wave chunks
constexpr int kMaxSortChunks = 1024;     // chunks of a radix pass and of the head scan
constexpr int kSortItems = 8;         // items per thread in a radix pass
constexpr int kSortTile = kBlock * kSortItems;           // 2048 pairs
constexpr int kSortBins = 256;        // max radix digit width 8 bits
constexpr int kMaxPasses = 6;         // 48 key bits
constexpr int kScanItems = 16;        // items per thread in the head scan
constexpr int kScanTile = kBlock * kScanItems;           // 4096 pairs
constexpr int kMeanTile = kBlock;                        // one voxel per thread
constexpr int kMaxPoseLds = 64;       // (frame, sweep) poses staged in LDS per filter chunk
constexpr uint32_t kSpinLimit = 1u << 20;

// Look-back status word: [63:32] tag, [31:30] flag, [29:0] value.
constexpr uint32_t kFlagAgg = 1u << 30;
constexpr uint32_t kFlagIncl = 2u << 30;
constexpr uint32_t kValueMask = (1u << 30) - 1u;

// Tag slots of the look-back launches of one call.
enum Slot : uint32_t {
  kSlotFilter = 0,
  kSlotSort0 = 1,        // .. kSlotSort0 + kMaxPasses - 1
  kSlotUnique = 7,
  kNumSlots = 16,
};

// Workspace header: per-call counters, rewritten by the first kernel of a call.
struct alignas(256) WsHeader {
  int32_t fault;              // byte 0: MMBEV_FAULT_* bits of the last call
  uint32_t epoch;             // call counter; tags look-back words
  uint32_t kept;              // K, kept points
  uint32_t voxels;            // V, distinct voxels over all frames
  uint32_t capped_voxels;     // voxels of frames over the cap
  uint32_t any_capped;        // 1 if some frame exceeds max_voxels
  uint32_t pad[10];
  uint32_t hist[kMaxPasses][kSortBins];      // digit histograms of the radix passes
};

// Frame and ROI range of one filter tile, precomputed by the staging kernel.
struct TileInfo {
  int32_t f0, f1;      // frames of the tile's first and last point
  int32_t r_lo, r_hi;  // ROIs of frames f0..f1 (clamped to [0, R])
};

// Everything a kernel needs, computed once on the host and passed by value.
struct Config {
  // inputs
  const float* feat;
  const uint8_t* sweep;
  const float* poses;
  const int64_t* frame_off;
  const mmbev_roi_t* rois;
  const int32_t* roi_off;
  const uint8_t* budget;
  int64_t stride;
  int32_t N;  // < 2^30
  int32_t C, B, S, M, cap;
  int32_t R, max_rois, W;  // W: 32-bit mask words per cell
  float mn[3], vs[3], Df[3];
  float inv_vs[3];         // 1/voxel_size, for the conservative cell lookup only
  float nmin_v[3];         // -range_min/voxel_size, same use
  int32_t cell_pad;        // voxels added around each ROI's cell rectangle
  uint32_t Dx, Dy, Dz;
  int32_t cell_shift, ncx, ncy, ncells;
  // keys: key_local = (iz*Dy + iy)*Dx + ix < 2^kb; frame b above it
  int32_t kb, fb, key_has_frame;  // key_has_frame: kb + fb <= 32, key = b << kb | key_local
  int32_t passes, dbits;
  int32_t vec;  // 16-byte vector loads allowed
  // outputs
  int32_t* out_coords;
  int32_t* out_counts;
  float* out_feats;
  int32_t* out_point_idx;
  int64_t* out_voxel_offsets;
  // workspace
  WsHeader* hdr;
  uint32_t* cellmask;      // [B][ncells][W]
  uint32_t* cellany;       // [B][ncells], OR of a cell's W words (== cellmask when W == 1)
  uint32_t* budgetmask;    // [B][S][W]
  TileInfo* tinfo;         // [filter tiles]
  uint32_t* fcount;        // [filter_chunks] kept pairs per filter wave chunk
  uint32_t* cnt;           // [256][max(filter_chunks, sort_chunks)] digit counts -> offsets
  uint32_t* tot;           // [256] digit totals of a radix pass
  uint32_t* hcount;        // [sort_chunks] voxel heads per chunk
  uint32_t* keys[2];
  uint32_t* vals[2];
  uint32_t* capkey;        // [N] first point index of each voxel of a capped frame
  uint32_t* out_rank;      // [N] row of a capped frame's voxel inside its frame, or ~0u
  uint32_t* seg_start;     // [N+1] first sorted position of voxel v
  uint32_t* vox_off;       // [B+1] first voxel of frame b
  int32_t filter_tiles;                          // kFilterTile-point tiles
  int32_t filter_grid, filter_chunk_tiles;       // persistent workgroups, tiles per workgroup
  int32_t filter_chunks, filter_chunk_points;    // wave chunks (kWaves per workgroup), points per wave chunk
  int32_t sort_chunks, mean_grid;
};

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  uint32_t l = __lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ uint32_t tag_of(uint32_t epoch, uint32_t slot) { return epoch * kNumSlots + slot; }

__device__ __forceinline__ uint64_t status_word(uint32_t tag, uint32_t flag, uint32_t value) {
  return ((uint64_t)tag << 32) | (uint64_t)(flag | (value & kValueMask));
}

__device__ __forceinline__ void status_store(uint64_t* p, uint64_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t status_load(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void raise_fault(WsHeader* h, int32_t bits) {
  __hip_atomic_fetch_or(&h->fault, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until a look-back status word carries this launch's tag and a flag.
// Bounded: on expiry the fault bit is raised and an inclusive zero returned.
__device__ __forceinline__ uint64_t status_wait(const uint64_t* p, uint32_t tag, WsHeader* h) {
  uint32_t spins = 0;
  for (;;) {
    const uint64_t w = status_load(p);
    if ((uint32_t)(w >> 32) == tag && ((uint32_t)w & (kFlagAgg | kFlagIncl))) return w;
    if (++spins >= kSpinLimit) {
      raise_fault(h, MMBEV_FAULT_WAIT);
      return status_word(tag, kFlagIncl, 0);
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Exclusive prefix of the tiles before `tile` (one value per tile), computed
// by one whole wave: each step reads 64 predecessors at once and stops at
// the nearest one that already holds an inclusive prefix.  When many tiles
// publish together, a lane-by-lane walk would cost one memory round trip per
// predecessor; this costs one per 64.  Every lane returns the same value.
__device__ __forceinline__ uint32_t look_back_wave(const uint64_t* status, int64_t tile, uint32_t tag, WsHeader* h) {
  const int lane = threadIdx.x & 63;
  uint32_t prefix = 0;
  for (int64_t hi = tile - 1; hi >= 0; hi -= 64) {
    const int64_t j = hi - lane;  // lane 0: nearest predecessor
    uint32_t flag = kFlagIncl, val = 0;
    if (j >= 0) {
      const uint64_t w = status_wait(status + j, tag, h);
      flag = (uint32_t)w & (kFlagAgg | kFlagIncl);
      val = (uint32_t)w & kValueMask;
    }
    const uint64_t incl = __ballot(flag == kFlagIncl);
    const int first = incl ? __builtin_ctzll(incl) : 64;
    uint32_t x = lane <= first ? val : 0u;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, 64);
    prefix += x;
    if (incl) break;
  }
  return prefix;
}

// Exclusive prefix of one digit over the tiles before `tile` (one thread per
// digit; status words of tile j for this digit at status[j * step]).  Reads
// kLookWindow predecessors per step with independent loads.
constexpr int kLookWindow = 8;
__device__ __forceinline__ uint32_t look_back_window(const uint64_t* status, int64_t tile, int64_t step,
                                                     uint32_t tag, WsHeader* h) {
  uint32_t prefix = 0;
  for (int64_t hi = tile - 1; hi >= 0; hi -= kLookWindow) {
    uint64_t w[kLookWindow];
#pragma unroll
    for (int k = 0; k < kLookWindow; ++k) w[k] = hi - k >= 0 ? status_load(status + (hi - k) * step) : 0ull;
#pragma unroll
    for (int k = 0; k < kLookWindow; ++k) {
      if (hi - k < 0) return prefix;
      uint64_t x = w[k];
      if (!((uint32_t)(x >> 32) == tag && ((uint32_t)x & (kFlagAgg | kFlagIncl))))
        x = status_wait(status + (hi - k) * step, tag, h);
      prefix += (uint32_t)x & kValueMask;
      if ((uint32_t)x & kFlagIncl) return prefix;
    }
  }
  return prefix;
}

// Exclusive prefix over the workgroup (kBlock threads, all must call);
// s_tmp holds kWaves words of LDS.  Returns the prefix, sets total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_tmp, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_tmp[wave] = x;
  __syncthreads();
  uint32_t wpre = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    uint32_t t = s_tmp[w];
    wpre += (w < wave) ? t : 0u;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return wpre + x - v;
}

// Chunk w of a compact array [0, K): kSortTile-aligned, at most G chunks,
// visited in order (radix passes and the voxel head scan).
__device__ __forceinline__ void chunk_range(uint32_t K, uint32_t w, uint32_t G, uint32_t& lo, uint32_t& hi) {
  uint32_t cs = (K + G - 1) / G;
  cs = (cs + kSortTile - 1) / kSortTile * kSortTile;
  const uint64_t l = (uint64_t)w * cs;
  lo = (uint32_t)min(l, (uint64_t)K);
  hi = (uint32_t)min(l + cs, (uint64_t)K);
}

// Frame of point index i: largest b with off[b] <= i, clamped to [0, B-1].
__device__ __forceinline__ int32_t frame_of_point(const int64_t* off, int32_t B, int64_t i) {
  int32_t lo = 0, hi = B - 1;
  while (lo < hi) {
    int32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// ------------------------------------------------ pinned point arithmetic
// The library is compiled with -ffp-contract=off and correctly rounded fp32
// division, so each operator below is one IEEE operation; fused
// multiply-adds are written out where the definition has them.
__device__ __forceinline__ float fma_rn(float a, float b, float c) { return __builtin_fmaf(a, b, c); }

// Eq. 6: p' = R p + T as one fused chain per row.
__device__ __forceinline__ void compensate(const float* P, float x, float y, float z, float& ox, float& oy,
                                           float& oz) {
  ox = fma_rn(P[0], x, fma_rn(P[1], y, fma_rn(P[2], z, P[3])));
  oy = fma_rn(P[4], x, fma_rn(P[5], y, fma_rn(P[6], z, P[7])));
  oz = fma_rn(P[8], x, fma_rn(P[9], y, fma_rn(P[10], z, P[11])));
}

// Alg. 1 keep test against one oriented box of ROI_L (edges inclusive).
__device__ __forceinline__ bool inside_roi(const mmbev_roi_t& r, float x, float y) {
  float dx = x - r.cx;
  float dy = y - r.cy;
  float s_dy = r.sin_yaw * dy;
  float s_dx = r.sin_yaw * dx;
  float lx = fma_rn(r.cos_yaw, dx, s_dy);
  float ly = fma_rn(r.cos_yaw, dy, -s_dx);
  return fabsf(lx) <= r.ext_x && fabsf(ly) <= r.ext_y;
}

// Grid coordinate on one axis; false when outside [0, D) or not a number.
__device__ __forceinline__ bool quantize_axis(float p, float mn, float vs, float Df, int32_t& i) {
  float f = (p - mn) / vs;
  bool ok = (f >= 0.0f) && (f < Df);
  i = ok ? (int32_t)f : 0;
  return ok;
}

}  // namespace mmbev
