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
// point filter
constexpr int kWaveTile = 256;        // points per filter wave tile (64 lanes x 4)
constexpr int kWaveQueue = 128;       // candidate ring of one filter wave (power of two, >= 128)
constexpr int kFilterDepth = 2;       // register buffers of a filter wave's tile pipeline (>= 2)
constexpr int kFilterWaveTarget = 16384;  // filter wave chunks aimed for (a few per resident wave: balance)
constexpr int kFilterMinWaves = 4096;     // fewest filter chunks for which two-tile chunks are taken over one-tile ones
constexpr int kMaxChunkPoints = 4096;  // points of one filter chunk at most
constexpr int kChunkWords = kMaxChunkPoints / 32;  // words of a chunk's kept bitmap
constexpr int kMaxLdsFrames = 64;     // frames of one filter workgroup staged in LDS
constexpr int kMaxLdsRois = 256;      // ROI records of one filter workgroup staged in LDS
constexpr int kMaxLdsBudgetWords = 256;
constexpr int kMaxPoseLds = 64;       // (frame, sweep) poses of one filter workgroup staged in LDS
constexpr int kSmallChunks = 2048;  // calls of at most this many filter chunks need no segments launch
constexpr int kFuseFrames = kBlock - 1;  // frames of a call whose point filter lays out the call itself (one per thread)
constexpr int kFuseWideFrames = 16;    // ... and with several ROI words per cell, at most this many frames
constexpr int kFuseWordCap = 8192;     // ... whose cells' ROI words (cells x words) fit this many LDS words
constexpr int kMaxCellSide = 64;      // coarse BEV cells per grid side (at most 64 x 64 per frame)
constexpr int kMaxLdsCells = 4096;    // cell words of one filter workgroup staged in LDS (16 KB)
// radix passes (segmented by frame) and the voxel head scan
constexpr int kMaxDigitBits = 9;
constexpr int kSortBins = 1 << kMaxDigitBits;  // 512
constexpr int kSortItems = 8;         // pairs per thread in a scatter tile
constexpr int kSortTile = kBlock * kSortItems;  // 2048 pairs
constexpr int kCountItems = 16;       // pairs per thread per batch of the count kernel
constexpr int kHalfTileFramePairs = 16 * kSortTile / 2;  // frames of at most this many pairs may take half-tile chunks
constexpr int kMaxFrameChunks = 64;   // pair chunks of one frame at most (chunks never straddle frames)
constexpr int kScanItems = 16;        // items per thread in the single-workgroup scans
constexpr int kScanTile = kBlock * kScanItems;  // 4096
constexpr int kMeanTile = kBlock;     // one voxel per thread
constexpr int kVoxTile = 2048;        // sorted pairs of a voxel tile (the heads, cap and mean kernels' unit)
constexpr int kCus = 256;            // compute units of the device (8 XCDs x 32)
constexpr int kScatterPerCu = 4;     // scatter workgroups resident per CU (its launch bounds hold it to 128 VGPRs: four)
constexpr int kCountGrid = 2048;     // count workgroups (eight per CU)

// Workspace header: per-call counters, rewritten by the first kernels of a call.
constexpr int kMaxCapSteps = 48;             // steps of a cap shared by several workgroups (frames of up to 1.5M pairs)
constexpr uint32_t kCapStepSlots = 1u << 15;  // slots of one step of a cap's flag pass

struct alignas(256) WsHeader {
  int32_t fault;              // byte 0: MMBEV_FAULT_* bits of the last call
  uint32_t epoch;             // call counter
  uint32_t kept;              // K, kept points
  uint32_t voxels;            // V, distinct voxels over all frames
  uint32_t capped_voxels;     // voxels of frames over the cap
  uint32_t any_capped;        // 1 if some frame exceeds max_voxels
  uint32_t fchunks;           // filter chunks (points of one frame each)
  uint32_t schunks;           // pair chunks (pairs of one frame each)
  uint32_t vtiles;            // voxel tiles (kVoxTile sorted pairs of one frame each, the last one shorter)
  uint32_t most_frame;        // the frame with the most pairs (the smallest index among equals)
  uint32_t most_pairs;        // its pairs
  uint32_t cap_steps[kMaxCapSteps];  // that frame's kept voxels per kCapStepSlots slots, when its cap is shared
};
static_assert(sizeof(WsHeader) == 256, "one 256-byte header");

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
  float inv_vs[3];         // 1/voxel_size, for the conservative cell lookup and the quantisation shortcut
  float nmin_v[3];         // -range_min/voxel_size, for the cell lookup only
  int32_t cell_pad;        // voxels added around each ROI's cell rectangle
  uint32_t Dx, Dy, Dz;
  int32_t cell_shift, ncx, ncy, ncells;
  // keys: (iz*Dy + iy)*Dx + ix < 2^kb, sorted within each frame in `passes`
  // least-significant-digit passes of dbits bits
  int32_t kb, passes, dbits;
  int32_t vec;  // 16-byte vector loads allowed
  int32_t fuse_stage;  // the point filter lays out the call and builds its frame's tables (no staging kernel)
  int32_t small_call;  // at most kSmallChunks filter chunks: the compaction launch does the segments kernel's work
  // out-of-ROI keep (Alg. 1 rate rho_out): threshold round(rho_out * 2^24)
  // on the top 24 bits of the point's SplitMix64 draw; 0 keeps none
  uint32_t bg_thr;
  uint64_t bg_seed;
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
  uint32_t* fchunk_first;  // [B+1] first filter chunk of frame b
  uint32_t* fbits;         // [fchunk_max][fchunk_words] bit j of chunk k: point fchunk_lo[k] + j is kept
  uint32_t* fcount;        // [fchunk_max] kept points of filter chunk k
  uint32_t* fchunk_lo;     // [fchunk_max] first point of filter chunk k
  uint32_t* fchunk_frame;  // [fchunk_max] frame of filter chunk k
  uint32_t* wg_frame;      // [filter_grid] frame of filter workgroup g's first chunk (kNoFrame: no chunk)
  const float* spare_tile; // kSpareTileBytes the filter's past-the-end pipeline loads read (values unused)
  uint32_t* fprefix;       // [fchunk_max + 1] kept pairs of the filter chunks before k
  uint32_t* fstart;        // [B+1] first sorted pair of frame b (kept pairs of the frames before it)
  uint32_t* schunk_first;  // [B+1] first pair chunk of frame b
  uint4* schunk;           // [schunk_max] pair chunk k: (first pair, end, frame, first pair of the frame)
  uint2* schunk_frame;     // [schunk_max] pair chunk k: its frame's chunks [x, y)
  uint32_t* cnt;           // [schunk_max][kSortBins] digit counts of chunk k in a pass
  uint4* vtile;            // [vtile_max] voxel tile t: (first pair, end, frame, first pair of the frame)
  uint32_t* vt_first;      // [B+1] first voxel tile of frame b
  uint32_t* hcount;        // [vtile_max] voxels (heads) of tile t
  uint32_t* hpre;          // [vtile_max + 1] voxels of the tiles before t (all frames)
  uint32_t* mtile;         // [N / kMeanTile + 2] tile of voxel i * kMeanTile (the mean's blocks)
  int64_t* trow;           // [vtile_max] output row of tile t's first voxel; -1 in a frame over the cap
  uint32_t* keys[2];       // [N] each: ping-pong buffers of the radix passes
  uint32_t* vals[2];       // the pair's record: its place in compact (point) order
  // records of the kept points in compact order, written by the compaction:
  // rec_words words each (1 + C rounded up to an even count: 4, 6, 8 or 10),
  // word 0 the point index, then x', y', z' (Eq. 6) and the raw features
  // 3..C-1 as float bits
  uint32_t* rec;           // [N][rec_words]
  int32_t rec_words;
  // per voxel, at slot vtile[t].x + j for voxel j of tile t
  uint32_t* hpos;          // [N] first sorted pair of the voxel
  uint32_t* hplace;        // [N] its place (its first point: places follow point order)
  uint32_t* capbits;       // frames with more pairs than max_voxels: three regions of N / 32 + B + 1
                           // words (first-place bits, set by the heads kernel; kept flags in slot
                           // order; the flag words' prefix; frame b from word fstart[b] / 32 + b of
                           // each), then [vtile_max] tiles' voxel counts (frame b from its first tile;
                           // frames whose tables exceed LDS)
  uint32_t* vox_off;       // [B+1] voxels of the frames before b
  // sizes
  int32_t fchunk_points;   // points per filter chunk (a multiple of kWaveTile, <= kMaxChunkPoints)
  int32_t fchunk_words;    // fchunk_points / 32
  int32_t fchunk_max;      // bound on filter chunks: ceil(N / fchunk_points) + kWaves * B
  int32_t filter_grid;     // ceil(fchunk_max / kWaves) workgroups, one chunk per wave
  // the filter's dynamic LDS: pose rows, ROI records (six rows of
  // lds_roi_cap floats from float offset lds_roi), budget-mask words (from
  // word offset lds_bm), the frame's cell row (lds_cell_cap words from word
  // offset lds_cell: a zero word, then the cell words); a cap of 0 means
  // "not staged"
  int32_t lds_pose_cap, lds_roi_cap, lds_bm_cap, lds_cell_cap, lds_roi, lds_bm, lds_cell, lds_dyn_bytes;
  int32_t lds_wmask;       // the filter's own per-cell ROI words (several words per cell), word offset; -1: none
  int32_t schunk_max;      // bound on pair chunks: min(N / (kSortTile / 2) + B, kMaxFrameChunks * B) + 1
  int32_t vtile_max;       // bound on voxel tiles: N / kVoxTile + B + 1
  int32_t mean_grid;
};

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ uint64_t lanemask_lt() {
  uint32_t l = __lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Set lanes of m below this lane (mbcnt: the popcount of m & lanemask_lt()).
__device__ __forceinline__ uint32_t count_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Work unit of workgroup b when n units are dealt to the eight XCDs in
// contiguous blocks: workgroups go to XCD b % 8 in turn, so XCD x takes
// units [x * per, (x + 1) * per) in order and neighbouring units share an
// L2 (their partial-line writes merge there; their common reads hit there).
// Returns n or more for a workgroup with no unit; the grid must hold at
// least 8 * ceil(n / 8) workgroups.
__device__ __forceinline__ uint32_t xcd_block_unit(uint32_t b, uint32_t n) {
  const uint32_t per = (n + 7u) / 8u;
  return b / 8u < per ? (b % 8u) * per + b / 8u : n;
}

__device__ __forceinline__ void raise_fault(WsHeader* h, int32_t bits) {
  __hip_atomic_fetch_or(&h->fault, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inclusive prefix sum over the 64 lanes of a wave (every lane active), in
// DPP moves instead of LDS permutes: shifts by 1, 2, 4 and 8 lanes inside
// each row of 16 lanes (a lane whose source lies before its row adds 0),
// then the last lane of rows 0 and 2 added to rows 1 and 3, then lane 31 to
// rows 2 and 3 (rows left out of a move's row mask add 0).
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Largest value over the 64 lanes of a wave (every lane active), by the
// same DPP moves (lanes left out of a move see 0, which leaves a maximum of
// unsigned values unchanged); the last lane's result is every lane's.
__device__ __forceinline__ uint32_t wave_max(uint32_t x) {
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false));  // row_shr:1
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false));  // row_shr:2
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false));  // row_shr:4
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false));  // row_shr:8
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false));  // row_bcast:15
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Exclusive prefix over the workgroup (WAVES wave64s, all threads must
// call); s_tmp holds WAVES words of LDS.  Returns the prefix, sets total.
template <int WAVES = kWaves>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_tmp, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t x = wave_inclusive_sum(v);
  if (lane == 63) s_tmp[wave] = x;
  __syncthreads();
  uint32_t wpre = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    uint32_t t = s_tmp[w];
    wpre += (w < wave) ? t : 0u;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return wpre + x - v;
}

// Exclusive prefix sums of two values per thread over the workgroup (one
// barrier pair for both); s_tmp holds 2 * WAVES words.
template <int WAVES>
__device__ __forceinline__ uint2 block_exclusive_scan2(uint32_t a, uint32_t b, uint32_t* s_tmp, uint2& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t xa = wave_inclusive_sum(a), xb = wave_inclusive_sum(b);
  if (lane == 63) {
    s_tmp[wave] = xa;
    s_tmp[WAVES + wave] = xb;
  }
  __syncthreads();
  uint32_t pa = 0, pb = 0, ta = 0, tb = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    const uint32_t u = s_tmp[w], v = s_tmp[WAVES + w];
    pa += (w < wave) ? u : 0u;
    pb += (w < wave) ? v : 0u;
    ta += u;
    tb += v;
  }
  __syncthreads();
  total = make_uint2(ta, tb);
  return make_uint2(pa + xa - a, pb + xb - b);
}

// kLds: the frame starts are built in LDS (B <= kSegLdsFrames) and copied
// out at the end; otherwise in the workspace directly.  (One address space per
// instance: a pointer that may be either compiles to generic instructions,
// whose waits cover both kinds of access.)
constexpr size_t kSpareTileBytes = 1024;  // one wave's 16-byte loads
constexpr uint32_t kNoFrame = 0xffffffffu;  // wg_frame of a filter workgroup past the last chunk

// Largest b in [0, B-1] with first[b] <= k (first[] non-decreasing): the
// frame of chunk k, skipping frames without chunks.
__device__ __forceinline__ int32_t frame_of_chunk(const uint32_t* first, int32_t B, uint32_t k) {
  int32_t lo = 0, hi = B - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (first[mid] <= k)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// Pairs per chunk of a frame of n kept pairs: at most kMaxFrameChunks
// chunks, each a whole number of scatter tiles, at least min_tiles of them;
// half tiles (the scatter ranks a chunk of at most half a tile four rounds
// per wave instead of eight) for a frame of at most kHalfTileFramePairs
// pairs when the call allows them (half: its half-tile chunks fit one round
// of the scatter's resident workgroups).
__device__ __forceinline__ uint32_t frame_chunk_pairs(uint32_t n, uint32_t min_tiles, bool half) {
  if (half && n <= (uint32_t)kHalfTileFramePairs) return (uint32_t)kSortTile / 2u;
  uint32_t ch = (n + kMaxFrameChunks - 1) / kMaxFrameChunks;
  ch = (ch + kSortTile - 1) / kSortTile * kSortTile;
  return max(ch, min_tiles * (uint32_t)kSortTile);
}

// Scatter tiles per pair chunk at least: one, unless the call's chunks (at
// most K / (tiles * kSortTile) + B) would not all fit one round of the
// scatter's resident workgroups; then as many as make them fit (at most 8).
__device__ __forceinline__ uint32_t chunk_min_tiles(uint32_t K, int32_t B) {
  constexpr uint32_t kResident = kScatterPerCu * kCus;
  if ((uint32_t)B >= kResident) return 1u;
  const uint32_t room = (kResident - (uint32_t)B) * (uint32_t)kSortTile;
  return min(max((K + room - 1) / room, 1u), 8u);
}

// Whether the call's frames of at most kHalfTileFramePairs pairs take
// half-tile chunks: all the call's pairs in half tiles (plus one partial
// chunk per frame) fit one round of the scatter's resident workgroups.
__device__ __forceinline__ bool half_tile_chunks(uint32_t K, int32_t B) {
  constexpr uint32_t kResident = kScatterPerCu * kCus;
  return (uint64_t)(K + kSortTile / 2 - 1) / (kSortTile / 2) + (uint64_t)B <= kResident;
}

// Point frame offset b clamped into [0, N].
__device__ __forceinline__ uint32_t point_offset(const Config& c, int32_t b) {
  return (uint32_t)min(max(c.frame_off[b], (int64_t)0), (int64_t)c.N);
}

// Points [lo, hi) of filter chunk k of frame b (chunk j = k - first[b] of
// the frame); empty for invalid offsets.
__device__ __forceinline__ void filter_chunk_points(const Config& c, int32_t b, uint32_t k, uint32_t& lo,
                                                    uint32_t& hi) {
  const uint32_t f0 = point_offset(c, b), f1 = max(point_offset(c, b + 1), f0);
  const uint64_t l = (uint64_t)f0 + (uint64_t)(k - c.fchunk_first[b]) * (uint32_t)c.fchunk_points;
  lo = (uint32_t)min(l, (uint64_t)f1);
  hi = (uint32_t)min(l + (uint32_t)c.fchunk_points, (uint64_t)f1);
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

// The out-of-ROI keep draw of Alg. 1 (rate rho_out): point i is drawn when
// the top 24 bits of the (i + 1)-th output of a SplitMix64 generator (Steele,
// Lea and Flood 2014) whose state starts at the seed lie below the threshold
// round(rho_out * 2^24).  The generator advances its state by the golden-
// ratio increment and mixes it with two xor-shift-multiply rounds.
__device__ __forceinline__ bool background_draw(const Config& c, uint32_t i) {
  uint64_t z = c.bg_seed + ((uint64_t)i + 1u) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return (uint32_t)(z >> 40) < c.bg_thr;
}

// Grid coordinate on one axis; false when outside [0, D) or not a number.
__device__ __forceinline__ bool quantize_axis(float p, float mn, float vs, float Df, int32_t& i) {
  float f = (p - mn) / vs;
  bool ok = (f >= 0.0f) && (f < Df);
  i = ok ? (int32_t)f : 0;
  return ok;
}

// Conservative cell rectangle [x0, x1] x [y0, y1] of one ROI; empty when x0 > x1.
__device__ __forceinline__ void roi_cell_rect(const Config& c, const mmbev_roi_t& r, int16_t* out) {
  const double u = 1.0 / 16777216.0;  // fp32 unit roundoff
  double cx = r.cx, cy = r.cy, co = r.cos_yaw, si = r.sin_yaw, ex = r.ext_x, ey = r.ext_y;
  int32_t x0 = 0, x1 = c.ncx - 1, y0 = 0, y1 = c.ncy - 1;
  bool finite = isfinite(cx) && isfinite(cy) && isfinite(co) && isfinite(si) && isfinite(ex) && isfinite(ey);
  if (finite && (ex < 0.0 || ey < 0.0)) {
    x0 = 1;  // |l| <= negative extent never holds
    x1 = 0;
  } else if (finite) {
    double n2 = co * co + si * si;
    double hx = (fabs(co) * ex + fabs(si) * ey) / n2;
    double hy = (fabs(si) * ex + fabs(co) * ey) / n2;
    double mag = fabs(cx) + fabs(cy) + hx + hy;
    for (int d = 0; d < 2; ++d) mag += fabs((double)c.mn[d]) + (double)c.vs[d] * (double)c.Df[d];
    double pad = 1e-3 + 16.0 * u * mag;
    if (isfinite(hx) && isfinite(hy) && isfinite(pad)) {
      int32_t lim[2][2];
      double ctr[2] = {cx, cy}, half[2] = {hx, hy};
      for (int d = 0; d < 2; ++d) {
        double lo = (ctr[d] - half[d] - pad - (double)c.mn[d]) / (double)c.vs[d];
        double hi = (ctr[d] + half[d] + pad - (double)c.mn[d]) / (double)c.vs[d];
        double D = (double)c.Df[d];
        lo = fmin(fmax(floor(lo) - (double)c.cell_pad, -1.0), D);
        hi = fmin(fmax(floor(hi) + (double)c.cell_pad, -1.0), D);
        int32_t ilo = (int32_t)lo, ihi = (int32_t)hi;
        if (ihi < 0 || ilo >= (int32_t)D) {
          lim[d][0] = 1;
          lim[d][1] = 0;
        } else {
          ilo = max(ilo, 0);
          ihi = min(ihi, (int32_t)D - 1);
          lim[d][0] = ilo >> c.cell_shift;
          lim[d][1] = ihi >> c.cell_shift;
        }
      }
      x0 = lim[0][0];
      x1 = lim[0][1];
      y0 = lim[1][0];
      y1 = lim[1][1];
    }
  }
  out[0] = (int16_t)x0;
  out[1] = (int16_t)x1;
  out[2] = (int16_t)y0;
  out[3] = (int16_t)y1;
}

// Filter chunks of a frame of n points: whole workgroups of kWaves chunks.
__device__ __forceinline__ uint32_t frame_chunks(uint32_t n, uint32_t P) {
  return (n + P - 1) / P + kWaves - 1 - ((n + P - 1) / P + kWaves - 1) % kWaves;
}

// Fault bits of frame f's offsets (f <= B; on, rn: frame min(f + 1, B)'s):
// point offsets must start at 0, end at N and not decrease; ROI offsets must
// start at 0, end at R, not decrease and give no frame more than
// max_rois_per_frame ROIs.
__device__ __forceinline__ int32_t offset_faults(const Config& c, int f, int64_t o, int64_t on, int32_t ro,
                                                 int32_t rn) {
  int32_t bad = 0;
  if (f == 0 && o != 0) bad |= MMBEV_FAULT_POINT_OFFSETS;
  if (f == c.B && o != (int64_t)c.N) bad |= MMBEV_FAULT_POINT_OFFSETS;
  if (f < c.B && on < o) bad |= MMBEV_FAULT_POINT_OFFSETS;
  if (f == 0 && ro != 0) bad |= MMBEV_FAULT_ROI_OFFSETS;
  if (f == c.B && ro != c.R) bad |= MMBEV_FAULT_ROI_OFFSETS;
  if (f < c.B && (rn < ro || rn - ro > c.max_rois)) bad |= MMBEV_FAULT_ROI_OFFSETS;
  return bad;
}

}  // namespace mmbev
