// C ABI of libmmbev: argument validation, launch configuration, workspace
// carve-up and the stream-ordered launch sequence of one call.  No
// allocation, no host synchronisation, no state kept between calls.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "launch.hpp"

using namespace mmbev;

namespace {

int bits_for(uint64_t maxval) {
  int b = 0;
  while (b < 64 && (maxval >> b) != 0) ++b;
  return b;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Words of a kept-point record: the point index and C features, rounded up to
// an even count (8-byte aligned records: 16, 24, 32 or 40 bytes).
int32_t record_words(int32_t C) { return (2 + C) & ~1; }

// Workspace of the connected-component proposer.
struct CcPlan {
  int64_t rows, cells, ncell, Wx, Wy, nwords, nblocks;
  size_t off_occ, off_wpre, off_bsum, off_parent, off_cnt, off_rcell, total;
};

mmbev_status_t cc_plan(const mmbev_grid_t* g, const mmbev_cluster_params_t* prm, CcPlan* p) {
  if (!g || !prm) return MMBEV_ERR_INVALID_ARG;
  for (int d = 0; d < 3; ++d)
    if (g->dims[d] < 1 || g->dims[d] >= (1 << 24)) return MMBEV_ERR_INVALID_ARG;
  if (g->max_voxels < 1 || g->num_frames < 1 || g->num_frames > 65535) return MMBEV_ERR_INVALID_ARG;
  if (prm->connectivity != 4 && prm->connectivity != 8) return MMBEV_ERR_INVALID_ARG;
  if (prm->cell_shift < 0 || prm->cell_shift > 8 || prm->min_cells < 1 || prm->reserved != 0)
    return MMBEV_ERR_INVALID_ARG;
  if ((uint64_t)g->num_frames * (uint64_t)g->max_voxels > (uint64_t)INT32_MAX) return MMBEV_ERR_UNSUPPORTED;
  const int64_t side = (int64_t)1 << prm->cell_shift;
  p->Wx = (g->dims[0] + side - 1) / side;
  p->Wy = (g->dims[1] + side - 1) / side;
  p->ncell = p->Wx * p->Wy;
  p->cells = p->ncell * g->num_frames;
  if (p->cells >= kCcMaxCells) return MMBEV_ERR_UNSUPPORTED;
  p->rows = (int64_t)g->num_frames * g->max_voxels;
  p->nwords = ((p->cells + 31) / 32 + 63) / 64 * 64;  // whole 256-byte blocks
  p->nblocks = (p->nwords + kBlock * 16 - 1) / (kBlock * 16);
  size_t off = 256;  // CcHeader
  p->off_occ = off;
  off += align256((size_t)p->nwords * 8);  // occ, then rootbits
  p->off_wpre = off;
  off += align256((size_t)p->nwords * 4);
  p->off_bsum = off;
  off += align256((size_t)p->nblocks * 4);
  p->off_parent = off;
  off += align256((size_t)p->cells * 4);
  p->off_cnt = off;
  off += align256((size_t)p->cells * 4);
  p->off_rcell = off;
  off += align256((size_t)p->rows * 4);
  p->total = off;
  return MMBEV_OK;
}

struct Plan {
  int64_t N;
  int32_t B, S, C, M, cap, max_rois, W;
  int32_t cell_shift, ncx, ncy, ncells;
  int32_t kb, passes, dbits;
  int64_t fchunk_points, fchunk_max, filter_grid, schunk_max, vtile_max, mean_grid;
  size_t off_hdr, off_cellmask, off_cellany, off_budgetmask, off_fchunk_first, off_fbits, off_fcount, off_fchunk_lo, off_fchunk_frame, off_wgframe, off_spare, off_fprefix,
      off_fstart, off_schunk_first, off_schunk, off_schunk_frame, off_cnt, off_vtile, off_vt_first, off_hcount, off_hpre, off_mtile, off_trow, off_keys[2], off_vals[2], off_rec,
      off_hpos, off_hplace, off_capbits, off_voxoff, total;
};

mmbev_status_t make_plan(const mmbev_grid_t* g, int64_t N, int32_t max_rois, int32_t C, Plan* p) {
  if (!g) return MMBEV_ERR_INVALID_ARG;
  if (N < 0 || max_rois < 0) return MMBEV_ERR_INVALID_ARG;
  if (C < 3 || C > 8) return MMBEV_ERR_INVALID_ARG;
  for (int d = 0; d < 3; ++d) {
    if (!std::isfinite(g->range_min[d]) || !std::isfinite(g->voxel_size[d]) || !(g->voxel_size[d] > 0.0f))
      return MMBEV_ERR_INVALID_ARG;
    if (g->dims[d] < 1 || g->dims[d] >= (1 << 24)) return MMBEV_ERR_INVALID_ARG;
  }
  if (g->max_points < 1 || g->max_points > 64) return MMBEV_ERR_INVALID_ARG;
  if (g->max_voxels < 1) return MMBEV_ERR_INVALID_ARG;
  if (g->num_sweeps < 1 || g->num_sweeps > 255) return MMBEV_ERR_INVALID_ARG;
  if (g->num_frames < 1 || g->num_frames > 65535) return MMBEV_ERR_INVALID_ARG;
  if (N >= (int64_t)1 << 30) return MMBEV_ERR_UNSUPPORTED;
  if (max_rois > 1024) return MMBEV_ERR_UNSUPPORTED;
  const uint64_t cells = (uint64_t)g->dims[0] * (uint64_t)g->dims[1] * (uint64_t)g->dims[2];
  if (cells > ((uint64_t)1 << 32)) return MMBEV_ERR_UNSUPPORTED;
  if ((uint64_t)g->num_frames * (uint64_t)g->max_voxels > (uint64_t)INT32_MAX) return MMBEV_ERR_UNSUPPORTED;

  p->N = N;
  p->B = g->num_frames;
  p->S = g->num_sweeps;
  p->C = C;
  p->M = g->max_points;
  p->cap = g->max_voxels;
  p->max_rois = max_rois;
  p->W = std::max(1, (max_rois + 31) / 32);
  int cs = 0;
  while ((((int64_t)g->dims[0] + (1 << cs) - 1) >> cs) > kMaxCellSide ||
         (((int64_t)g->dims[1] + (1 << cs) - 1) >> cs) > kMaxCellSide)
    ++cs;
  p->cell_shift = cs;
  p->ncx = (int32_t)(((int64_t)g->dims[0] + (1 << cs) - 1) >> cs);
  p->ncy = (int32_t)(((int64_t)g->dims[1] + (1 << cs) - 1) >> cs);
  p->ncells = p->ncx * p->ncy;
  p->kb = std::max(1, bits_for(cells - 1));
  p->passes = (p->kb + kMaxDigitBits - 1) / kMaxDigitBits;
  p->dbits = (p->kb + p->passes - 1) / p->passes;

  const int64_t n1 = std::max<int64_t>(N, 1);
  // filter chunks: about kFilterWaveTarget of them over the whole input (a
  // few per resident wave), a multiple of the wave tile and at most
  // kMaxChunkPoints points (a wave keeps its chunk's bitmap in LDS); a frame
  // adds at most one partial chunk and up to kWaves - 1 empty ones (its
  // chunks fill whole filter workgroups)
  {
    const int64_t target = kFilterWaveTarget > 2 * (int64_t)p->B ? kFilterWaveTarget - p->B : kFilterWaveTarget;
    int64_t P = (N + target - 1) / target;
    P = std::max<int64_t>(kWaveTile, (P + kWaveTile - 1) / kWaveTile * kWaveTile);
    // chunks of one wave tile only while two-tile chunks would leave too few
    // waves to fill the chip (measured: 8 frames of 347,200 points 147.5 ->
    // 142 us per call with two tiles; one frame is faster with one)
    if (P < 2 * kWaveTile && N >= (int64_t)2 * kWaveTile * kFilterMinWaves) P = 2 * kWaveTile;
    P = std::min<int64_t>(P, kMaxChunkPoints);
    p->fchunk_points = P;
    p->fchunk_max = (N + P - 1) / P + (int64_t)kWaves * p->B;  // each frame rounded up to whole workgroups
    p->filter_grid = std::max<int64_t>(1, (p->fchunk_max + kWaves - 1) / kWaves);
  }
  p->schunk_max = std::min<int64_t>(N / (kSortTile / 2) + p->B, (int64_t)kMaxFrameChunks * p->B) + 1;  // half-tile chunks too
  p->vtile_max = N / kVoxTile + p->B + 1;
  p->mean_grid = std::min<int64_t>((n1 + kMeanTile - 1) / kMeanTile, 2048);  // measured best (1536 and 4096 slower)
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align256(o + bytes);
    return at;
  };
  p->off_hdr = take(sizeof(WsHeader));
  p->off_cellmask = take((size_t)p->B * p->ncells * p->W * 4);
  p->off_cellany = p->W > 1 ? take((size_t)p->B * p->ncells * 4) : p->off_cellmask;
  p->off_budgetmask = take((size_t)p->B * p->S * p->W * 4);
  p->off_fchunk_first = take((size_t)(p->B + 1) * 4);
  p->off_fbits = take((size_t)p->fchunk_max * (p->fchunk_points / 32) * 4);
  p->off_fcount = take((size_t)p->fchunk_max * 4);
  p->off_fchunk_lo = take((size_t)p->fchunk_max * 4);
  p->off_fchunk_frame = take((size_t)p->fchunk_max * 4);
  p->off_wgframe = take((size_t)p->filter_grid * 4);
  p->off_spare = take(kSpareTileBytes);
  p->off_fprefix = take((size_t)(p->fchunk_max + 1) * 4);
  p->off_fstart = take((size_t)(p->B + 1) * 4);
  p->off_schunk_first = take((size_t)(p->B + 1) * 4);
  p->off_schunk = take((size_t)p->schunk_max * 16);
  p->off_schunk_frame = take((size_t)p->schunk_max * 8);
  p->off_cnt = take((size_t)p->schunk_max * kSortBins * 4);
  p->off_vtile = take((size_t)p->vtile_max * 16);
  p->off_vt_first = take((size_t)(p->B + 1) * 4);
  p->off_hcount = take((size_t)p->vtile_max * 4);
  p->off_hpre = take((size_t)(p->vtile_max + 1) * 4);
  p->off_mtile = take(((size_t)n1 / kMeanTile + 2) * 4);
  p->off_trow = take((size_t)p->vtile_max * 8);
  for (int q = 0; q < 2; ++q) {
    p->off_keys[q] = take((size_t)n1 * 4);
    p->off_vals[q] = take((size_t)n1 * 4);
  }
  p->off_rec = take((size_t)n1 * 4 * (size_t)record_words(p->C));
  p->off_hpos = take((size_t)n1 * 4);
  p->off_hplace = take((size_t)n1 * 4);
  p->off_capbits = take((3 * ((size_t)n1 / 32 + p->B + 1) + (size_t)p->vtile_max + 1) * 4);
  p->off_voxoff = take((size_t)(p->B + 1) * 4);
  p->total = o;
  return MMBEV_OK;
}

}  // namespace

extern "C" {

int32_t mmbev_abi_version(void) { return MMBEV_ABI_VERSION; }

const char* mmbev_status_string(mmbev_status_t s) {
  switch (s) {
    case MMBEV_OK: return "ok";
    case MMBEV_ERR_INVALID_ARG: return "invalid argument";
    case MMBEV_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case MMBEV_ERR_UNSUPPORTED: return "size beyond the supported limits";
    case MMBEV_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

size_t mmbev_roi_voxelize_workspace_bytes(const mmbev_grid_t* grid, int64_t num_points, int32_t num_features,
                                          int32_t max_rois_per_frame) {
  Plan p;
  if (make_plan(grid, num_points, max_rois_per_frame, num_features, &p) != MMBEV_OK) return 0;
  return p.total;
}

mmbev_status_t mmbev_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || ((uintptr_t)workspace & 255)) return MMBEV_ERR_WORKSPACE;
  if (workspace_bytes == 0) return MMBEV_OK;
  return launch_fill_zero(workspace, workspace_bytes, (hipStream_t)stream) == hipSuccess ? MMBEV_OK
                                                                                           : MMBEV_ERR_HIP;
}

}  // extern "C"

namespace {

// Records the caller's profiling events between launches (none when absent).
struct EventTrail {
  void* const* events = nullptr;
  int32_t n = 0, used = 0;
  hipError_t mark(hipStream_t s) {
    if (used >= n) return hipSuccess;
    return hipEventRecord((hipEvent_t)events[used++], s);
  }
};

// round(rho * 2^24) clamped to [0, 2^24]; NaN and rho <= 0 give 0.
uint32_t keep_threshold(float rho) {
  const double t = (double)rho * 16777216.0;
  if (!(t > 0.0)) return 0;
  if (t >= 16777216.0) return 1u << 24;
  return (uint32_t)std::floor(t + 0.5);
}

// Every argument check of a call except the workspace's; fills the plan.
mmbev_status_t check_args(const mmbev_points_t* points, const uint8_t* sweep_ids, const float* sweep_poses,
                          const mmbev_rois_t* rois, const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid,
                          const mmbev_options_t* opt, int32_t* out_coords, int32_t* out_counts, float* out_feats,
                          int32_t* out_point_idx, int64_t* out_voxel_offsets, Plan* p) {
  if (!points || !rois || !grid) return MMBEV_ERR_INVALID_ARG;
  if (opt && opt->reserved != 0) return MMBEV_ERR_INVALID_ARG;
  const int64_t N = points->num_points;
  mmbev_status_t st = make_plan(grid, N, rois->max_rois_per_frame, points->num_features, p);
  if (st != MMBEV_OK) return st;
  if (points->stride < N || points->stride >= ((int64_t)1 << 40)) return MMBEV_ERR_INVALID_ARG;
  if (N > 0 && (!points->feat || !sweep_ids)) return MMBEV_ERR_INVALID_ARG;
  if (!points->frame_offsets || !sweep_poses || !rois->frame_offsets) return MMBEV_ERR_INVALID_ARG;
  if (rois->num_rois < 0) return MMBEV_ERR_INVALID_ARG;
  if (rois->num_rois > 0 && (!rois->boxes || !roi_sweep_budget)) return MMBEV_ERR_INVALID_ARG;
  if (!out_coords || !out_counts || !out_feats || !out_point_idx || !out_voxel_offsets)
    return MMBEV_ERR_INVALID_ARG;
  return MMBEV_OK;
}

mmbev_status_t voxelize(const mmbev_points_t* points, const uint8_t* sweep_ids, const float* sweep_poses,
                        const mmbev_rois_t* rois, const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid,
                        const mmbev_options_t* opt, int32_t* out_coords, int32_t* out_counts, float* out_feats,
                        int32_t* out_point_idx, int64_t* out_voxel_offsets, void* workspace,
                        size_t workspace_bytes, void* stream, EventTrail& ev) {
  Plan p;
  mmbev_status_t st = check_args(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, opt, out_coords,
                                 out_counts, out_feats, out_point_idx, out_voxel_offsets, &p);
  if (st != MMBEV_OK) return st;
  const int64_t N = points->num_points;
  if (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < p.total) return MMBEV_ERR_WORKSPACE;

  Config c;
  std::memset(&c, 0, sizeof(c));
  c.feat = points->feat;
  c.sweep = sweep_ids;
  c.poses = sweep_poses;
  c.frame_off = points->frame_offsets;
  c.rois = rois->boxes;
  c.roi_off = rois->frame_offsets;
  c.budget = roi_sweep_budget;
  c.stride = points->stride;
  c.N = (int32_t)N;
  c.C = p.C;
  c.B = p.B;
  c.S = p.S;
  c.M = p.M;
  c.cap = p.cap;
  c.R = rois->num_rois;
  c.max_rois = p.max_rois;
  c.W = p.W;
  c.bg_thr = opt ? keep_threshold(opt->out_of_roi_keep_rate) : 0u;
  c.bg_seed = opt ? opt->seed : 0u;
  for (int d = 0; d < 3; ++d) {
    c.mn[d] = grid->range_min[d];
    c.vs[d] = grid->voxel_size[d];
    c.Df[d] = (float)grid->dims[d];
    c.inv_vs[d] = (float)(1.0 / (double)grid->voxel_size[d]);
    c.nmin_v[d] = (float)(-(double)grid->range_min[d] / (double)grid->voxel_size[d]);
  }
  {
    // the approximate cell lookup x'*(1/v) - min/v is off from the exact
    // (x' - min)/v by at most (2|min/v| + D) * 2^-22 voxels for points that
    // can be kept; pad every ROI's cell rectangle by one voxel more than that
    double err = 0.0;
    for (int d = 0; d < 2; ++d)
      err = std::max(err, (2.0 * std::fabs((double)grid->range_min[d] / (double)grid->voxel_size[d]) +
                           (double)grid->dims[d]) * std::ldexp(1.0, -22));
    c.cell_pad = 2 + (int32_t)std::ceil(err);
  }
  c.Dx = (uint32_t)grid->dims[0];
  c.Dy = (uint32_t)grid->dims[1];
  c.Dz = (uint32_t)grid->dims[2];
  c.cell_shift = p.cell_shift;
  c.ncx = p.ncx;
  c.ncy = p.ncy;
  c.ncells = p.ncells;
  c.kb = p.kb;
  c.passes = p.passes;
  c.dbits = p.dbits;
  c.vec = (((uintptr_t)points->feat & 15) == 0 && (points->stride & 3) == 0 && ((uintptr_t)sweep_ids & 3) == 0) ? 1
                                                                                                                : 0;
  c.out_coords = out_coords;
  c.out_counts = out_counts;
  c.out_feats = out_feats;
  c.out_point_idx = out_point_idx;
  c.out_voxel_offsets = out_voxel_offsets;
  char* ws = (char*)workspace;
  c.hdr = (WsHeader*)(ws + p.off_hdr);
  c.cellmask = (uint32_t*)(ws + p.off_cellmask);
  c.cellany = (uint32_t*)(ws + p.off_cellany);
  c.budgetmask = (uint32_t*)(ws + p.off_budgetmask);
  c.fchunk_first = (uint32_t*)(ws + p.off_fchunk_first);
  c.fbits = (uint32_t*)(ws + p.off_fbits);
  c.fcount = (uint32_t*)(ws + p.off_fcount);
  c.fchunk_lo = (uint32_t*)(ws + p.off_fchunk_lo);
  c.fchunk_frame = (uint32_t*)(ws + p.off_fchunk_frame);
  c.wg_frame = (uint32_t*)(ws + p.off_wgframe);
  c.spare_tile = (const float*)(ws + p.off_spare);
  c.fprefix = (uint32_t*)(ws + p.off_fprefix);
  c.fstart = (uint32_t*)(ws + p.off_fstart);
  c.schunk_first = (uint32_t*)(ws + p.off_schunk_first);
  c.schunk = (uint4*)(ws + p.off_schunk);
  c.schunk_frame = (uint2*)(ws + p.off_schunk_frame);
  c.cnt = (uint32_t*)(ws + p.off_cnt);
  c.vtile = (uint4*)(ws + p.off_vtile);
  c.vt_first = (uint32_t*)(ws + p.off_vt_first);
  c.hcount = (uint32_t*)(ws + p.off_hcount);
  c.hpre = (uint32_t*)(ws + p.off_hpre);
  c.mtile = (uint32_t*)(ws + p.off_mtile);
  c.trow = (int64_t*)(ws + p.off_trow);
  for (int q = 0; q < 2; ++q) {
    c.keys[q] = (uint32_t*)(ws + p.off_keys[q]);
    c.vals[q] = (uint32_t*)(ws + p.off_vals[q]);
  }
  c.rec = (uint32_t*)(ws + p.off_rec);
  c.rec_words = record_words(p.C);
  c.hpos = (uint32_t*)(ws + p.off_hpos);
  c.hplace = (uint32_t*)(ws + p.off_hplace);
  c.capbits = (uint32_t*)(ws + p.off_capbits);
  c.vox_off = (uint32_t*)(ws + p.off_voxoff);
  c.fchunk_points = (int32_t)p.fchunk_points;
  c.fchunk_words = (int32_t)(p.fchunk_points / 32);
  c.fchunk_max = (int32_t)p.fchunk_max;
  c.filter_grid = (int32_t)p.filter_grid;
  // one frame per filter workgroup: its poses, ROI records, budget masks and cell words
  c.lds_pose_cap = p.S <= kMaxPoseLds ? p.S : 0;
  c.lds_roi_cap = std::max(1, std::min(p.max_rois, kMaxLdsRois));
  c.lds_bm_cap = p.S * p.W <= kMaxLdsBudgetWords ? p.S * p.W : 0;
  c.lds_cell_cap = p.ncells <= kMaxLdsCells ? p.ncells + 1 : 0;  // a zero word, then the cells
  c.lds_roi = c.lds_pose_cap * 12;
  c.lds_bm = c.lds_roi + 6 * c.lds_roi_cap;
  c.lds_cell = c.lds_bm + c.lds_bm_cap;
  // every table of a frame in LDS and a thread per frame: each filter
  // workgroup lays out the call and builds its frame's tables itself, and the
  // staging kernel is not launched; with several ROI words per cell only for
  // a few frames whose cells' words fit in LDS too (they take a larger share
  // of the filter's LDS, which a few frames' workgroups can afford)
  const bool fits = p.B <= kFuseFrames && c.lds_pose_cap == p.S && c.lds_bm_cap == p.S * p.W &&
                    c.lds_cell_cap == p.ncells + 1 && c.lds_roi_cap >= p.max_rois && p.S <= kBlock;
  c.fuse_stage = fits && (p.W == 1 || (p.B <= kFuseWideFrames && (int64_t)p.ncells * p.W <= kFuseWordCap));
  c.lds_wmask = c.fuse_stage && p.W > 1 ? c.lds_cell + c.lds_cell_cap : -1;
  const int32_t lds_words = c.lds_wmask >= 0 ? c.lds_wmask + p.ncells * p.W : c.lds_cell + c.lds_cell_cap;
  c.lds_dyn_bytes = (int32_t)(((size_t)lds_words * 4 + 15) / 16 * 16);
  c.small_call = p.fchunk_max <= kSmallChunks;
  c.schunk_max = (int32_t)p.schunk_max;
  c.vtile_max = (int32_t)p.vtile_max;
  c.mean_grid = (int32_t)p.mean_grid;

  hipStream_t s = (hipStream_t)stream;
#define MMBEV_TRY(call)                                                   \
  do {                                                                    \
    if (ev.mark(s) != hipSuccess || (call) != hipSuccess) return MMBEV_ERR_HIP; \
  } while (0)

  MMBEV_TRY(c.fuse_stage ? hipSuccess : launch_stage(c, s));
  MMBEV_TRY(launch_filter(c, s));
  // sorted pairs ping-pong: keys compacted into [1], pass p writes [p % 2];
  // pass 0 reads no values, its value for each key is the key's compacted
  // position
  MMBEV_TRY(c.small_call ? hipSuccess : launch_segments(c, s));
  MMBEV_TRY(launch_compact(c, c.keys[1], s));
  for (int pass = 0; pass < c.passes; ++pass)
    MMBEV_TRY(launch_radix_pass(c, pass, c.keys[1 - pass % 2], pass == 0 ? nullptr : c.vals[1 - pass % 2],
                                c.keys[pass % 2], c.vals[pass % 2], s));
  const uint32_t* keys = c.keys[(c.passes - 1) % 2];
  const uint32_t* vals = c.vals[(c.passes - 1) % 2];
  MMBEV_TRY(launch_heads(c, keys, vals, s));
  MMBEV_TRY(launch_fincap(c, s));
  MMBEV_TRY(launch_mean(c, keys, vals, s));
#undef MMBEV_TRY
  if (ev.mark(s) != hipSuccess) return MMBEV_ERR_HIP;
  return MMBEV_OK;
}

}  // namespace

extern "C" {

mmbev_status_t mmbev_roi_voxelize(const mmbev_points_t* points, const uint8_t* sweep_ids, const float* sweep_poses,
                                  const mmbev_rois_t* rois, const uint8_t* roi_sweep_budget,
                                  const mmbev_grid_t* grid, int32_t* out_coords, int32_t* out_counts,
                                  float* out_feats, int32_t* out_point_idx, int64_t* out_voxel_offsets,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  EventTrail ev;
  return voxelize(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, nullptr, out_coords, out_counts,
                  out_feats, out_point_idx, out_voxel_offsets, workspace, workspace_bytes, stream, ev);
}

mmbev_status_t mmbev_roi_voxelize_profiled(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                           const float* sweep_poses, const mmbev_rois_t* rois,
                                           const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid,
                                           int32_t* out_coords, int32_t* out_counts, float* out_feats,
                                           int32_t* out_point_idx, int64_t* out_voxel_offsets, void* workspace,
                                           size_t workspace_bytes, void* stream, void* const* events,
                                           int32_t num_events, int32_t* events_recorded) {
  EventTrail ev;
  ev.events = events;
  ev.n = (events && num_events > 0) ? num_events : 0;
  mmbev_status_t st = voxelize(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, nullptr, out_coords,
                               out_counts, out_feats, out_point_idx, out_voxel_offsets, workspace, workspace_bytes,
                               stream, ev);
  if (events_recorded) *events_recorded = ev.used;
  return st;
}

mmbev_status_t mmbev_roi_voxelize_ex(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                     const float* sweep_poses, const mmbev_rois_t* rois,
                                     const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid,
                                     const mmbev_options_t* options, int32_t* out_coords, int32_t* out_counts,
                                     float* out_feats, int32_t* out_point_idx, int64_t* out_voxel_offsets,
                                     void* workspace, size_t workspace_bytes, void* stream, void* const* events,
                                     int32_t num_events, int32_t* events_recorded) {
  EventTrail ev;
  ev.events = events;
  ev.n = (events && num_events > 0) ? num_events : 0;
  mmbev_status_t st = voxelize(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, options, out_coords,
                               out_counts, out_feats, out_point_idx, out_voxel_offsets, workspace, workspace_bytes,
                               stream, ev);
  if (events_recorded) *events_recorded = ev.used;
  return st;
}

}  // extern "C"

// Workspace of mmbev_roi_voxelize_noalloc: MMBEV_NOALLOC_SCRATCH_BYTES of
// device memory that the code object holds on every device it is loaded on,
// until the process ends.  Host code never uses this name as an address (on
// the host it only stands for the symbol): the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[MMBEV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch[kMaxScratchDevices];  // device address of `scratch` on device d (null until set up)

// The current device's scratch.  On the first call on a device: its address,
// and its header cleared on `stream` by a kernel (the call counter starts at
// zero; every other field is rewritten by each call).
mmbev_status_t scratch_of_current_device(hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return MMBEV_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return MMBEV_ERR_HIP;
    if (launch_fill_zero(ptr, sizeof(WsHeader), stream) != hipSuccess) return MMBEV_ERR_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return MMBEV_OK;
}

}  // namespace

extern "C" {

mmbev_status_t mmbev_roi_voxelize_noalloc(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                          const float* sweep_poses, const mmbev_rois_t* rois,
                                          const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid,
                                          int32_t* out_coords, int32_t* out_counts, float* out_feats,
                                          int32_t* out_point_idx, int64_t* out_voxel_offsets, int32_t* out_fault,
                                          void* stream) {
  Plan p;
  mmbev_status_t st = check_args(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, nullptr, out_coords,
                                 out_counts, out_feats, out_point_idx, out_voxel_offsets, &p);
  if (st != MMBEV_OK) return st;
  if (p.total > (size_t)MMBEV_NOALLOC_SCRATCH_BYTES) return MMBEV_ERR_UNSUPPORTED;
  void* ws = nullptr;
  st = scratch_of_current_device((hipStream_t)stream, &ws);
  if (st != MMBEV_OK) return st;
  EventTrail ev;
  st = voxelize(points, sweep_ids, sweep_poses, rois, roi_sweep_budget, grid, nullptr, out_coords, out_counts,
                out_feats, out_point_idx, out_voxel_offsets, ws, (size_t)MMBEV_NOALLOC_SCRATCH_BYTES, stream, ev);
  if (st != MMBEV_OK) return st;
  if (out_fault && launch_copy_fault(reinterpret_cast<const WsHeader*>(ws), out_fault, (hipStream_t)stream) != hipSuccess)
    return MMBEV_ERR_HIP;
  return MMBEV_OK;
}

mmbev_status_t mmbev_scatter_to_bev(const int32_t* coords, const float* feats, const int64_t* voxel_offsets,
                                    int32_t num_features, const mmbev_grid_t* grid, float* bev_map,
                                    int32_t* fault, void* stream) {
  if (!grid || !coords || !feats || !voxel_offsets || !bev_map) return MMBEV_ERR_INVALID_ARG;
  if (((uintptr_t)coords & 15) != 0) return MMBEV_ERR_INVALID_ARG;
  if (num_features < 1 || num_features > 64) return MMBEV_ERR_INVALID_ARG;
  for (int d = 0; d < 3; ++d)
    if (grid->dims[d] < 1 || grid->dims[d] >= (1 << 24)) return MMBEV_ERR_INVALID_ARG;
  if (grid->max_voxels < 1 || grid->num_frames < 1 || grid->num_frames > 65535) return MMBEV_ERR_INVALID_ARG;
  const uint64_t plane = (uint64_t)grid->dims[0] * (uint64_t)grid->dims[1];
  if (plane * (uint64_t)grid->dims[2] > ((uint64_t)1 << 32)) return MMBEV_ERR_UNSUPPORTED;
  if ((uint64_t)grid->num_frames * (uint64_t)grid->max_voxels > (uint64_t)INT32_MAX) return MMBEV_ERR_UNSUPPORTED;
  BevConfig c{};
  c.coords = reinterpret_cast<const int4*>(coords);
  c.feats = feats;
  c.voff = voxel_offsets;
  c.map = bev_map;
  c.fault = fault;
  c.rows = (int64_t)grid->num_frames * grid->max_voxels;
  c.plane = plane;
  c.Dx = (uint32_t)grid->dims[0];
  c.Dy = (uint32_t)grid->dims[1];
  c.Dz = (uint32_t)grid->dims[2];
  c.B = grid->num_frames;
  c.C = num_features;
  c.max_voxels = grid->max_voxels;
  c.vec = ((uintptr_t)bev_map & 15) == 0;
  return launch_bev(c, (hipStream_t)stream) == hipSuccess ? MMBEV_OK : MMBEV_ERR_HIP;
}

size_t mmbev_voxel_clusters_workspace_bytes(const mmbev_grid_t* grid, const mmbev_cluster_params_t* params) {
  CcPlan p;
  return cc_plan(grid, params, &p) == MMBEV_OK ? p.total : 0;
}

mmbev_status_t mmbev_voxel_clusters(const int32_t* coords, const int32_t* counts, const int64_t* voxel_offsets,
                                    const mmbev_grid_t* grid, const mmbev_cluster_params_t* params,
                                    mmbev_cluster_t* out_clusters, int64_t* out_cluster_offsets,
                                    int32_t* out_voxel_labels, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  CcPlan p;
  const mmbev_status_t st = cc_plan(grid, params, &p);
  if (st != MMBEV_OK) return st;
  if (!coords || !counts || !voxel_offsets || !out_clusters || !out_cluster_offsets || !out_voxel_labels)
    return MMBEV_ERR_INVALID_ARG;
  if (((uintptr_t)coords & 15) != 0 || ((uintptr_t)out_clusters & 7) != 0) return MMBEV_ERR_INVALID_ARG;
  if (!workspace || ((uintptr_t)workspace & 255) != 0 || workspace_bytes < p.total) return MMBEV_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  CcConfig c{};
  c.coords = reinterpret_cast<const int4*>(coords);
  c.counts = counts;
  c.voff = voxel_offsets;
  c.out = out_clusters;
  c.out_off = out_cluster_offsets;
  c.labels = out_voxel_labels;
  c.hdr = (CcHeader*)ws;
  c.occ = (uint32_t*)(ws + p.off_occ);
  c.rootbits = c.occ + p.nwords;
  c.wpre = (uint32_t*)(ws + p.off_wpre);
  c.bsum = (uint32_t*)(ws + p.off_bsum);
  c.parent = (int32_t*)(ws + p.off_parent);
  c.cnt = (int32_t*)(ws + p.off_cnt);
  c.rcell = (int32_t*)(ws + p.off_rcell);
  c.rows = p.rows;
  c.cells = p.cells;
  c.nwords = (uint32_t)p.nwords;
  c.nblocks = (uint32_t)p.nblocks;
  c.Dx = (uint32_t)grid->dims[0];
  c.Dy = (uint32_t)grid->dims[1];
  c.Dz = (uint32_t)grid->dims[2];
  c.B = grid->num_frames;
  c.max_voxels = grid->max_voxels;
  c.ncell = (int32_t)p.ncell;
  c.Wx = (int32_t)p.Wx;
  c.Wy = (int32_t)p.Wy;
  c.shift = params->cell_shift;
  c.z_min = params->z_min;
  c.z_max = params->z_max;
  c.conn = params->connectivity;
  c.min_cells = params->min_cells;
  return launch_clusters(c, (hipStream_t)stream) == hipSuccess ? MMBEV_OK : MMBEV_ERR_HIP;
}

}  // extern "C"
