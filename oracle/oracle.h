/*
 * CPU ORACLE for ROI-aware multi-sweep voxelisation -- TEST INFRASTRUCTURE.
 *
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
 * call this code.  The product path (the HIP library) never links, loads or
 * calls it, and it shares no code, header or constant with that library.
 *
 * What it computes (paper: Sec. IV-D Eq. 6-7, Sec. IV-C Eq. 1, Sec. IV-F
 * Alg. 1; the out-of-ROI keep rate rho_out is zero unless a *_bg entry
 * point is given one), for every frame b:
 *   1. a point of sweep s >= num_sweeps is dropped;
 *   2. it is moved into the current frame, p' = R_{b,s} p + T_{b,s}
 *      (Eq. 6/7), in fp32 as the fused chain
 *        x' = fma(R00, x, fma(R01, y, fma(R02, z, T0)))   (rows 1, 2 alike);
 *   3. it is kept iff some ROI j of frame b admits its sweep (s < budget_j)
 *      and contains it in bird's-eye view (Alg. 1 keep test; ROI_L of Eq. 1
 *      read as a union of oriented boxes):
 *        dx = x' - cx, dy = y' - cy,
 *        lx = fma(cos, dx, sin*dy), ly = fma(cos, dy, -(sin*dx)),
 *        |lx| <= ext_x  and  |ly| <= ext_y;
 *      otherwise it is kept with probability rho_out (Alg. 1), drawn from a
 *      counter-based generator so that the draw is a function of the point:
 *      kept iff (splitmix64(seed, i + 1) >> 40) < round(rho_out * 2^24),
 *      i the point's index in the batch;
 *   4. it is quantised (Alg. 1 "Voxelize"): f_d = (p'_d - min_d) / v_d in
 *      fp32 (correctly rounded), kept iff 0 <= f_d < D_d on all three axes,
 *      i_d = trunc(f_d), key = ((b*Dz + iz)*Dy + iy)*Dx + ix;
 *   5. the kept (key, index) pairs are sorted; equal keys form a voxel, which
 *      keeps its max_points lowest point indices;
 *   6. a frame with more than max_voxels voxels keeps the max_voxels voxels
 *      whose lowest point index is smallest, still listed in key order;
 *   7. each voxel's feature c is the mean over its kept points of p'_c
 *      (c < 3) or of the raw column c (c >= 3), summed in double in
 *      ascending point order and rounded once to fp32 (Alg. 1 "VoxelFeature-
 *      Encoder" read as mean pooling);
 *   8. ScatterToBEV (Alg. 1's return value; Sec. IV-F: the features are
 *      written into a zero-initialised bird's-eye-view map by voxel
 *      coordinate, the map having the shape a dense pipeline would produce):
 *      the height axis becomes channels, map[b][c*Dz + iz][iy][ix] = feature
 *      c of voxel (b, iz, iy, ix), 0 where no voxel lies;
 *   9. the voxel-grid connected-component proposer (robot deployment,
 *      Sec. VI: object clusters found on the voxel grid): in each frame a
 *      bird's-eye-view cell (x, y) = (ix >> s, iy >> s) is occupied when a
 *      voxel of a layer iz in [z_min, z_max) lies in it; clusters are the
 *      connected components of the occupied cells (4- or 8-neighbourhood)
 *      with at least min_cells cells, listed per frame by their smallest
 *      cell index y*Wx + x (Wx = ceil(Dx / 2^s)), found here by flood fill
 *      in ascending cell order.
 *
 * Build: plain C, -O2 -ffp-contract=off, no fast-math.
 */
#ifndef MMBEV_ORACLE_H
#define MMBEV_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Oriented BEV box in the current frame: 32 bytes. */
typedef struct {
  float cx, cy;           /* centre [m] */
  float cos_yaw, sin_yaw; /* rounded once from double */
  float ext_x, ext_y;     /* half length + margin, half width + margin [m] */
  float unused0, unused1;
} oracle_roi;

typedef struct {
  float range_min[3];
  float voxel_size[3];
  int32_t dims[3]; /* Dx, Dy, Dz */
  int32_t max_points;
  int32_t max_voxels; /* per frame */
  int32_t num_sweeps;
  int32_t num_frames;
} oracle_grid;

/* ROI record from a descriptor: centre, full length and width, yaw, margin
 * (Eq. 1 buffer r added to each half extent), all rounded once to fp32. */
void oracle_make_roi(double cx, double cy, double length, double width, double yaw, double margin,
                     oracle_roi* out);

/* Step 2 alone: p' for one point under one 3x4 pose. */
void oracle_compensate(const float* pose12, float x, float y, float z, float* out3);

/* Step 3 alone: 1 if (x', y') lies in the ROI. */
int32_t oracle_inside(const oracle_roi* roi, float x, float y);

/* Step 4 alone: 1 and the three indices if p' lies in the grid. */
int32_t oracle_quantize(const oracle_grid* g, const float* p3, int32_t* ijk);

/* SplitMix64: the n-th output (n >= 1) of the generator seeded with seed. */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t n);

/* round(rho * 2^24) clamped to [0, 2^24]: the background keep threshold. */
uint32_t oracle_background_threshold(float rho);

/* 1 if point i is drawn for the background keep (see step 3). */
int32_t oracle_background_keep(uint64_t seed, uint32_t threshold, int64_t i);

/* Steps 1-4 for all points, out-of-ROI keep rate rho_out with seed. */
int64_t oracle_keep_bg(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                       const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                       const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                       const oracle_grid* g, float rho_out, uint64_t seed, uint64_t* keys, int64_t* idx);

/* The whole path with out-of-ROI keep rate rho_out and seed. */
int64_t oracle_roi_voxelize_bg(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                               const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                               const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                               const oracle_grid* g, float rho_out, uint64_t seed, int32_t* out_coords,
                               int32_t* out_counts, float* out_feats, int32_t* out_point_idx,
                               int64_t* out_voxel_offsets);

/* Steps 1-4 for all points: kept (key, index) pairs in index order.
 * Returns K, or -1 on a bad argument. keys/idx must hold N entries. */
int64_t oracle_keep(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                    const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                    const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                    const oracle_grid* g, uint64_t* keys, int64_t* idx);

/* The whole path.  Outputs sized for num_frames * max_voxels rows:
 * coords int32 [.][4] = (b, iz, iy, ix); counts int32 [.]; feats fp32 [.][C];
 * point_idx int32 [.][max_points] padded with -1; voxel_offsets int64 [B+1].
 * Returns the total number of voxels written, or -1 on a bad argument. */
int64_t oracle_roi_voxelize(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                            const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                            const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                            const oracle_grid* g, int32_t* out_coords, int32_t* out_counts,
                            float* out_feats, int32_t* out_point_idx, int64_t* out_voxel_offsets);

/* Step 8: the BEV map [num_frames][C*Dz][Dy][Dx] (fp32, every element
 * written) from voxels as returned by the whole path (frame b's voxels are
 * rows [voxel_offsets[b], voxel_offsets[b+1])).  Returns 0, or -1 on a bad
 * argument (sizes, or a voxel whose coordinates lie outside the grid or
 * name another frame). */
int32_t oracle_scatter_to_bev(const int32_t* coords, const float* feats, const int64_t* voxel_offsets,
                              int32_t num_frames, int32_t num_features, const int32_t* dims, float* map);

/* Step 9 parameters. */
typedef struct {
  int32_t z_min, z_max;  /* voxel layers iz in [z_min, z_max) count */
  int32_t cell_shift;    /* s: a cell is 2^s x 2^s voxel columns, 0..8 */
  int32_t connectivity;  /* 4 or 8 */
  int32_t min_cells;     /* smaller components are not clusters, >= 1 */
  int32_t reserved;
} oracle_cc_params;

/* One cluster: 56 bytes. */
typedef struct {
  int32_t frame;
  int32_t root;                   /* smallest cell index y*Wx + x of the cluster */
  int32_t cells, voxels, points;  /* occupied cells; voxels in the layers; their kept points */
  int32_t x0, y0, x1, y1;         /* bounding box in cells, inclusive */
  int32_t unused;
  int64_t sum_x, sum_y;           /* sums of the cells' x and y */
} oracle_cluster;

/* Step 9 over voxels as returned by the whole path.  out must hold one
 * entry per voxel row, cluster_offsets num_frames + 1, voxel_labels one per
 * row (the cluster's index in out, or -1).  Returns the number of clusters,
 * or -1 on a bad argument. */
int64_t oracle_clusters(const int32_t* coords, const int32_t* counts, const int64_t* voxel_offsets,
                        int32_t num_frames, const int32_t* dims, const oracle_cc_params* p,
                        oracle_cluster* out, int64_t* cluster_offsets, int32_t* voxel_labels);

#ifdef __cplusplus
}
#endif
#endif
