/*
 * mmbev -- ROI-aware multi-sweep LiDAR voxelisation on AMD Instinct MI355X
 * (gfx950).  C ABI of libmmbev.so.
 *
 * The library implements the LiDAR half of the paper's sparse ROI-aware
 * feature extraction (Sec. IV-F, Alg. 1 "ROIAwareVoxelization", invoked as
 * "ROIVoxelize(ROI_L, n sweeps)" in the coordination loop of Alg. 2): every
 * point of a multi-sweep cloud is moved into the current frame by its sweep's
 * ego pose (Sec. IV-D, Eq. 6/7), kept only if it lies inside one of the
 * frame's temporal ROIs (Sec. IV-C, Eq. 1, read as oriented bird's-eye-view
 * boxes) whose sweep budget admits its sweep (Sec. IV-G budget management,
 * read per ROI), quantised to a voxel grid, grouped by voxel, capped at
 * max_points points per voxel and max_voxels voxels per frame ("hard
 * voxelisation", Sec. IV-F), and mean-pooled into a sparse voxel tensor
 * (the Voxel Feature Encoder of Alg. 1, read as mean pooling).  Points
 * outside every ROI are dropped (Alg. 1's out-of-ROI keep rate set to zero),
 * or, through mmbev_roi_voxelize_ex, kept with a given probability.
 *
 * Exact semantics (every decision is taken in fp32 in this operation order;
 * the library is bit-exact against this definition):
 *   frame b of the batch holds points [points.frame_offsets[b],
 *   points.frame_offsets[b+1]) and ROIs [rois.frame_offsets[b],
 *   rois.frame_offsets[b+1]).  For point i of frame b with sweep s =
 *   sweep_ids[i]:
 *   1. s >= grid.num_sweeps: dropped.
 *   2. P = sweep_poses + (b*num_sweeps + s)*12 (row-major [R | T]);
 *        x' = fma(P0, x, fma(P1, y, fma(P2,  z, P3)))
 *        y' = fma(P4, x, fma(P5, y, fma(P6,  z, P7)))
 *        z' = fma(P8, x, fma(P9, y, fma(P10, z, P11)))
 *   3. kept iff for some ROI j of frame b: s < roi_sweep_budget[j] and
 *        dx = x' - cx; dy = y' - cy;
 *        lx = fma(cos_yaw, dx, sin_yaw*dy); ly = fma(cos_yaw, dy, -(sin_yaw*dx));
 *        |lx| <= ext_x and |ly| <= ext_y            (products rounded to fp32)
 *      or, with an out-of-ROI keep rate rho (mmbev_options_t), iff
 *        (splitmix64(seed, i + 1) >> 40) < round(rho * 2^24), clamped to
 *        [0, 2^24] (NaN: 0), where splitmix64(seed, n) is the n-th output of
 *        the SplitMix64 generator whose 64-bit state starts at seed
 *        (state += 0x9E3779B97F4A7C15, then the state mixed: z ^= z >> 30,
 *        z *= 0xBF58476D1CE4E5B9, z ^= z >> 27, z *= 0x94D049BB133111EB,
 *        z ^= z >> 31) and i the point's index in the batch;
 *   4. f_d = (p'_d - range_min[d]) / voxel_size[d]  (IEEE fp32, correctly rounded);
 *      kept iff 0 <= f_d < dims[d] for d = x, y, z (NaN fails); i_d = trunc(f_d).
 *      Voxel key = (b, iz, iy, ix) in lexicographic order.
 *   5. Voxels are the distinct keys of frame b.  A voxel keeps its max_points
 *      lowest point indices.  A frame with more than max_voxels voxels keeps
 *      the max_voxels voxels whose lowest point index is smallest.
 *   6. Output, per frame in ascending key order: coords (b, iz, iy, ix), the
 *      kept count, the kept point indices ascending (padded with -1), and the
 *      mean of each feature over the kept points -- x', y', z' for features
 *      0..2, the raw column for features 3.. -- summed in double in ascending
 *      point order and rounded once to fp32.
 */
#ifndef MMBEV_H
#define MMBEV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MMBEV_ABI_VERSION 7

/* ------------------------------------------------------------- status */
typedef int32_t mmbev_status_t;
#define MMBEV_OK 0
#define MMBEV_ERR_INVALID_ARG (-1) /* null pointer, bad size or range */
#define MMBEV_ERR_WORKSPACE (-2)   /* workspace missing, too small or misaligned */
#define MMBEV_ERR_UNSUPPORTED (-3) /* sizes beyond the documented limits */
#define MMBEV_ERR_HIP (-4)         /* a HIP call failed; no partial results */

/* Device-side data faults.  The kernels never read or write out of bounds,
 * whatever the data; when the content of a device array breaks the contract
 * they OR one of these bits into the int32 at byte 0 of the workspace and the
 * output is unspecified.  Read it after the stream has completed. */
#define MMBEV_FAULT_POINT_OFFSETS 1 /* point frame offsets not 0 .. num_points, non-decreasing
                                       (the call then keeps no point: no voxel is written) */
#define MMBEV_FAULT_ROI_OFFSETS 2   /* ROI frame offsets not 0 .. num_rois, non-decreasing,
                                       or a frame with more than max_rois_per_frame ROIs */
#define MMBEV_FAULT_INTERNAL 4      /* an internal consistency check failed (never with valid inputs) */
#define MMBEV_FAULT_VOXELS 8        /* mmbev_scatter_to_bev, mmbev_voxel_clusters: voxel rows break
                                       the contract (offsets, coordinates outside the grid or of
                                       another frame; for the scatter also keys not strictly
                                       ascending inside a frame) */

/* ------------------------------------------------------------- inputs */

/* Points, structure of arrays in device memory: feature c of point i is
 * feat[c*stride + i].  Features 0..2 are x, y, z in the frame of the point's
 * sweep [m]; features 3.. (e.g. intensity, sweep time offset) are passed
 * through to the mean.  Frames are contiguous point ranges. */
typedef struct {
  const float* feat;            /* device, [num_features][stride] */
  int64_t stride;               /* >= num_points */
  int32_t num_features;         /* C, 3..8 */
  int32_t reserved;             /* 0 */
  int64_t num_points;           /* N, 0 .. 2^30-1 over all frames */
  const int64_t* frame_offsets; /* device, [num_frames+1], 0 = off[0] <= ... <= off[B] = N */
} mmbev_points_t;

/* One temporal ROI (Eq. 1 footprint buffered by the margin r): an oriented
 * bird's-eye-view box in the current frame, 32 bytes.  Build with
 * mmbev_make_rois; the kernels never recompute cos/sin. */
typedef struct {
  float cx, cy;           /* centre [m] */
  float cos_yaw, sin_yaw; /* box x axis = (cos_yaw, sin_yaw) */
  float ext_x, ext_y;     /* half length + margin, half width + margin [m] */
  float reserved[2];
} mmbev_roi_t;

/* ROIs of all frames, grouped by frame.  The order inside a frame (e.g. a
 * criticality ranking) does not change the result. */
typedef struct {
  const mmbev_roi_t* boxes;     /* device, [num_rois] */
  const int32_t* frame_offsets; /* device, [num_frames+1] */
  int32_t num_rois;             /* >= 0 */
  int32_t max_rois_per_frame;   /* upper bound on any frame's count, 0..1024 */
} mmbev_rois_t;

typedef struct {
  float range_min[3];  /* grid origin x, y, z [m] */
  float voxel_size[3]; /* > 0 [m] */
  int32_t dims[3];     /* Dx, Dy, Dz >= 1, Dx*Dy*Dz <= 2^32 */
  int32_t max_points;  /* M, 1..64 points kept per voxel */
  int32_t max_voxels;  /* voxels kept per frame, >= 1 */
  int32_t num_sweeps;  /* S, 1..255 */
  int32_t num_frames;  /* B, 1..65535 */
} mmbev_grid_t;

/* Options of mmbev_roi_voxelize_ex (Alg. 1 keep loop). */
typedef struct {
  float out_of_roi_keep_rate; /* rho in [0, 1]: probability that a point in no ROI is kept; 0 keeps none */
  uint32_t reserved;          /* 0 */
  uint64_t seed;              /* seed of the per-point draw (a function of seed and point index only) */
} mmbev_options_t;

/* ------------------------------------------------------------ queries */
int32_t mmbev_abi_version(void);
const char* mmbev_status_string(mmbev_status_t status);

/* Workspace bytes mmbev_roi_voxelize needs for these sizes (0 if they are
 * invalid).  The workspace depends only on the grid, num_points,
 * num_features (C, 3..8) and max_rois_per_frame. */
size_t mmbev_roi_voxelize_workspace_bytes(const mmbev_grid_t* grid, int64_t num_points, int32_t num_features,
                                          int32_t max_rois_per_frame);

/* Zero-fill a workspace on `stream` (a hipStream_t; NULL = default stream).
 * A workspace must be initialised once before its first use; after that it
 * is reused across calls as is. */
mmbev_status_t mmbev_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------ helpers */

/* Host helper: ROI records from descriptor rows of 6 doubles (cx, cy,
 * length, width, yaw, margin).  cos/sin are taken in double and rounded once;
 * ext = size/2 + margin rounded once.  desc and out are host memory. */
mmbev_status_t mmbev_make_rois(const double* desc, int64_t count, mmbev_roi_t* out);

/* ------------------------------------------------------------ the path */

/*
 * Voxelise a batch of frames (semantics at the top of this file).
 *
 * All array arguments are device pointers; the structs themselves are host
 * memory read during the call.  Outputs have room for
 * num_frames * max_voxels rows:
 *   out_coords        int32 [rows][4]   (b, iz, iy, ix)
 *   out_counts        int32 [rows]      kept points per voxel, 1..max_points
 *   out_feats         fp32  [rows][num_features]
 *   out_point_idx     int32 [rows][max_points], -1 padded
 *   out_voxel_offsets int64 [num_frames+1]; frame b's voxels are rows
 *                     [off[b], off[b+1]) in ascending key order
 * Rows past off[num_frames] are left untouched.
 *
 * sweep_ids          uint8 [num_points], 0 = the current (newest) sweep
 * sweep_poses        fp32  [num_frames][num_sweeps][12], row-major [R | T]
 *                    taking sweep-s coordinates into the current frame
 * roi_sweep_budget   uint8 [num_rois]: ROI j admits sweeps s < budget[j]
 *                    (0 disables the ROI)
 *
 * Ownership: the caller owns every buffer; the library allocates nothing and
 * keeps no state between calls.  Work is enqueued on `stream` (a
 * hipStream_t; NULL = default stream) and the call returns without waiting;
 * results are valid once the stream has reached this point.  The workspace
 * (size from mmbev_roi_voxelize_workspace_bytes, 256-byte aligned,
 * initialised once by mmbev_workspace_init) must not be used by two calls
 * that can run at the same time.
 *
 * Errors: argument errors are detected on the host before anything is
 * enqueued and returned as MMBEV_ERR_*; a failed launch returns
 * MMBEV_ERR_HIP.  Problems in the content of device arrays are reported
 * through the fault word (MMBEV_FAULT_*).
 */
mmbev_status_t mmbev_roi_voxelize(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                  const float* sweep_poses, const mmbev_rois_t* rois,
                                  const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid_params,
                                  int32_t* out_coords, int32_t* out_counts, float* out_feats,
                                  int32_t* out_point_idx, int64_t* out_voxel_offsets, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * Same call as mmbev_roi_voxelize, for measurement: before each of its
 * launch groups, and once after the last, it records the next of the
 * caller's events (hipEvent_t, created with timing enabled) on `stream`, as
 * long as events remain.  The groups, in order: ROI staging, point filter,
 * chunk layout (segments), compaction and records, then one radix pass per
 * key digit of at most 9 bits (count and scatter launches), voxel heads,
 * finalisation with the per-frame voxel cap, mean pooling.  Returns the number of events recorded through *events_recorded
 * (host int32, may be NULL).  Elapsed time between events k and k+1 is the
 * duration of group k.
 */
mmbev_status_t mmbev_roi_voxelize_profiled(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                           const float* sweep_poses, const mmbev_rois_t* rois,
                                           const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid_params,
                                           int32_t* out_coords, int32_t* out_counts, float* out_feats,
                                           int32_t* out_point_idx, int64_t* out_voxel_offsets, void* workspace,
                                           size_t workspace_bytes, void* stream, void* const* events,
                                           int32_t num_events, int32_t* events_recorded);

/*
 * The same call with options (NULL: the defaults, out-of-ROI keep rate 0)
 * and, like mmbev_roi_voxelize_profiled, optional events (events may be NULL
 * and num_events 0).  Alg. 1 keeps points outside every ROI with probability
 * rho_out; here the draw of point i is the counter-based function of
 * (seed, i) given at the top of this file, so a result is reproducible and
 * independent of the launch layout.  Errors: MMBEV_ERR_INVALID_ARG also for
 * a nonzero reserved field.
 */
mmbev_status_t mmbev_roi_voxelize_ex(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                     const float* sweep_poses, const mmbev_rois_t* rois,
                                     const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid_params,
                                     const mmbev_options_t* options, int32_t* out_coords, int32_t* out_counts,
                                     float* out_feats, int32_t* out_point_idx, int64_t* out_voxel_offsets,
                                     void* workspace, size_t workspace_bytes, void* stream, void* const* events,
                                     int32_t num_events, int32_t* events_recorded);

/* ---------------------------------------- callers that cannot allocate */

/* Bytes of the library's own device scratch (64 MiB): the largest workspace
 * mmbev_roi_voxelize_noalloc can use -- enough for about a million points of
 * five features with up to 32 ROIs per frame (mmbev_roi_voxelize_workspace_bytes
 * gives the exact need of given sizes). */
#define MMBEV_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * mmbev_roi_voxelize without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same semantics, arguments, outputs,
 * ownership and errors as mmbev_roi_voxelize; the workspace is instead an
 * array of MMBEV_NOALLOC_SCRATCH_BYTES bytes of device memory inside the
 * library, one per device, which every GPU the library runs on holds until
 * the process ends.  The call allocates nothing.
 *
 * The first call on a device (the current device; `stream` must belong to
 * it) looks up that device's array and clears its header on `stream`.  All
 * calls on one device share its array, which keeps the last call's
 * contents: calls that can overlap on one GPU (on different streams, or from
 * host threads without ordering between them) race and leave unspecified
 * results; order them on one stream.
 *
 * out_fault  device int32, may be NULL: receives the call's fault word
 *            (MMBEV_FAULT_*, 0 for none) when the stream reaches the end of
 *            the call (the array's own fault word is not reachable otherwise).
 * Errors: as mmbev_roi_voxelize; MMBEV_ERR_UNSUPPORTED also when the sizes
 * need a workspace larger than MMBEV_NOALLOC_SCRATCH_BYTES; MMBEV_ERR_HIP
 * when the device's array cannot be looked up.
 */
mmbev_status_t mmbev_roi_voxelize_noalloc(const mmbev_points_t* points, const uint8_t* sweep_ids,
                                          const float* sweep_poses, const mmbev_rois_t* rois,
                                          const uint8_t* roi_sweep_budget, const mmbev_grid_t* grid_params,
                                          int32_t* out_coords, int32_t* out_counts, float* out_feats,
                                          int32_t* out_point_idx, int64_t* out_voxel_offsets, int32_t* out_fault,
                                          void* stream);

/* ------------------------------ temporal ROIs and criticality (host) */

/* Object classes of the criticality thresholds (Sec. IV-C). */
#define MMBEV_CLASS_VRU 0       /* pedestrians, cyclists: TTC threshold tau_vru */
#define MMBEV_CLASS_MOTORIZED 1 /* vehicles: tau_motorized */
#define MMBEV_CLASS_STATIC 2    /* barriers, cones: geometry-critical only */

/* A detection of frame t-1 (an entry of the detection cache B^{t-1}), in the
 * ego frame of t-1: x forward, y left [m], yaw [rad] about z; velocity is the
 * object's own (ground) velocity expressed in those axes [m/s].  64 bytes. */
typedef struct {
  double x, y, yaw;
  double length, width;
  double vx, vy;
  int32_t cls;      /* MMBEV_CLASS_* */
  int32_t reserved; /* 0 */
} mmbev_detection_t;

/* Ego state of frame t: speed [m/s] along +x, and the rigid motion from the
 * ego frame of t-1 to that of t (a point p of frame t-1 is
 * R(dyaw) p + (dx, dy) in frame t). */
typedef struct {
  double speed;
  double dx, dy, dyaw;
} mmbev_ego_t;

/* Selector and coordinator parameters (Sec. IV-C, IV-G). */
typedef struct {
  double dt;                          /* Delta t between frames [s] */
  double margin;                      /* r of Eq. 1 [m] */
  double a_brake, d_min;              /* Eq. 4 [m/s^2], [m] */
  double theta_max_deg, theta_min_deg; /* cone half-angle at and below speed_wide / at and above speed_narrow */
  double speed_wide, speed_narrow;    /* [m/s]; theta is linear in speed between them */
  double tau_vru, tau_motorized;      /* Eq. 5 thresholds [s] */
  double r_coll;                      /* Eq. 8 collision radius [m] */
  double slow_speed;                  /* ego slower than this: the reduced sweep count */
  int32_t dense_count;                /* this many detections or more: the reduced sweep count */
  int32_t n_full, n_reduced;          /* sweep counts (1..255): mandatory ROIs always get n_full */
  int32_t max_optional;               /* optional detections kept per frame (by rank); the rest dropped */
  int32_t reserved;                   /* 0 */
  double fallback_length, fallback_width; /* empty cache: one ego-centred box of this size, n_full sweeps (0: none) */
} mmbev_policy_t;

/* Per-detection outcome.  Flags: */
#define MMBEV_CRIT_GEOM 1      /* Eq. 3: inside the forward braking cone */
#define MMBEV_CRIT_SAFETY 2    /* Eq. 5: TTC at or below the class threshold */
#define MMBEV_CRIT_MANDATORY 4 /* GEOM or SAFETY */
#define MMBEV_CRIT_DROPPED 8   /* optional and ranked past max_optional: its ROIs get budget 0 */
typedef struct {
  double ttc;    /* Eq. 8 [s]; +infinity when there is no approach within r_coll */
  int32_t flags; /* MMBEV_CRIT_* */
  int32_t rank;  /* position of the detection in its frame's ranking, 0 = most critical */
} mmbev_criticality_t;

/*
 * The Criticality-Ranked Temporal-ROI Selector and the sweep-count knob of
 * the coordinator (Sec. IV-C, IV-G; Alg. 2 TemporalROI, ComputeTTC,
 * ScaleCompute), producing the rois and roi_sweep_budget arguments of
 * mmbev_roi_voxelize.  Host code; every array is host memory.  Per frame b,
 * for each detection i (all arithmetic in double, in this order):
 *   1. footprints: the box at t-1 and the box moved by (vx, vy)*dt (Eq. 1),
 *      both taken into frame t by the ego motion (centre rotated by dyaw and
 *      shifted by (dx, dy); yaw + dyaw);
 *   2. criticality from the moved box in frame t: p = its centre, the
 *      relative velocity w = R(dyaw)(vx, vy) - (speed, 0);
 *      d_max = max(d_min, speed^2 / (2 a_brake))                     (Eq. 4)
 *      theta = theta_max at speed <= speed_wide, theta_min at speed >=
 *        speed_narrow, linear in between (degrees, then radians)
 *      GEOM iff p.x >= 0 and |p| <= d_max and atan2(|p.y|, p.x) <= theta (Eq. 3)
 *      t* = -(p . w) / |w|^2; TTC = t* iff |w| > 0, t* > 0 and
 *        |p + t* w| <= r_coll, else +inf                             (Eq. 8)
 *      SAFETY iff the class is not STATIC and TTC <= tau_class        (Eq. 5)
 *      MANDATORY iff GEOM or SAFETY;
 *   3. ranking: mandatory before optional, then ascending TTC, then
 *      ascending |p|, then input order; optional detections ranked past
 *      max_optional among the optional ones are DROPPED;
 *   4. sweep count n = n_reduced if speed < slow_speed or the frame has at
 *      least dense_count detections, else n_full (written to out_sweeps);
 *   5. ROI records, in rank order, two per detection (its footprint at t-1,
 *      then the moved one), built like mmbev_make_rois from (cx, cy, length,
 *      width, yaw, margin); budget n_full if mandatory, 0 if dropped, else n.
 *      A frame without detections gets the fallback box (centre 0, yaw 0, no
 *      margin) with budget n_full, unless its size is 0.
 *
 * dets [det_offsets[B]], det_offsets [B+1] (non-decreasing, from 0); ego [B].
 * Outputs: out_rois and out_budgets hold 2 * det_offsets[B] + B entries,
 * out_roi_offsets B+1 (frame b's records are [off[b], off[b+1])),
 * out_crit det_offsets[B] (in input order), out_sweeps B.
 * Errors: MMBEV_ERR_INVALID_ARG for a null pointer, bad offsets, a
 * non-finite or out-of-range parameter (dt, r_coll, a_brake > 0; margin,
 * d_min >= 0; 0 <= theta_min <= theta_max <= 90; speed_wide <= speed_narrow;
 * 1 <= n_reduced <= n_full <= 255; max_optional >= 0), an unknown class or a
 * nonzero reserved field; nothing is written then.
 */
mmbev_status_t mmbev_build_rois(const mmbev_detection_t* dets, const int32_t* det_offsets, int32_t num_frames,
                                const mmbev_ego_t* ego, const mmbev_policy_t* policy, mmbev_roi_t* out_rois,
                                uint8_t* out_budgets, int32_t* out_roi_offsets, mmbev_criticality_t* out_crit,
                                int32_t* out_sweeps);

/* ------------------------------------------------ ScatterToBEV (Alg. 1) */

/*
 * Write voxel features into a dense bird's-eye-view map (Alg. 1's return
 * value, "ScatterToBEV"; Sec. IV-F: features go into a zero-initialised BEV
 * map by voxel coordinate, the map having the shape a dense pipeline would
 * produce).  The height axis is folded into channels:
 *   bev_map[b][c*Dz + iz][iy][ix] = feats[v][c]   for every voxel v of frame b
 *                                                 with coords[v] = (b, iz, iy, ix),
 *   0.0f everywhere else                          (Dz = 1: the pillar map [B][C][Dy][Dx]).
 *
 * coords         int32 [rows][4], device, 16-byte aligned
 * feats          fp32  [rows][num_features], device
 * voxel_offsets  int64 [num_frames+1], device: frame b's voxels are rows
 *                [off[b], off[b+1]); rows = num_frames * max_voxels
 *                These are exactly the outputs of mmbev_roi_voxelize: inside
 *                a frame the keys (iz*Dy + iy)*Dx + ix are strictly ascending.
 * num_features   C, 1..64
 * grid           dims, max_voxels and num_frames are read (host struct)
 * bev_map        fp32 [num_frames][C*Dz][Dy][Dx], device; every element is
 *                written (no clearing needed beforehand)
 * fault          device int32, may be NULL.  If given, the rows are checked
 *                and MMBEV_FAULT_VOXELS is ORed into it when they break the
 *                contract above (the caller clears it); the map is then
 *                unspecified.  Whatever the rows hold, no access leaves the
 *                buffers described here.
 *
 * Ownership and errors as for mmbev_roi_voxelize: caller-owned buffers, no
 * allocation, work enqueued on `stream` (NULL = default stream) without
 * waiting; argument errors return MMBEV_ERR_INVALID_ARG or
 * MMBEV_ERR_UNSUPPORTED before anything is enqueued.
 */
mmbev_status_t mmbev_scatter_to_bev(const int32_t* coords, const float* feats, const int64_t* voxel_offsets,
                                    int32_t num_features, const mmbev_grid_t* grid, float* bev_map,
                                    int32_t* fault, void* stream);

/* ----------------------------- voxel-grid connected-component proposer */

/* Parameters of mmbev_voxel_clusters. */
typedef struct {
  int32_t z_min, z_max;  /* voxel layers iz in [z_min, z_max) count (e.g. above the ground) */
  int32_t cell_shift;    /* s, 0..8: a cell is 2^s x 2^s voxel columns */
  int32_t connectivity;  /* 4 or 8 (edge or edge-and-corner neighbours) */
  int32_t min_cells;     /* components with fewer cells are not clusters, >= 1 */
  int32_t reserved;      /* 0 */
} mmbev_cluster_params_t;

/* One cluster, 56 bytes.  Cell coordinates are x = ix >> s, y = iy >> s;
 * cell index y*Wx + x with Wx = ceil(Dx / 2^s), Wy = ceil(Dy / 2^s). */
typedef struct {
  int32_t frame;
  int32_t root;          /* smallest cell index of the cluster (its identity inside the frame) */
  int32_t cells;         /* occupied cells */
  int32_t voxels;        /* voxels in the layer band */
  int32_t points;        /* kept points of those voxels (sum of their counts) */
  int32_t x0, y0, x1, y1; /* bounding box in cells, inclusive */
  int32_t reserved;
  int64_t sum_x, sum_y;  /* sums of the cells' x and y (the centroid is sum / cells) */
} mmbev_cluster_t;

/* Workspace bytes of mmbev_voxel_clusters (0 if the sizes are invalid or
 * unsupported: num_frames * Wx * Wy must stay below 2^29 cells). */
size_t mmbev_voxel_clusters_workspace_bytes(const mmbev_grid_t* grid, const mmbev_cluster_params_t* params);

/*
 * Object clusters on the voxel grid: the lightweight connected-component
 * proposer of the paper's robot deployment (Sec. VI), whose cluster set
 * feeds the adaptive keyframe scheduler's cluster-shift trigger.  Reading:
 * in each frame a bird's-eye-view cell (ix >> s, iy >> s) is occupied when a
 * voxel of a layer in [z_min, z_max) lies in it; clusters are the connected
 * components of the occupied cells (4- or 8-neighbourhood) with at least
 * min_cells cells, listed per frame in ascending order of their smallest
 * cell index.  Every field is an integer, so the result is unique.
 *
 * coords, counts, voxel_offsets: device arrays as written by
 *   mmbev_roi_voxelize (rows = num_frames * max_voxels; frame b's voxels are
 *   rows [off[b], off[b+1]); the order inside a frame does not matter)
 * out_clusters         device, [rows]; clusters [0, off'[B]) are written
 * out_cluster_offsets  device, int64 [num_frames+1]: frame b's clusters are
 *                      [off'[b], off'[b+1])
 * out_voxel_labels     device, int32 [rows]: for rows [0, off[B]) the index of
 *                      the voxel's cluster, or -1 (outside the layer band or in
 *                      a component below min_cells); other rows untouched
 * workspace            device, 256-byte aligned, size from
 *                      mmbev_voxel_clusters_workspace_bytes; needs no
 *                      initialisation; its int32 at byte 0 receives
 *                      MMBEV_FAULT_VOXELS when rows break the contract (such
 *                      rows are skipped; every access stays inside the buffers)
 *
 * Ownership, streams and errors as for mmbev_roi_voxelize.
 */
mmbev_status_t mmbev_voxel_clusters(const int32_t* coords, const int32_t* counts, const int64_t* voxel_offsets,
                                    const mmbev_grid_t* grid, const mmbev_cluster_params_t* params,
                                    mmbev_cluster_t* out_clusters, int64_t* out_cluster_offsets,
                                    int32_t* out_voxel_labels, void* workspace, size_t workspace_bytes,
                                    void* stream);

#ifdef __cplusplus
}
#endif
#endif /* MMBEV_H */
