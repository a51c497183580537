/* Seeded synthetic LiDAR scenes: inputs for the voxeliser and its oracle. */
#ifndef SYNTH_GEN_H
#define SYNTH_GEN_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t beams;        /* rows of the organised scan */
  int32_t azimuths;     /* columns per revolution */
  double elev_lo_deg;   /* lowest beam elevation */
  double elev_hi_deg;   /* highest beam elevation */
  double sensor_h;      /* sensor height above ground [m] */
  double range_sigma;   /* range noise std-dev [m] */
  double r_max;         /* no-return range [m] */
  int32_t num_sweeps;   /* sweeps per frame */
  int32_t num_features; /* 3..8: x, y, z, intensity, dt, zeros */
  double sweep_dt;      /* seconds between sweeps */
  double speed_lo, speed_hi;     /* ego speed range [m/s] */
  double yawrate_lo, yawrate_hi; /* ego yaw-rate range [rad/s] */
  int32_t num_obstacles;         /* <= 64 */
  int32_t axis_aligned;          /* 1: obstacle yaw 0 */
  double obs_len, obs_wid, obs_hgt; /* nominal obstacle size [m] */
  double obs_jitter;                /* relative size jitter (0.1 = +-10%) */
  double obs_r_lo, obs_r_hi;        /* annulus of obstacle centres [m] */
} synth_scene_t;

typedef struct {
  int32_t num_on_obstacles; /* ROIs on the footprints of the first obstacles */
  int32_t num_extrapolated; /* shifted copies of the first obstacles */
  int32_t num_random;       /* free-standing ROIs */
  int32_t num_overlapping;  /* how many of the random ones sit on an earlier ROI */
  double extrap_speed, extrap_dt; /* shift = speed * dt along the obstacle heading */
  double rand_extent;             /* random centres uniform in +-extent [m] */
  double rand_len, rand_wid;      /* nominal random ROI size (+-10%) [m] */
  double margin;                  /* margin recorded in every descriptor [m] */
  int32_t budget_lo, budget_hi;   /* sweep budgets uniform in [lo, hi] */
} synth_roi_recipe_t;

/* Obstacles as rows of 7 doubles (cx, cy, cz, length, width, height, yaw) in
 * the current frame.  Returns the number placed (<= num_obstacles). */
int64_t synth_obstacles(const synth_scene_t* sc, uint64_t seed, double* obs);

/* One frame of num_sweeps sweeps written at points [offset, offset + S*beams*azimuths)
 * of the SoA array feat[c*stride + i]; sweep ids alongside; poses [S][12]
 * row-major [R | T] mapping sweep-s coordinates into the current frame.
 * Returns the number of points written, or -1 if num_obs > 64. */
int64_t synth_frame(const synth_scene_t* sc, uint64_t seed, const double* obs, int64_t num_obs,
                    float* feat, int64_t stride, int64_t offset, uint8_t* sweep_ids, float* poses);

/* ROI descriptors as rows of 6 doubles (cx, cy, length, width, yaw, margin)
 * plus one sweep budget per ROI.  Returns the number of ROIs written. */
int64_t synth_rois(const synth_roi_recipe_t* rc, uint64_t seed, const double* obs, int64_t num_obs,
                   double* desc, uint8_t* budgets);

#ifdef __cplusplus
}
#endif
#endif
