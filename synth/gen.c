/*
 * Seeded synthetic multi-sweep LiDAR scenes.
 *
 * This module produces INPUTS only: organised spinning-LiDAR scans cast
 * against a ground plane and static boxes, per-sweep ego poses, and ROI
 * descriptors (centre, size, yaw, margin) with per-ROI sweep budgets.  It
 * holds none of the voxelisation arithmetic: no compensation of points into
 * the current frame, no ROI membership test, no quantisation.  Both the GPU
 * path and the CPU oracle consume what it writes.
 *
 * Everything is deterministic for a given seed on any IEEE-754 host:
 *   - RNG: xoshiro256** seeded through SplitMix64 (published generators of
 *     Blackman & Vigna), uniforms from the top 53 bits, normals by
 *     Box-Muller in double;
 *   - geometry in double, rounded once to fp32 on store.
 *
 * Scene model (stands in for the paper's nuScenes 32-beam sweeps and the
 * robot's Ouster OS1-128 frames, neither of which is available here):
 *   - the ego frame of every sweep has the ground at z = 0 and the sensor at
 *     z = sensor_h; rays of beam k (elevations linspace over [lo, hi]) and
 *     azimuth column a (uniform steps plus a per-sweep phase) hit the nearest
 *     of the ground plane and the obstacle boxes; range noise N(0, sigma)
 *     along the ray; rays with no hit within r_max return a point at r_max;
 *   - the ego follows a constant-turn-rate-and-velocity path; sweep s was
 *     taken tau = -s * sweep_dt seconds before the current sweep, so its pose
 *     maps sweep-s coordinates into the current frame;
 *   - obstacles are static in the current frame and are seen by each sweep
 *     from that sweep's own pose;
 *   - points are stored sweep-major (s = 0, the newest, first), and inside a
 *     sweep beam-major (organised rows), column index fastest.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "gen.h"

static const double kPi = 3.14159265358979323846;

/* ---------------------------------------------------------------- RNG */
typedef struct {
  uint64_t s[4];
} rng_t;

static uint64_t splitmix64(uint64_t* x) {
  uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static void rng_seed(rng_t* r, uint64_t seed) {
  uint64_t x = seed;
  for (int k = 0; k < 4; ++k) r->s[k] = splitmix64(&x);
}

static uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static uint64_t rng_next(rng_t* r) {
  uint64_t* s = r->s;
  uint64_t result = rotl(s[1] * 5, 7) * 9;
  uint64_t t = s[1] << 17;
  s[2] ^= s[0];
  s[3] ^= s[1];
  s[1] ^= s[2];
  s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return result;
}

/* uniform in [0, 1) from the top 53 bits */
static double rng_u01(rng_t* r) { return (double)(rng_next(r) >> 11) * 0x1.0p-53; }

static double rng_uniform(rng_t* r, double lo, double hi) { return lo + (hi - lo) * rng_u01(r); }

/* integer uniform in [lo, hi] */
static int rng_int(rng_t* r, int lo, int hi) {
  uint64_t span = (uint64_t)(hi - lo + 1);
  return lo + (int)((rng_next(r) >> 11) % span);
}

static double rng_normal(rng_t* r) {
  double u1 = 1.0 - rng_u01(r); /* (0, 1] */
  double u2 = rng_u01(r);
  return sqrt(-2.0 * log(u1)) * cos(2.0 * kPi * u2);
}

/* ------------------------------------------------------------ helpers */
static const double kDeg = kPi / 180.0;

/* Ego pose of the sweep taken tau seconds before now (tau <= 0 passed as
 * its value), constant speed v and yaw rate w: heading psi and planar
 * position (px, py) expressed in the current frame. */
static void ctrv_pose(double v, double w, double tau, double* psi, double* px, double* py) {
  *psi = w * tau;
  if (fabs(w) < 1e-9) {
    *px = v * tau;
    *py = 0.0;
  } else {
    *px = (v / w) * sin(w * tau);
    *py = (v / w) * (1.0 - cos(w * tau));
  }
}

/* Slab test of the ray o + t d against an axis-aligned box centred at the
 * origin with half sizes h[3].  Returns the entry distance, or INFINITY. */
static double ray_box(const double o[3], const double d[3], const double h[3]) {
  double t0 = -INFINITY, t1 = INFINITY;
  for (int k = 0; k < 3; ++k) {
    if (fabs(d[k]) < 1e-15) {
      if (o[k] < -h[k] || o[k] > h[k]) return INFINITY;
      continue;
    }
    double a = (-h[k] - o[k]) / d[k];
    double b = (h[k] - o[k]) / d[k];
    if (a > b) {
      double t = a;
      a = b;
      b = t;
    }
    if (a > t0) t0 = a;
    if (b < t1) t1 = b;
    if (t0 > t1) return INFINITY;
  }
  if (t1 <= 0.0) return INFINITY;
  if (t0 <= 0.0) return INFINITY; /* sensor inside the box: ignore */
  return t0;
}

/* --------------------------------------------------------- obstacles */
int64_t synth_obstacles(const synth_scene_t* sc, uint64_t seed, double* obs) {
  rng_t r;
  rng_seed(&r, seed ^ 0x0B57AC1E5EEDull);
  int n = 0;
  int attempts = 0;
  while (n < sc->num_obstacles && attempts < 100000) {
    ++attempts;
    double jit = sc->obs_jitter;
    double len = sc->obs_len * rng_uniform(&r, 1.0 - jit, 1.0 + jit);
    double wid = sc->obs_wid * rng_uniform(&r, 1.0 - jit, 1.0 + jit);
    double hgt = sc->obs_hgt * rng_uniform(&r, 1.0 - jit, 1.0 + jit);
    double rad = sqrt(rng_uniform(&r, sc->obs_r_lo * sc->obs_r_lo, sc->obs_r_hi * sc->obs_r_hi));
    double az = rng_uniform(&r, 0.0, 2.0 * kPi);
    double yaw = sc->axis_aligned ? 0.0 : rng_uniform(&r, 0.0, 2.0 * kPi);
    double cx = rad * cos(az), cy = rad * sin(az);
    double br = 0.5 * sqrt(len * len + wid * wid);
    int clash = 0;
    for (int k = 0; k < n && !clash; ++k) {
      const double* o = obs + 7 * k;
      double ok = 0.5 * sqrt(o[3] * o[3] + o[4] * o[4]);
      double dx = cx - o[0], dy = cy - o[1];
      if (sqrt(dx * dx + dy * dy) < br + ok + 0.5) clash = 1;
    }
    /* keep the sensor column clear */
    if (rad < br + 1.0) clash = 1;
    if (clash) continue;
    double* o = obs + 7 * n;
    o[0] = cx;
    o[1] = cy;
    o[2] = 0.5 * hgt;
    o[3] = len;
    o[4] = wid;
    o[5] = hgt;
    o[6] = yaw;
    ++n;
  }
  return n;
}

/* ------------------------------------------------------------- sweeps */
int64_t synth_frame(const synth_scene_t* sc, uint64_t seed, const double* obs, int64_t num_obs,
                    float* feat, int64_t stride, int64_t offset, uint8_t* sweep_ids, float* poses) {
  if (num_obs > 64) return -1;
  rng_t r;
  rng_seed(&r, seed);
  const int S = sc->num_sweeps;
  const int nb = sc->beams, na = sc->azimuths;
  const int64_t per_sweep = (int64_t)nb * na;

  double v = rng_uniform(&r, sc->speed_lo, sc->speed_hi);
  double w = rng_uniform(&r, sc->yawrate_lo, sc->yawrate_hi);

  for (int s = 0; s < S; ++s) {
    double tau = -(double)s * sc->sweep_dt;
    double psi, px, py;
    ctrv_pose(v, w, tau, &psi, &px, &py);
    double c = cos(psi), sn = sin(psi);
    /* [R | T], row-major 3x4: sweep-s coordinates -> current frame */
    float* P = poses + 12 * s;
    P[0] = (float)c;
    P[1] = (float)(-sn);
    P[2] = 0.0f;
    P[3] = (float)px;
    P[4] = (float)sn;
    P[5] = (float)c;
    P[6] = 0.0f;
    P[7] = (float)py;
    P[8] = 0.0f;
    P[9] = 0.0f;
    P[10] = 1.0f;
    P[11] = 0.0f;

    /* obstacles seen from this sweep: centre_s = R^T (centre - T), yaw_s = yaw - psi */
    double lc[64][4]; /* cx, cy, cos(-yaw_s), sin(-yaw_s) */
    int nobs = (int)num_obs;
    for (int k = 0; k < nobs; ++k) {
      const double* o = obs + 7 * k;
      double dx = o[0] - px, dy = o[1] - py;
      double sx = c * dx + sn * dy;
      double sy = -sn * dx + c * dy;
      double ys = o[6] - psi;
      lc[k][0] = sx;
      lc[k][1] = sy;
      lc[k][2] = cos(-ys);
      lc[k][3] = sin(-ys);
    }

    double phase = rng_uniform(&r, 0.0, 2.0 * kPi / na);
    for (int b = 0; b < nb; ++b) {
      double el = (nb == 1) ? sc->elev_lo_deg * kDeg
                            : (sc->elev_lo_deg + (sc->elev_hi_deg - sc->elev_lo_deg) * b / (nb - 1)) * kDeg;
      double ce = cos(el), se = sin(el);
      for (int a = 0; a < na; ++a) {
        double az = phase + 2.0 * kPi * a / na;
        double d[3] = {ce * cos(az), ce * sin(az), se};
        double t = INFINITY;
        if (d[2] < -1e-12) t = -sc->sensor_h / d[2];
        for (int k = 0; k < nobs; ++k) {
          const double* o = obs + 7 * k;
          /* ray in the box frame (box centred at (lc0, lc1, o[2])) */
          double ox = 0.0 - lc[k][0], oy = 0.0 - lc[k][1], oz = sc->sensor_h - o[2];
          double cb = lc[k][2], sb = lc[k][3];
          double ob[3] = {cb * ox - sb * oy, sb * ox + cb * oy, oz};
          double db[3] = {cb * d[0] - sb * d[1], sb * d[0] + cb * d[1], d[2]};
          double h[3] = {0.5 * o[3], 0.5 * o[4], 0.5 * o[5]};
          double tb = ray_box(ob, db, h);
          if (tb < t) t = tb;
        }
        double noise = rng_normal(&r) * sc->range_sigma;
        double inten = rng_uniform(&r, 0.0, 255.0);
        double rr;
        if (t > sc->r_max) {
          rr = sc->r_max;
        } else {
          rr = t + noise;
          if (rr < 0.05) rr = 0.05;
        }
        int64_t i = offset + (int64_t)s * per_sweep + (int64_t)b * na + a;
        feat[0 * stride + i] = (float)(rr * d[0]);
        feat[1 * stride + i] = (float)(rr * d[1]);
        feat[2 * stride + i] = (float)(sc->sensor_h + rr * d[2]);
        if (sc->num_features > 3) feat[3 * stride + i] = (float)inten;
        if (sc->num_features > 4) feat[4 * stride + i] = (float)(s * sc->sweep_dt);
        for (int cc = 5; cc < sc->num_features; ++cc) feat[(int64_t)cc * stride + i] = 0.0f;
        sweep_ids[i] = (uint8_t)s;
      }
    }
  }
  return (int64_t)S * per_sweep;
}

/* --------------------------------------------------------------- ROIs */
int64_t synth_rois(const synth_roi_recipe_t* rc, uint64_t seed, const double* obs, int64_t num_obs,
                   double* desc, uint8_t* budgets) {
  rng_t r;
  rng_seed(&r, seed ^ 0x5EED0F0A15ull);
  int64_t n = 0;
  int on = rc->num_on_obstacles < num_obs ? rc->num_on_obstacles : (int)num_obs;
  /* footprints of detected obstacles */
  for (int k = 0; k < on; ++k) {
    const double* o = obs + 7 * k;
    double* d = desc + 6 * n;
    d[0] = o[0];
    d[1] = o[1];
    d[2] = o[3];
    d[3] = o[4];
    d[4] = o[6];
    d[5] = rc->margin;
    ++n;
  }
  /* motion-extrapolated copies of the first obstacles (the second member
   * of the current/extrapolated footprint union), shifted along heading */
  for (int k = 0; k < rc->num_extrapolated && k < on; ++k) {
    const double* o = obs + 7 * k;
    double* d = desc + 6 * n;
    double shift = rc->extrap_speed * rc->extrap_dt;
    d[0] = o[0] + shift * cos(o[6]);
    d[1] = o[1] + shift * sin(o[6]);
    d[2] = o[3];
    d[3] = o[4];
    d[4] = o[6];
    d[5] = rc->margin;
    ++n;
  }
  /* free-standing boxes; the last num_overlapping of them are placed on top
   * of a random earlier ROI */
  for (int k = 0; k < rc->num_random; ++k) {
    double* d = desc + 6 * n;
    double len = rc->rand_len * rng_uniform(&r, 0.9, 1.1);
    double wid = rc->rand_wid * rng_uniform(&r, 0.9, 1.1);
    double yaw = rng_uniform(&r, 0.0, 2.0 * kPi);
    double cx, cy;
    if (k >= rc->num_random - rc->num_overlapping && n > 0) {
      int64_t j = rng_int(&r, 0, (int)(n - 1));
      const double* e = desc + 6 * j;
      cx = e[0] + rng_uniform(&r, -0.5, 0.5) * e[2];
      cy = e[1] + rng_uniform(&r, -0.5, 0.5) * e[2];
    } else {
      cx = rng_uniform(&r, -rc->rand_extent, rc->rand_extent);
      cy = rng_uniform(&r, -rc->rand_extent, rc->rand_extent);
    }
    d[0] = cx;
    d[1] = cy;
    d[2] = len;
    d[3] = wid;
    d[4] = yaw;
    d[5] = rc->margin;
    ++n;
  }
  for (int64_t k = 0; k < n; ++k) budgets[k] = (uint8_t)rng_int(&r, rc->budget_lo, rc->budget_hi);
  return n;
}
