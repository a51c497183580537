/* Host-only driver for the sanitizer build (AddressSanitizer and
 * UndefinedBehaviorSanitizer) of the CPU code: the synthetic-input generator
 * (synth/gen.c), the oracle (oracle/oracle.c) and the temporal-ROI selector
 * of the library (roi_policy.cpp, host code).  It runs each entry point on a
 * small seeded workload, including edge cases (an empty frame, budgets 0,
 * one sweep, the background keep rate), and prints a checksum; the
 * sanitizers abort the process on the first memory error or undefined
 * operation.  Built and run by tests/test_host_sanitizers.py with gcc/g++. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "gen.h"
#include "mmbev.h"
#include "oracle.h"

static uint64_t mix(uint64_t h, uint64_t v) { return (h ^ v) * 0x100000001b3ull; }

static void* xcalloc(size_t n, size_t sz) {
  void* p = calloc(n ? n : 1, sz);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

/* One batch of frames through the oracle's whole path and its add-ons. */
static uint64_t run_batch(int frames, int sweeps, int features, int empty_frame, float rho, uint64_t seed) {
  synth_scene_t sc;
  memset(&sc, 0, sizeof sc);
  sc.beams = 8;
  sc.azimuths = 96;
  sc.elev_lo_deg = -25.0;
  sc.elev_hi_deg = 5.0;
  sc.sensor_h = 1.8;
  sc.range_sigma = 0.02;
  sc.r_max = 60.0;
  sc.num_sweeps = sweeps;
  sc.num_features = features;
  sc.sweep_dt = 0.05;
  sc.speed_lo = 0.0;
  sc.speed_hi = 12.0;
  sc.yawrate_lo = -0.3;
  sc.yawrate_hi = 0.3;
  sc.num_obstacles = 6;
  sc.obs_len = 4.5;
  sc.obs_wid = 1.9;
  sc.obs_hgt = 1.7;
  sc.obs_jitter = 0.1;
  sc.obs_r_lo = 3.0;
  sc.obs_r_hi = 25.0;
  synth_roi_recipe_t rc;
  memset(&rc, 0, sizeof rc);
  rc.num_on_obstacles = 4;
  rc.num_extrapolated = 2;
  rc.num_random = 3;
  rc.num_overlapping = 1;
  rc.extrap_speed = 5.0;
  rc.extrap_dt = 0.5;
  rc.rand_extent = 30.0;
  rc.rand_len = 4.0;
  rc.rand_wid = 2.0;
  rc.margin = 0.5;
  rc.budget_lo = 0;
  rc.budget_hi = sweeps;

  const int64_t per_frame = (int64_t)sweeps * sc.beams * sc.azimuths;
  const int64_t cap_points = per_frame * frames;
  float* feat = xcalloc((size_t)(cap_points * features), sizeof(float));
  uint8_t* sweep_ids = xcalloc((size_t)cap_points, 1);
  float* poses = xcalloc((size_t)frames * sweeps * 12, sizeof(float));
  int64_t* frame_off = xcalloc((size_t)frames + 1, sizeof(int64_t));
  double* desc = xcalloc((size_t)frames * 16 * 6, sizeof(double));
  uint8_t* budgets = xcalloc((size_t)frames * 16, 1);
  int32_t* roi_off = xcalloc((size_t)frames + 1, sizeof(int32_t));
  double obs[64 * 7];
  int64_t n = 0;
  int32_t r = 0;
  for (int b = 0; b < frames; ++b) {
    frame_off[b] = n;
    roi_off[b] = r;
    if (b == empty_frame) continue;  /* no points and no ROIs */
    const int64_t no = synth_obstacles(&sc, seed + 17u * (uint64_t)b, obs);
    const int64_t w = synth_frame(&sc, seed + 31u * (uint64_t)b, obs, no, feat, cap_points, n, sweep_ids,
                                  poses + (size_t)b * sweeps * 12);
    if (w < 0) exit(3);
    n += w;
    r += (int32_t)synth_rois(&rc, seed + 7u * (uint64_t)b, obs, no, desc + (size_t)r * 6, budgets + r);
  }
  frame_off[frames] = n;
  roi_off[frames] = r;

  oracle_roi* rois = xcalloc((size_t)r, sizeof(oracle_roi));
  for (int32_t j = 0; j < r; ++j) {
    const double* d = desc + (size_t)j * 6;
    oracle_make_roi(d[0], d[1], d[2], d[3], d[4], d[5], &rois[j]);
  }
  oracle_grid g;
  memset(&g, 0, sizeof g);
  g.range_min[0] = -32.0f;
  g.range_min[1] = -32.0f;
  g.range_min[2] = -3.0f;
  g.voxel_size[0] = 0.25f;
  g.voxel_size[1] = 0.25f;
  g.voxel_size[2] = 0.5f;
  g.dims[0] = 256;
  g.dims[1] = 256;
  g.dims[2] = 16;
  g.max_points = 5;
  g.max_voxels = 300;
  g.num_sweeps = sweeps;
  g.num_frames = frames;

  const size_t rows = (size_t)frames * (size_t)g.max_voxels;
  int32_t* coords = xcalloc(rows * 4, sizeof(int32_t));
  int32_t* counts = xcalloc(rows, sizeof(int32_t));
  float* feats = xcalloc(rows * (size_t)features, sizeof(float));
  int32_t* pidx = xcalloc(rows * (size_t)g.max_points, sizeof(int32_t));
  int64_t* voff = xcalloc((size_t)frames + 1, sizeof(int64_t));
  const int64_t V = rho > 0.0f
                        ? oracle_roi_voxelize_bg(feat, cap_points, features, n, frame_off, sweep_ids, poses, rois,
                                                 roi_off, budgets, &g, rho, seed, coords, counts, feats, pidx, voff)
                        : oracle_roi_voxelize(feat, cap_points, features, n, frame_off, sweep_ids, poses, rois, roi_off,
                                              budgets, &g, coords, counts, feats, pidx, voff);
  if (V < 0) exit(4);
  uint64_t h = mix(0xcbf29ce484222325ull, (uint64_t)V);
  for (int64_t v = 0; v < V; ++v) h = mix(h, (uint64_t)(uint32_t)counts[v] ^ ((uint64_t)(uint32_t)coords[4 * v + 3] << 32));

  /* keep lists alone */
  uint64_t* keys = xcalloc((size_t)n, sizeof(uint64_t));
  int64_t* idx = xcalloc((size_t)n, sizeof(int64_t));
  const int64_t K = oracle_keep(feat, cap_points, features, n, frame_off, sweep_ids, poses, rois, roi_off, budgets, &g,
                                keys, idx);
  if (K < 0) exit(5);
  h = mix(h, (uint64_t)K);
  printf("batch frames=%d voxels=%lld kept=%lld\n", frames, (long long)V, (long long)K);

  /* ScatterToBEV */
  const size_t map_n = (size_t)frames * (size_t)features * g.dims[2] * g.dims[1] * g.dims[0];
  float* map = xcalloc(map_n, sizeof(float));
  if (oracle_scatter_to_bev(coords, feats, voff, frames, features, g.dims, map) != 0) exit(6);
  double acc = 0.0;
  for (size_t i = 0; i < map_n; ++i) acc += map[i];
  h = mix(h, (uint64_t)(int64_t)llround(acc * 16.0));

  /* connected components of the occupied cells */
  oracle_cc_params p = {2, 16, 1, 8, 1, 0};
  oracle_cluster* cl = xcalloc((size_t)(V > 0 ? V : 1), sizeof(oracle_cluster));
  int64_t* coff = xcalloc((size_t)frames + 1, sizeof(int64_t));
  int32_t* labels = xcalloc((size_t)(V > 0 ? V : 1), sizeof(int32_t));
  const int64_t ncl = oracle_clusters(coords, counts, voff, frames, g.dims, &p, cl, coff, labels);
  if (ncl < 0) exit(7);
  h = mix(h, (uint64_t)ncl);

  free(feat); free(sweep_ids); free(poses); free(frame_off); free(desc); free(budgets); free(roi_off);
  free(rois); free(coords); free(counts); free(feats); free(pidx); free(voff); free(keys); free(idx);
  free(map); free(cl); free(coff); free(labels);
  return h;
}

/* The library's temporal-ROI selector on random detection caches. */
static uint64_t run_selector(uint64_t seed) {
  const int frames = 5;
  int32_t det_off[6] = {0, 7, 7, 19, 20, 32};  /* frame 1 has no detection: the fallback box */
  const int nd = det_off[frames];
  mmbev_detection_t* dets = xcalloc((size_t)nd, sizeof(mmbev_detection_t));
  uint64_t s = seed;
  for (int i = 0; i < nd; ++i) {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    const double u = (double)(s >> 11) / 9007199254740992.0;
    dets[i].x = -20.0 + 60.0 * u;
    dets[i].y = -15.0 + 30.0 * fmod(u * 7.0, 1.0);
    dets[i].yaw = 6.28 * fmod(u * 13.0, 1.0);
    dets[i].length = 0.6 + 4.0 * fmod(u * 3.0, 1.0);
    dets[i].width = 0.6 + 1.5 * fmod(u * 5.0, 1.0);
    dets[i].vx = -8.0 + 16.0 * fmod(u * 11.0, 1.0);
    dets[i].vy = -2.0 + 4.0 * fmod(u * 17.0, 1.0);
    dets[i].cls = (int32_t)(s >> 62) % 3;
  }
  mmbev_ego_t ego[5];
  for (int b = 0; b < frames; ++b) {
    ego[b].speed = 2.0 + 5.0 * b;
    ego[b].dx = 0.1 * b;
    ego[b].dy = 0.01 * b;
    ego[b].dyaw = 0.02 * (b - 2);
  }
  mmbev_policy_t pol;
  memset(&pol, 0, sizeof pol);
  pol.dt = 0.5; pol.margin = 0.5; pol.a_brake = 6.0; pol.d_min = 2.0;
  pol.theta_max_deg = 60.0; pol.theta_min_deg = 15.0; pol.speed_wide = 5.0; pol.speed_narrow = 30.0;
  pol.tau_vru = 1.5; pol.tau_motorized = 2.5; pol.r_coll = 2.0; pol.slow_speed = 5.0;
  pol.dense_count = 10; pol.n_full = 10; pol.n_reduced = 5; pol.max_optional = 4;
  pol.fallback_length = 108.0; pol.fallback_width = 108.0;
  const int nr = 2 * nd + frames;
  mmbev_roi_t* rois = xcalloc((size_t)nr, sizeof(mmbev_roi_t));
  uint8_t* bud = xcalloc((size_t)nr, 1);
  int32_t roff[6];
  mmbev_criticality_t* crit = xcalloc((size_t)nd, sizeof(mmbev_criticality_t));
  int32_t sweeps[5];
  if (mmbev_build_rois(dets, det_off, frames, ego, &pol, rois, bud, roff, crit, sweeps) != MMBEV_OK) exit(8);
  uint64_t h = 0x84222325cbf29ce4ull;
  for (int i = 0; i <= frames; ++i) h = mix(h, (uint64_t)roff[i]);
  for (int i = 0; i < roff[frames]; ++i) h = mix(h, bud[i]);
  for (int i = 0; i < nd; ++i) h = mix(h, (uint64_t)crit[i].rank * 8u + (uint64_t)crit[i].flags);
  /* rejected arguments write nothing and report the error */
  pol.n_reduced = 0;
  if (mmbev_build_rois(dets, det_off, frames, ego, &pol, rois, bud, roff, crit, sweeps) == MMBEV_OK) exit(9);
  free(dets); free(rois); free(bud); free(crit);
  return h;
}

int main(void) {
  uint64_t h = 0;
  h ^= run_batch(3, 4, 5, 1, 0.0f, 11);   /* an empty frame in the middle */
  h ^= run_batch(2, 1, 3, -1, 0.0f, 12);  /* one sweep, three features */
  h ^= run_batch(2, 3, 8, -1, 0.25f, 13); /* eight features, background keep rate */
  h ^= run_selector(21);
  printf("checksum %016llx\n", (unsigned long long)h);
  return 0;
}
