/*
 * CPU ORACLE for ROI-aware multi-sweep voxelisation -- TEST INFRASTRUCTURE.
 * Plain, single-threaded, deliberately unoptimised.  See oracle.h for the
 * definition this file follows step by step and for who may call it.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

void oracle_make_roi(double cx, double cy, double length, double width, double yaw, double margin,
                     oracle_roi* out) {
  out->cx = (float)cx;
  out->cy = (float)cy;
  out->cos_yaw = (float)cos(yaw);
  out->sin_yaw = (float)sin(yaw);
  out->ext_x = (float)(0.5 * length + margin);
  out->ext_y = (float)(0.5 * width + margin);
  out->unused0 = 0.0f;
  out->unused1 = 0.0f;
}

/* Sec. IV-D, Eq. 6: p' = R p + T, one fused chain per output row. */
void oracle_compensate(const float* P, float x, float y, float z, float* o) {
  o[0] = fmaf(P[0], x, fmaf(P[1], y, fmaf(P[2], z, P[3])));
  o[1] = fmaf(P[4], x, fmaf(P[5], y, fmaf(P[6], z, P[7])));
  o[2] = fmaf(P[8], x, fmaf(P[9], y, fmaf(P[10], z, P[11])));
}

/* Alg. 1 keep test against one box of ROI_L (Eq. 1), bird's-eye view only:
 * rotate the offset from the centre into the box frame, compare with the
 * half extents (edges inclusive). */
int32_t oracle_inside(const oracle_roi* r, float x, float y) {
  float dx = x - r->cx;
  float dy = y - r->cy;
  float s_dy = r->sin_yaw * dy;
  float s_dx = r->sin_yaw * dx;
  float lx = fmaf(r->cos_yaw, dx, s_dy);
  float ly = fmaf(r->cos_yaw, dy, -s_dx);
  return fabsf(lx) <= r->ext_x && fabsf(ly) <= r->ext_y;
}

/* The n-th output (n >= 1) of the SplitMix64 generator (Steele, Lea and
 * Flood, OOPSLA 2014, in the form of Vigna's public-domain reference code)
 * whose state starts at `seed`: the state advances by the golden-ratio
 * increment per output and each output is the state mixed by two
 * xor-shift-multiply rounds and a final xor-shift. */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t n) {
  uint64_t z = seed + n * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Alg. 1 keep rate of out-of-ROI points, as a 24-bit threshold:
 * round(rho * 2^24), clamped to [0, 2^24] (NaN and rho <= 0 give 0). */
uint32_t oracle_background_threshold(float rho) {
  double t = (double)rho * 16777216.0;
  if (!(t > 0.0)) return 0;
  if (t >= 16777216.0) return 16777216u;
  return (uint32_t)floor(t + 0.5);
}

/* Whether point i is drawn for the background keep: the top 24 bits of the
 * generator's (i + 1)-th output lie below the threshold. */
int32_t oracle_background_keep(uint64_t seed, uint32_t threshold, int64_t i) {
  return (uint32_t)(oracle_splitmix64(seed, (uint64_t)i + 1u) >> 40) < threshold;
}

/* Alg. 1 "Voxelize": grid coordinate of p' on each axis. */
int32_t oracle_quantize(const oracle_grid* g, const float* p, int32_t* ijk) {
  for (int d = 0; d < 3; ++d) {
    float f = (p[d] - g->range_min[d]) / g->voxel_size[d];
    if (!(f >= 0.0f && f < (float)g->dims[d])) return 0;
    ijk[d] = (int32_t)f;
  }
  return 1;
}

static int bad_args(int32_t C, int64_t N, const oracle_grid* g) {
  if (C < 3 || N < 0 || !g) return 1;
  if (g->num_frames < 1 || g->num_sweeps < 1 || g->max_points < 1 || g->max_voxels < 1) return 1;
  for (int d = 0; d < 3; ++d)
    if (g->dims[d] < 1) return 1;
  return 0;
}

/* Steps 1-4 of oracle.h for frame b, appended to (keys, idx); out-of-ROI
 * points are drawn with threshold bg_thr (0: none). */
static int64_t keep_frame(int32_t b, const float* feat, int64_t stride, const int64_t* frame_offsets,
                          const uint8_t* sweep_ids, const float* poses, const oracle_roi* rois,
                          const int32_t* roi_offsets, const uint8_t* budgets, const oracle_grid* g,
                          uint32_t bg_thr, uint64_t bg_seed, uint64_t* keys, int64_t* idx, int64_t k) {
  const int S = g->num_sweeps;
  const uint64_t Dx = (uint64_t)g->dims[0], Dy = (uint64_t)g->dims[1], Dz = (uint64_t)g->dims[2];
  for (int64_t i = frame_offsets[b]; i < frame_offsets[b + 1]; ++i) {
    int s = sweep_ids[i];
    if (s >= S) continue;
    float p[3];
    oracle_compensate(poses + ((int64_t)b * S + s) * 12, feat[i], feat[stride + i], feat[2 * stride + i], p);
    int keep = 0;
    for (int32_t j = roi_offsets[b]; j < roi_offsets[b + 1] && !keep; ++j)
      if (s < budgets[j] && oracle_inside(&rois[j], p[0], p[1])) keep = 1;
    if (!keep) keep = oracle_background_keep(bg_seed, bg_thr, i);
    if (!keep) continue;
    int32_t ijk[3];
    if (!oracle_quantize(g, p, ijk)) continue;
    keys[k] = (((uint64_t)b * Dz + (uint64_t)ijk[2]) * Dy + (uint64_t)ijk[1]) * Dx + (uint64_t)ijk[0];
    idx[k] = i;
    ++k;
  }
  return k;
}

int64_t oracle_keep_bg(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                       const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                       const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                       const oracle_grid* g, float rho_out, uint64_t seed, uint64_t* keys, int64_t* idx) {
  if (bad_args(num_features, num_points, g)) return -1;
  const uint32_t thr = oracle_background_threshold(rho_out);
  int64_t k = 0;
  for (int32_t b = 0; b < g->num_frames; ++b)
    k = keep_frame(b, feat, stride, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets, g, thr, seed,
                   keys, idx, k);
  return k;
}

int64_t oracle_keep(const float* feat, int64_t stride, int32_t num_features, int64_t num_points,
                    const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                    const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                    const oracle_grid* g, uint64_t* keys, int64_t* idx) {
  return oracle_keep_bg(feat, stride, num_features, num_points, frame_offsets, sweep_ids, poses, rois,
                        roi_offsets, budgets, g, 0.0f, 0, keys, idx);
}

typedef struct {
  uint64_t key;
  int64_t idx;
} pair_t;

static int cmp_pair(const void* a, const void* b) {
  const pair_t* x = (const pair_t*)a;
  const pair_t* y = (const pair_t*)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
  return 0;
}

typedef struct {
  int64_t start; /* first pair of the voxel in sorted order */
  int64_t run;   /* number of kept points that fell in it */
  int64_t first; /* smallest point index in it */
  int64_t pos;   /* position in key order */
} voxel_t;

static int cmp_first(const void* a, const void* b) {
  const voxel_t* x = (const voxel_t*)a;
  const voxel_t* y = (const voxel_t*)b;
  return x->first < y->first ? -1 : (x->first > y->first ? 1 : 0);
}

static int cmp_pos(const void* a, const void* b) {
  const voxel_t* x = (const voxel_t*)a;
  const voxel_t* y = (const voxel_t*)b;
  return x->pos < y->pos ? -1 : (x->pos > y->pos ? 1 : 0);
}

int64_t oracle_roi_voxelize_bg(const float* feat, int64_t stride, int32_t C, int64_t N,
                               const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                               const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                               const oracle_grid* g, float rho_out, uint64_t seed, int32_t* out_coords,
                               int32_t* out_counts, float* out_feats, int32_t* out_point_idx,
                               int64_t* out_voxel_offsets) {
  if (bad_args(C, N, g)) return -1;
  const uint32_t bg_thr = oracle_background_threshold(rho_out);
  const int S = g->num_sweeps;
  const int M = g->max_points;
  const int64_t cap = g->max_voxels;
  const uint64_t Dx = (uint64_t)g->dims[0], Dy = (uint64_t)g->dims[1], Dz = (uint64_t)g->dims[2];
  int64_t total = 0;
  out_voxel_offsets[0] = 0;
  for (int32_t b = 0; b < g->num_frames; ++b) {
    int64_t n_b = frame_offsets[b + 1] - frame_offsets[b];
    uint64_t* keys = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(n_b > 0 ? n_b : 1));
    int64_t* idx = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_b > 0 ? n_b : 1));
    /* steps 1-4 */
    int64_t K = keep_frame(b, feat, stride, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets, g,
                           bg_thr, seed, keys, idx, 0);
    /* step 5: sort (key, index) */
    pair_t* pairs = (pair_t*)malloc(sizeof(pair_t) * (size_t)(K > 0 ? K : 1));
    for (int64_t k = 0; k < K; ++k) {
      pairs[k].key = keys[k];
      pairs[k].idx = idx[k];
    }
    qsort(pairs, (size_t)K, sizeof(pair_t), cmp_pair);
    /* equal keys form a voxel */
    voxel_t* vox = (voxel_t*)malloc(sizeof(voxel_t) * (size_t)(K > 0 ? K : 1));
    int64_t V = 0;
    for (int64_t k = 0; k < K; ++k) {
      if (k == 0 || pairs[k].key != pairs[k - 1].key) {
        vox[V].start = k;
        vox[V].run = 0;
        vox[V].first = pairs[k].idx;
        vox[V].pos = V;
        ++V;
      }
      vox[V - 1].run += 1;
    }
    /* step 6: per-frame voxel cap by first appearance */
    int64_t Vout = V;
    if (V > cap) {
      qsort(vox, (size_t)V, sizeof(voxel_t), cmp_first);
      Vout = cap;
      qsort(vox, (size_t)Vout, sizeof(voxel_t), cmp_pos);
    }
    /* step 7: outputs and means */
    for (int64_t v = 0; v < Vout; ++v) {
      int64_t row = total + v;
      const voxel_t* vx = &vox[v];
      uint64_t key = pairs[vx->start].key;
      uint64_t ix = key % Dx, rest = key / Dx;
      uint64_t iy = rest % Dy;
      rest /= Dy;
      uint64_t iz = rest % Dz;
      out_coords[row * 4 + 0] = b;
      out_coords[row * 4 + 1] = (int32_t)iz;
      out_coords[row * 4 + 2] = (int32_t)iy;
      out_coords[row * 4 + 3] = (int32_t)ix;
      int64_t cnt = vx->run < M ? vx->run : M;
      out_counts[row] = (int32_t)cnt;
      for (int m = 0; m < M; ++m)
        out_point_idx[row * M + m] = m < cnt ? (int32_t)pairs[vx->start + m].idx : -1;
      for (int c = 0; c < C; ++c) {
        double sum = 0.0;
        for (int64_t m = 0; m < cnt; ++m) {
          int64_t i = pairs[vx->start + m].idx;
          float val;
          if (c < 3) {
            float p[3];
            int s = sweep_ids[i];
            oracle_compensate(poses + ((int64_t)b * S + s) * 12, feat[i], feat[stride + i],
                              feat[2 * stride + i], p);
            val = p[c];
          } else {
            val = feat[(int64_t)c * stride + i];
          }
          sum += (double)val;
        }
        out_feats[row * C + c] = (float)(sum / (double)cnt);
      }
    }
    total += Vout;
    out_voxel_offsets[b + 1] = total;
    free(vox);
    free(pairs);
    free(idx);
    free(keys);
  }
  return total;
}

int64_t oracle_roi_voxelize(const float* feat, int64_t stride, int32_t C, int64_t N,
                            const int64_t* frame_offsets, const uint8_t* sweep_ids, const float* poses,
                            const oracle_roi* rois, const int32_t* roi_offsets, const uint8_t* budgets,
                            const oracle_grid* g, int32_t* out_coords, int32_t* out_counts,
                            float* out_feats, int32_t* out_point_idx, int64_t* out_voxel_offsets) {
  return oracle_roi_voxelize_bg(feat, stride, C, N, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets,
                                g, 0.0f, 0, out_coords, out_counts, out_feats, out_point_idx, out_voxel_offsets);
}

/* Step 8 (ScatterToBEV, Alg. 1; Sec. IV-F): clear the map, then one store
 * per voxel and feature at its coordinate, the height index folded into the
 * channel as c*Dz + iz. */
int32_t oracle_scatter_to_bev(const int32_t* coords, const float* feats, const int64_t* voxel_offsets,
                              int32_t B, int32_t C, const int32_t* dims, float* map) {
  if (B < 1 || C < 1 || dims[0] < 1 || dims[1] < 1 || dims[2] < 1) return -1;
  const int64_t Dx = dims[0], Dy = dims[1], Dz = dims[2];
  const int64_t total = (int64_t)B * C * Dz * Dy * Dx;
  for (int64_t e = 0; e < total; ++e) map[e] = 0.0f;
  for (int32_t b = 0; b < B; ++b) {
    for (int64_t v = voxel_offsets[b]; v < voxel_offsets[b + 1]; ++v) {
      const int32_t* q = coords + 4 * v;
      if (q[0] != b || q[1] < 0 || q[1] >= Dz || q[2] < 0 || q[2] >= Dy || q[3] < 0 || q[3] >= Dx) return -1;
      for (int32_t c = 0; c < C; ++c) {
        const int64_t channel = (int64_t)c * Dz + q[1];
        map[(((int64_t)b * C * Dz + channel) * Dy + q[2]) * Dx + q[3]] = feats[v * C + c];
      }
    }
  }
  return 0;
}

/* Step 9: per frame, occupied cells from the voxels in the layer band, then
 * a flood fill from every unlabelled occupied cell in ascending cell order;
 * the cell a fill starts from is the smallest of its component (every
 * smaller occupied cell was labelled by an earlier fill). */
int64_t oracle_clusters(const int32_t* coords, const int32_t* counts, const int64_t* voxel_offsets, int32_t B,
                        const int32_t* dims, const oracle_cc_params* p, oracle_cluster* out,
                        int64_t* cluster_offsets, int32_t* voxel_labels) {
  if (B < 1 || dims[0] < 1 || dims[1] < 1 || dims[2] < 1) return -1;
  if (p->cell_shift < 0 || p->cell_shift > 8 || p->min_cells < 1) return -1;
  if (p->connectivity != 4 && p->connectivity != 8) return -1;
  const int64_t Wx = ((int64_t)dims[0] + (1 << p->cell_shift) - 1) >> p->cell_shift;
  const int64_t Wy = ((int64_t)dims[1] + (1 << p->cell_shift) - 1) >> p->cell_shift;
  const int64_t ncell = Wx * Wy;
  static const int dx8[8] = {-1, 1, 0, 0, -1, 1, -1, 1}, dy8[8] = {0, 0, -1, 1, -1, -1, 1, 1};
  const int nn = p->connectivity;
  uint8_t* occ = (uint8_t*)malloc((size_t)ncell);
  int32_t* comp = (int32_t*)malloc(sizeof(int32_t) * (size_t)ncell);
  int64_t* stack = (int64_t*)malloc(sizeof(int64_t) * (size_t)ncell);
  int64_t total = 0;
  cluster_offsets[0] = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int64_t v0 = voxel_offsets[b], v1 = voxel_offsets[b + 1];
    memset(occ, 0, (size_t)ncell);
    for (int64_t c = 0; c < ncell; ++c) comp[c] = -1;
    for (int64_t v = v0; v < v1; ++v) {
      const int32_t* q = coords + 4 * v;
      if (q[0] != b || q[1] < 0 || q[1] >= dims[2] || q[2] < 0 || q[2] >= dims[1] || q[3] < 0 || q[3] >= dims[0]) {
        free(occ);
        free(comp);
        free(stack);
        return -1;
      }
      if (q[1] >= p->z_min && q[1] < p->z_max) occ[(int64_t)(q[2] >> p->cell_shift) * Wx + (q[3] >> p->cell_shift)] = 1;
    }
    /* flood fill: components numbered in order of their smallest cell */
    int64_t ncomp = 0;
    for (int64_t c = 0; c < ncell; ++c) {
      if (!occ[c] || comp[c] >= 0) continue;
      int64_t top = 0;
      stack[top++] = c;
      comp[c] = (int32_t)ncomp;
      while (top > 0) {
        const int64_t u = stack[--top];
        const int64_t ux = u % Wx, uy = u / Wx;
        for (int k = 0; k < nn; ++k) {
          const int64_t x = ux + dx8[k], y = uy + dy8[k];
          if (x < 0 || x >= Wx || y < 0 || y >= Wy) continue;
          const int64_t n = y * Wx + x;
          if (occ[n] && comp[n] < 0) {
            comp[n] = (int32_t)ncomp;
            stack[top++] = n;
          }
        }
      }
      ++ncomp;
    }
    /* per-component cell statistics; kept components get their output index */
    int64_t* size = (int64_t*)calloc((size_t)(ncomp > 0 ? ncomp : 1), sizeof(int64_t));
    int64_t* idx = (int64_t*)malloc(sizeof(int64_t) * (size_t)(ncomp > 0 ? ncomp : 1));
    for (int64_t c = 0; c < ncell; ++c)
      if (comp[c] >= 0) size[comp[c]] += 1;
    int64_t kept = 0;
    for (int64_t k = 0; k < ncomp; ++k) idx[k] = size[k] >= p->min_cells ? total + kept++ : -1;
    for (int64_t k = 0; k < ncomp; ++k) {
      if (idx[k] < 0) continue;
      oracle_cluster* o = &out[idx[k]];
      memset(o, 0, sizeof(*o));
      o->frame = b;
      o->root = -1;
      o->x0 = o->y0 = INT32_MAX;
      o->x1 = o->y1 = -1;
    }
    for (int64_t c = 0; c < ncell; ++c) {
      if (comp[c] < 0 || idx[comp[c]] < 0) continue;
      oracle_cluster* o = &out[idx[comp[c]]];
      const int32_t x = (int32_t)(c % Wx), y = (int32_t)(c / Wx);
      if (o->root < 0) o->root = (int32_t)c;
      o->cells += 1;
      if (x < o->x0) o->x0 = x;
      if (y < o->y0) o->y0 = y;
      if (x > o->x1) o->x1 = x;
      if (y > o->y1) o->y1 = y;
      o->sum_x += x;
      o->sum_y += y;
    }
    for (int64_t v = v0; v < v1; ++v) {
      const int32_t* q = coords + 4 * v;
      voxel_labels[v] = -1;
      if (q[1] < p->z_min || q[1] >= p->z_max) continue;
      const int32_t k = comp[(int64_t)(q[2] >> p->cell_shift) * Wx + (q[3] >> p->cell_shift)];
      if (idx[k] < 0) continue;
      voxel_labels[v] = (int32_t)idx[k];
      out[idx[k]].voxels += 1;
      out[idx[k]].points += counts[v];
    }
    total += kept;
    cluster_offsets[b + 1] = total;
    free(idx);
    free(size);
  }
  free(occ);
  free(comp);
  free(stack);
  return total;
}
