// Criticality-ranked temporal-ROI selector and the sweep-count knob of the
// latency-aware coordinator (Sec. IV-C, IV-G): detections of frame t-1 in,
// ROI records and per-ROI sweep budgets for mmbev_roi_voxelize out.  Host
// code: a frame has tens to hundreds of detections, and its outputs are
// arguments of the device call that follows.  Double precision throughout,
// every expression evaluated in the order the header states (no fused
// multiply-adds: the library is built with -ffp-contract=off).
#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

#include "mmbev.h"

namespace {

constexpr double kPi = 3.14159265358979323846;

bool fin(double v) { return std::isfinite(v); }

bool policy_ok(const mmbev_policy_t& p) {
  const double all[] = {p.dt, p.margin, p.a_brake, p.d_min, p.theta_max_deg, p.theta_min_deg, p.speed_wide,
                        p.speed_narrow, p.tau_vru, p.tau_motorized, p.r_coll, p.slow_speed, p.fallback_length,
                        p.fallback_width};
  for (double v : all)
    if (!fin(v)) return false;
  return p.dt > 0.0 && p.margin >= 0.0 && p.a_brake > 0.0 && p.d_min >= 0.0 && p.theta_min_deg >= 0.0 &&
         p.theta_min_deg <= p.theta_max_deg && p.theta_max_deg <= 90.0 && p.speed_wide <= p.speed_narrow &&
         p.tau_vru >= 0.0 && p.tau_motorized >= 0.0 && p.r_coll > 0.0 && p.dense_count >= 0 &&
         p.n_reduced >= 1 && p.n_reduced <= p.n_full && p.n_full <= 255 && p.max_optional >= 0 &&
         p.reserved == 0 && p.fallback_length >= 0.0 && p.fallback_width >= 0.0;
}

bool detection_ok(const mmbev_detection_t& d) {
  return fin(d.x) && fin(d.y) && fin(d.yaw) && fin(d.length) && fin(d.width) && fin(d.vx) && fin(d.vy) &&
         d.length >= 0.0 && d.width >= 0.0 && d.cls >= MMBEV_CLASS_VRU && d.cls <= MMBEV_CLASS_STATIC &&
         d.reserved == 0;
}

// Forward-cone half-angle (radians) at ego speed v: piecewise linear.
double cone_half_angle(const mmbev_policy_t& p, double v) {
  double deg;
  if (v <= p.speed_wide)
    deg = p.theta_max_deg;
  else if (v >= p.speed_narrow)
    deg = p.theta_min_deg;
  else
    deg = p.theta_max_deg + (p.theta_min_deg - p.theta_max_deg) * (v - p.speed_wide) / (p.speed_narrow - p.speed_wide);
  return deg * kPi / 180.0;
}

// Eq. 8: time of closest approach of relative position (px, py) under
// relative velocity (wx, wy), if the approach comes within r_coll.
double time_to_collision(double px, double py, double wx, double wy, double r_coll) {
  const double w2 = wx * wx + wy * wy;
  if (!(w2 > 0.0)) return std::numeric_limits<double>::infinity();
  const double t = -(px * wx + py * wy) / w2;
  if (!(t > 0.0)) return std::numeric_limits<double>::infinity();
  const double mx = px + t * wx, my = py + t * wy;
  return std::sqrt(mx * mx + my * my) <= r_coll ? t : std::numeric_limits<double>::infinity();
}

struct Ranked {
  int32_t i;       // index in the frame
  bool mandatory;
  double ttc, dist;
};

}  // namespace

// ROI records from (cx, cy, length, width, yaw, margin) descriptors: the box
// of Eq. 1's footprint inflated by the margin r, with cos/sin of the yaw
// rounded once from double (the kernels never recompute them).
extern "C" mmbev_status_t mmbev_make_rois(const double* desc, int64_t count, mmbev_roi_t* out) {
  if (count < 0 || (count > 0 && (!desc || !out))) return MMBEV_ERR_INVALID_ARG;
  for (int64_t k = 0; k < count; ++k) {
    const double* d = desc + 6 * k;
    mmbev_roi_t r;
    r.cx = (float)d[0];
    r.cy = (float)d[1];
    r.cos_yaw = (float)std::cos(d[4]);
    r.sin_yaw = (float)std::sin(d[4]);
    r.ext_x = (float)(0.5 * d[2] + d[5]);
    r.ext_y = (float)(0.5 * d[3] + d[5]);
    r.reserved[0] = 0.0f;
    r.reserved[1] = 0.0f;
    out[k] = r;
  }
  return MMBEV_OK;
}

extern "C" mmbev_status_t mmbev_build_rois(const mmbev_detection_t* dets, const int32_t* det_offsets,
                                           int32_t num_frames, const mmbev_ego_t* ego,
                                           const mmbev_policy_t* policy, mmbev_roi_t* out_rois,
                                           uint8_t* out_budgets, int32_t* out_roi_offsets,
                                           mmbev_criticality_t* out_crit, int32_t* out_sweeps) {
  if (num_frames < 1 || !det_offsets || !ego || !policy || !out_rois || !out_budgets || !out_roi_offsets ||
      !out_crit || !out_sweeps)
    return MMBEV_ERR_INVALID_ARG;
  const mmbev_policy_t& P = *policy;
  if (!policy_ok(P) || det_offsets[0] != 0) return MMBEV_ERR_INVALID_ARG;
  for (int32_t b = 0; b < num_frames; ++b) {
    if (det_offsets[b + 1] < det_offsets[b]) return MMBEV_ERR_INVALID_ARG;
    const mmbev_ego_t& e = ego[b];
    if (!fin(e.speed) || !fin(e.dx) || !fin(e.dy) || !fin(e.dyaw)) return MMBEV_ERR_INVALID_ARG;
  }
  const int32_t total = det_offsets[num_frames];
  if (total > 0 && !dets) return MMBEV_ERR_INVALID_ARG;
  for (int32_t k = 0; k < total; ++k)
    if (!detection_ok(dets[k])) return MMBEV_ERR_INVALID_ARG;

  std::vector<Ranked> order;
  std::vector<double> desc;
  int32_t roi = 0;
  out_roi_offsets[0] = 0;
  for (int32_t b = 0; b < num_frames; ++b) {
    const mmbev_ego_t& e = ego[b];
    const int32_t lo = det_offsets[b], count = det_offsets[b + 1] - lo;
    const double c = std::cos(e.dyaw), s = std::sin(e.dyaw);
    const double d_max = std::max(P.d_min, e.speed * e.speed / (2.0 * P.a_brake));  // Eq. 4
    const double theta = cone_half_angle(P, e.speed);
    // step 4: the sweep count of the frame's optional ROIs
    const int32_t n = (e.speed < P.slow_speed || count >= P.dense_count) ? P.n_reduced : P.n_full;
    out_sweeps[b] = n;

    // steps 1-2: footprints in frame t, criticality
    order.clear();
    desc.assign((size_t)count * 12, 0.0);
    for (int32_t k = 0; k < count; ++k) {
      const mmbev_detection_t& d = dets[lo + k];
      const double x1 = d.x + d.vx * P.dt, y1 = d.y + d.vy * P.dt;  // b_i + v_i dt (Eq. 1), frame t-1
      const double X0 = c * d.x - s * d.y + e.dx, Y0 = s * d.x + c * d.y + e.dy;
      const double X1 = c * x1 - s * y1 + e.dx, Y1 = s * x1 + c * y1 + e.dy;
      const double yaw = d.yaw + e.dyaw;
      const double w0[6] = {X0, Y0, d.length, d.width, yaw, P.margin};
      const double w1[6] = {X1, Y1, d.length, d.width, yaw, P.margin};
      std::copy(w0, w0 + 6, desc.begin() + 12 * k);
      std::copy(w1, w1 + 6, desc.begin() + 12 * k + 6);
      const double wx = c * d.vx - s * d.vy - e.speed, wy = s * d.vx + c * d.vy;  // Eq. 8 relative velocity
      const double dist = std::sqrt(X1 * X1 + Y1 * Y1);
      const bool geom = X1 >= 0.0 && dist <= d_max && std::atan2(std::fabs(Y1), X1) <= theta;  // Eq. 3
      const double ttc = time_to_collision(X1, Y1, wx, wy, P.r_coll);
      const bool safety = d.cls != MMBEV_CLASS_STATIC &&
                          ttc <= (d.cls == MMBEV_CLASS_VRU ? P.tau_vru : P.tau_motorized);  // Eq. 5
      mmbev_criticality_t& o = out_crit[lo + k];
      o.ttc = ttc;
      o.flags = (geom ? MMBEV_CRIT_GEOM : 0) | (safety ? MMBEV_CRIT_SAFETY : 0) |
                ((geom || safety) ? MMBEV_CRIT_MANDATORY : 0);
      order.push_back({k, geom || safety, ttc, dist});
    }
    // step 3: ranking (a strict total order, so any sort gives this result)
    std::sort(order.begin(), order.end(), [](const Ranked& a, const Ranked& b) {
      if (a.mandatory != b.mandatory) return a.mandatory;
      if (a.ttc != b.ttc) return a.ttc < b.ttc;
      if (a.dist != b.dist) return a.dist < b.dist;
      return a.i < b.i;
    });
    int32_t optional_seen = 0;
    for (int32_t r = 0; r < count; ++r) {
      const Ranked& q = order[r];
      mmbev_criticality_t& o = out_crit[lo + q.i];
      o.rank = r;
      uint8_t budget = (uint8_t)P.n_full;
      if (!q.mandatory) {
        if (optional_seen++ < P.max_optional) {
          budget = (uint8_t)n;
        } else {
          budget = 0;
          o.flags |= MMBEV_CRIT_DROPPED;
        }
      }
      // step 5: two records per detection, in rank order
      mmbev_make_rois(desc.data() + 12 * q.i, 2, out_rois + roi);
      out_budgets[roi] = budget;
      out_budgets[roi + 1] = budget;
      roi += 2;
    }
    if (count == 0 && P.fallback_length > 0.0 && P.fallback_width > 0.0) {
      const double fb[6] = {0.0, 0.0, P.fallback_length, P.fallback_width, 0.0, 0.0};
      mmbev_make_rois(fb, 1, out_rois + roi);
      out_budgets[roi] = (uint8_t)P.n_full;
      roi += 1;
    }
    out_roi_offsets[b + 1] = roi;
  }
  return MMBEV_OK;
}
