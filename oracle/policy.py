"""Oracle of the criticality-ranked temporal-ROI selector and the sweep-count
knob of the coordinator -- TEST INFRASTRUCTURE (same rules as the rest of
``oracle/``: only the tests, the smoke check and the benchmark's CPU leg use
it; the product never does).

Plain Python floats (IEEE double, no fused operations), one detection at a
time, following the paper:
  Eq. 1   ROI_L: the union over detections of the box at t-1 and the box
          moved by v*dt, each buffered by the margin r (two oriented records
          per detection, taken into frame t by the ego motion);
  Eq. 3   geometry-critical: x >= 0, |p| <= d_max, |atan(y/x)| <= theta;
  Eq. 4   d_max = max(d_min, v_ego^2 / (2 a_brake));
  Sec. IV-C theta piecewise linear in ego speed between its bounds;
  Eq. 8   t* = -p.v / |v|^2, TTC = t* if t* > 0 and the miss distance
          |p + t* v| <= R_coll, else infinity; v relative (object minus ego);
  Eq. 5   safety-critical: TTC <= tau of the class (static: never);
  Sec. IV-C mandatory = geometry or safety; ROIs ranked by criticality;
  Sec. IV-G sweep count reduced from n_full to n_reduced when the ego is
          slow or the scene dense; mandatory ROIs keep full fidelity;
          optional ones may be dropped.
"""
from __future__ import annotations

import math

import numpy as np

from . import make_rois

VRU, MOTORIZED, STATIC = 0, 1, 2
GEOM, SAFETY, MANDATORY, DROPPED = 1, 2, 4, 8


def braking_distance(speed: float, a_brake: float, d_min: float) -> float:
    """Eq. 4."""
    return max(d_min, speed * speed / (2.0 * a_brake))


def cone_half_angle(speed: float, pol: dict) -> float:
    """The forward-cone half-angle (radians): theta_max at or below speed_wide,
    theta_min at or above speed_narrow, linear in between (Sec. IV-C)."""
    if speed <= pol["speed_wide"]:
        deg = pol["theta_max_deg"]
    elif speed >= pol["speed_narrow"]:
        deg = pol["theta_min_deg"]
    else:
        deg = pol["theta_max_deg"] + (pol["theta_min_deg"] - pol["theta_max_deg"]) * (speed - pol["speed_wide"]) / (
            pol["speed_narrow"] - pol["speed_wide"])
    return deg * math.pi / 180.0


def ttc(px: float, py: float, wx: float, wy: float, r_coll: float) -> float:
    """Eq. 8: time of closest approach if it comes within r_coll, else inf."""
    w2 = wx * wx + wy * wy
    if not w2 > 0.0:
        return math.inf
    t = -(px * wx + py * wy) / w2
    if not t > 0.0:
        return math.inf
    mx, my = px + t * wx, py + t * wy
    return t if math.sqrt(mx * mx + my * my) <= r_coll else math.inf


def geometry_critical(px: float, py: float, d_max: float, theta: float) -> bool:
    """Eq. 3 (|atan(y/x)| taken as atan2(|y|, x), defined at x = 0)."""
    return px >= 0.0 and math.sqrt(px * px + py * py) <= d_max and math.atan2(abs(py), px) <= theta


def build_rois(dets: list[list[dict]], ego: list[dict], pol: dict) -> dict:
    """dets[b]: detections of frame b (dicts x, y, yaw, length, width, vx, vy,
    cls); ego[b]: speed, dx, dy, dyaw.  Returns ROI records (oracle ROI
    dtype), budgets, roi_offsets, per-detection ttc / flags / rank (in input
    order, frames concatenated) and the sweep count of each frame."""
    descs, budgets, offsets = [], [], [0]
    ttcs, flags, ranks, sweeps = [], [], [], []
    for frame, e in zip(dets, ego):
        c, s = math.cos(e["dyaw"]), math.sin(e["dyaw"])
        d_max = braking_distance(e["speed"], pol["a_brake"], pol["d_min"])
        theta = cone_half_angle(e["speed"], pol)
        slow_or_dense = e["speed"] < pol["slow_speed"] or len(frame) >= pol["dense_count"]
        n = pol["n_reduced"] if slow_or_dense else pol["n_full"]
        sweeps.append(n)
        rows = []
        for i, d in enumerate(frame):
            # Eq. 1: the box at t-1 and the box moved by v dt, into frame t
            x1, y1 = d["x"] + d["vx"] * pol["dt"], d["y"] + d["vy"] * pol["dt"]
            X0, Y0 = c * d["x"] - s * d["y"] + e["dx"], s * d["x"] + c * d["y"] + e["dy"]
            X1, Y1 = c * x1 - s * y1 + e["dx"], s * x1 + c * y1 + e["dy"]
            yaw = d["yaw"] + e["dyaw"]
            # criticality of the moved box
            wx, wy = c * d["vx"] - s * d["vy"] - e["speed"], s * d["vx"] + c * d["vy"]
            t = ttc(X1, Y1, wx, wy, pol["r_coll"])
            geom = geometry_critical(X1, Y1, d_max, theta)
            tau = pol["tau_vru"] if d["cls"] == VRU else pol["tau_motorized"]
            safety = d["cls"] != STATIC and t <= tau
            mand = geom or safety
            rows.append({"i": i, "mand": mand, "ttc": t, "dist": math.sqrt(X1 * X1 + Y1 * Y1),
                         "flags": (GEOM if geom else 0) | (SAFETY if safety else 0) | (MANDATORY if mand else 0),
                         "descs": [(X0, Y0, d["length"], d["width"], yaw, pol["margin"]),
                                   (X1, Y1, d["length"], d["width"], yaw, pol["margin"])]})
        # ranking: mandatory first, then ascending TTC, then distance, then input order
        ranked = sorted(rows, key=lambda q: (not q["mand"], q["ttc"], q["dist"], q["i"]))
        f_flags = [0] * len(frame)
        f_rank = [0] * len(frame)
        optional = 0
        for r, q in enumerate(ranked):
            f_rank[q["i"]] = r
            fl = q["flags"]
            if q["mand"]:
                bud = pol["n_full"]
            elif optional < pol["max_optional"]:
                bud = n
                optional += 1
            else:
                bud = 0
                optional += 1
                fl |= DROPPED
            f_flags[q["i"]] = fl
            descs.extend(q["descs"])
            budgets.extend([bud, bud])
        if not frame and pol["fallback_length"] > 0.0 and pol["fallback_width"] > 0.0:
            descs.append((0.0, 0.0, pol["fallback_length"], pol["fallback_width"], 0.0, 0.0))
            budgets.append(pol["n_full"])
        offsets.append(len(descs))
        ttcs.extend(q["ttc"] for q in sorted(rows, key=lambda q: q["i"]))
        flags.extend(f_flags)
        ranks.extend(f_rank)
    recs = make_rois(np.array(descs, dtype=np.float64).reshape(-1, 6))
    return {"rois": recs, "budgets": np.array(budgets, dtype=np.uint8), "roi_offsets": np.array(offsets, np.int32),
            "ttc": np.array(ttcs, dtype=np.float64), "flags": np.array(flags, dtype=np.int32),
            "rank": np.array(ranks, dtype=np.int32), "sweeps": np.array(sweeps, dtype=np.int32)}
