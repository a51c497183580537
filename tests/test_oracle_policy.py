"""Pins of the oracle's temporal-ROI selector and sweep-count knob (Sec.
IV-C Eq. 1, 3, 4, 5; Sec. IV-G Eq. 8 and budget management).

Closed forms for Eq. 4 and Eq. 8 and the cone angle; the paper's thresholds
(1.5 s and 2.5 s, 15-60 degrees, 10 and 5 sweeps); the Eq. 1 union checked
geometrically (points of the physical boxes, moved by homogeneous 3x3
transforms, fall in the records; points beyond the margin do not); the
ranking and budget rules as invariants over random caches.
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import synth
from oracle import policy as P

POL = dict(dt=0.5, margin=0.5, a_brake=6.0, d_min=10.0, theta_max_deg=60.0, theta_min_deg=15.0, speed_wide=5.0,
           speed_narrow=30.0, tau_vru=1.5, tau_motorized=2.5, r_coll=2.0, slow_speed=5.0, dense_count=64, n_full=10,
           n_reduced=5, max_optional=64, fallback_length=108.0, fallback_width=108.0)


def det(x, y, vx=0.0, vy=0.0, cls=1, yaw=0.0, length=4.0, width=2.0):
    return dict(x=x, y=y, vx=vx, vy=vy, cls=cls, yaw=yaw, length=length, width=width)


def ego(speed=0.0, dx=0.0, dy=0.0, dyaw=0.0):
    return dict(speed=speed, dx=dx, dy=dy, dyaw=dyaw)


def as_dicts(d, off, e):
    dets = [[{k: (int(r[k]) if k == "cls" else float(r[k])) for k in ("x", "y", "yaw", "length", "width", "vx",
                                                                       "vy", "cls")} for r in d[off[b]:off[b + 1]]]
            for b in range(len(off) - 1)]
    egos = [{k: float(r[k]) for k in ("speed", "dx", "dy", "dyaw")} for r in e]
    return dets, egos


def test_braking_distance_eq4():
    assert P.braking_distance(20.0, 5.0, 10.0) == 40.0
    assert P.braking_distance(5.0, 5.0, 10.0) == 10.0
    assert P.braking_distance(0.0, 6.0, 0.0) == 0.0


def test_cone_angle_piecewise():
    assert P.cone_half_angle(0.0, POL) == 60.0 * math.pi / 180.0
    assert P.cone_half_angle(5.0, POL) == 60.0 * math.pi / 180.0
    assert P.cone_half_angle(30.0, POL) == 15.0 * math.pi / 180.0
    assert P.cone_half_angle(99.0, POL) == 15.0 * math.pi / 180.0
    assert P.cone_half_angle(17.5, POL) == pytest.approx(37.5 * math.pi / 180.0, rel=1e-15)


def test_ttc_closed_forms_eq8():
    # head-on: 20 m ahead closing at 10 m/s
    assert P.ttc(20.0, 0.0, -10.0, 0.0, 2.0) == 2.0
    # receding, or no relative motion: never
    assert P.ttc(20.0, 0.0, 10.0, 0.0, 2.0) == math.inf
    assert P.ttc(20.0, 0.0, 0.0, 0.0, 2.0) == math.inf
    # crossing: closest approach at t* = 1 s, 10 m away: beyond R_coll
    assert P.ttc(10.0, 5.0, 0.0, -5.0, 2.0) == math.inf
    # crossing with a 1.5 m miss: t* = (p.v) / |v|^2 with p = (8, 1.5), v = (-4, 0) -> 2 s
    assert P.ttc(8.0, 1.5, -4.0, 0.0, 2.0) == 2.0
    assert P.ttc(8.0, 2.5, -4.0, 0.0, 2.0) == math.inf


def test_geometry_and_safety_thresholds():
    pol = dict(POL)
    # ego at 10 m/s: d_max = max(10, 100 / 12) = 10 m, cone 60 - 45 * 5 / 25 = 51 degrees
    out = P.build_rois([[det(5.0, 0.0, cls=2), det(5.0, 7.0, cls=2), det(-1.0, 0.0, cls=2), det(11.0, 0.0, cls=2)]],
                       [ego(10.0)], pol)
    geom = (out["flags"] & P.GEOM) != 0
    assert geom.tolist() == [True, False, False, False]  # 54.5 degrees off axis; behind; beyond 10 m
    # static objects are never safety-critical; VRU at TTC 2 s is not (1.5 s), a car at 2 s is (2.5 s)
    out = P.build_rois([[det(30.0, 0.0, cls=2), det(30.0, 0.0, cls=0), det(30.0, 0.0, cls=1)]], [ego(15.0)], pol)
    assert out["ttc"].tolist() == [2.0, 2.0, 2.0]
    assert ((out["flags"] & P.SAFETY) != 0).tolist() == [False, False, True]


def test_ranking_budgets_and_sweep_count():
    pol = dict(POL, max_optional=1)
    frame = [det(40.0, 30.0), det(30.0, 0.0, cls=1), det(-20.0, 3.0), det(8.0, 0.0, cls=0), det(-50.0, -50.0)]
    out = P.build_rois([frame], [ego(15.0)], pol)
    # ego at 15 m/s: d_max 18.75 m, cone 42 degrees.  Mandatory: the car 30 m ahead (TTC 2 s <= 2.5 s) and the
    # pedestrian 8 m ahead (in the cone, and TTC 0.53 s <= 1.5 s)
    mand = (out["flags"] & P.MANDATORY) != 0
    assert mand.tolist() == [False, True, False, True, False]
    # ranking: mandatory by TTC (pedestrian 0.53 s, car 2 s), then optional by distance
    assert out["rank"].tolist() == [3, 1, 2, 0, 4]
    # budgets per record pair in rank order: mandatory 10 sweeps; one optional kept at n = 10 (fast, sparse);
    # the rest dropped
    assert out["budgets"].tolist() == [10, 10, 10, 10, 10, 10, 0, 0, 0, 0]
    assert ((out["flags"] & P.DROPPED) != 0).tolist() == [True, False, False, False, True]
    assert out["sweeps"].tolist() == [10]
    # slow ego, or a dense scene: the reduced count for optional ROIs only
    out = P.build_rois([frame], [ego(2.0)], dict(POL))
    assert out["sweeps"].tolist() == [5]
    assert sorted(set(out["budgets"].tolist())) == [5, 10]
    out = P.build_rois([frame], [ego(15.0)], dict(POL, dense_count=5))
    assert out["sweeps"].tolist() == [5]


def test_empty_cache_falls_back_to_the_full_frame():
    out = P.build_rois([[], [det(5.0, 0.0)]], [ego(1.0), ego(1.0)], dict(POL))
    assert out["roi_offsets"].tolist() == [0, 1, 3]
    r = out["rois"][0]
    assert (r["cx"], r["cy"], r["ext_x"], r["ext_y"], r["cos_yaw"], r["sin_yaw"]) == (0.0, 0.0, 54.0, 54.0, 1.0, 0.0)
    assert out["budgets"][0] == 10
    out = P.build_rois([[]], [ego(1.0)], dict(POL, fallback_length=0.0))
    assert out["roi_offsets"].tolist() == [0, 0]


def _hom(theta, tx, ty):
    c, s = math.cos(theta), math.sin(theta)
    return np.array([[c, -s, tx], [s, c, ty], [0.0, 0.0, 1.0]])


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_records_cover_both_footprints_eq1(seed):
    """Points of the box at t-1 and of the box moved by v dt, taken to frame t by the ego motion, lie in one
    of the detection's two records; points beyond the margin of both boxes lie in neither."""
    d, off, e = synth.detections(seed, 3, count=(5, 12))
    dets, egos = as_dicts(d, off, e)
    out = P.build_rois(dets, egos, dict(POL, max_optional=1000))
    rng = np.random.default_rng(seed)
    for b, (frame, eg) in enumerate(zip(dets, egos)):
        M = _hom(eg["dyaw"], eg["dx"], eg["dy"])
        ranks = out["rank"][off[b]:off[b + 1]]
        base = out["roi_offsets"][b]
        for i, q in enumerate(frame):
            recs = out["rois"][base + 2 * ranks[i]: base + 2 * ranks[i] + 2]
            for shift in ((0.0, 0.0), (q["vx"] * POL["dt"], q["vy"] * POL["dt"])):
                box = _hom(q["yaw"], q["x"] + shift[0], q["y"] + shift[1])
                for _ in range(40):
                    u = rng.uniform(-0.49, 0.49, 2) * [q["length"], q["width"]]
                    p = M @ box @ np.array([u[0], u[1], 1.0])
                    assert any(oracle.inside(r, float(p[0]), float(p[1])) for r in recs)
            # a point beyond the margin of both footprints, along the box's own x axis
            far = 0.5 * q["length"] + POL["margin"] + 0.05 + abs(q["vx"]) * POL["dt"] + abs(q["vy"]) * POL["dt"]
            box = _hom(q["yaw"], q["x"], q["y"])
            for sgn in (-1, 1):
                p = M @ box @ np.array([sgn * (far + 0.5 * q["length"] + 1.0), 0.0, 1.0])
                q2 = M @ box @ np.array([0.0, sgn * (far + 0.5 * q["width"] + 1.0), 1.0])
                for pt in (p, q2):
                    moved = np.linalg.inv(M @ _hom(q["yaw"], q["x"] + q["vx"] * POL["dt"],
                                                   q["y"] + q["vy"] * POL["dt"])) @ pt
                    if abs(moved[0]) > 0.5 * q["length"] + POL["margin"] + 0.01 or \
                            abs(moved[1]) > 0.5 * q["width"] + POL["margin"] + 0.01:
                        assert not oracle.inside(recs[0], float(pt[0]), float(pt[1]))
                        assert not oracle.inside(recs[1], float(pt[0]), float(pt[1]))


@pytest.mark.parametrize("seed", [4, 5])
def test_invariants_on_random_caches(seed):
    d, off, e = synth.detections(seed, 6, count=(0, 200))
    dets, egos = as_dicts(d, off, e)
    pol = dict(POL, max_optional=40)
    out = P.build_rois(dets, egos, pol)
    for b, frame in enumerate(dets):
        lo, hi = off[b], off[b + 1]
        fl, rk, tt = out["flags"][lo:hi], out["rank"][lo:hi], out["ttc"][lo:hi]
        assert sorted(rk.tolist()) == list(range(hi - lo))
        mand = (fl & P.MANDATORY) != 0
        assert np.all(mand == (((fl & P.GEOM) != 0) | ((fl & P.SAFETY) != 0)))
        # mandatory ranked before optional; optional beyond max_optional dropped
        if mand.any() and (~mand).any():
            assert rk[mand].max() < rk[~mand].min()
        assert int(((fl & P.DROPPED) != 0).sum()) == max(0, int((~mand).sum()) - 40)
        # safety flags agree with the thresholds
        cls = np.array([q["cls"] for q in frame], dtype=np.int32)
        tau = np.where(cls == 0, 1.5, 2.5)
        assert np.all(((fl & P.SAFETY) != 0) == ((cls != 2) & (tt <= tau)))
        # budgets: record pairs in rank order
        bud = out["budgets"][out["roi_offsets"][b]:out["roi_offsets"][b + 1]]
        if hi > lo:
            order = np.argsort(rk)
            exp = np.where(mand[order], 10, np.where((fl[order] & P.DROPPED) != 0, 0, out["sweeps"][b]))
            assert bud.tolist() == np.repeat(exp, 2).tolist()
