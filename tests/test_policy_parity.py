"""Parity of the library's temporal-ROI selector (mmbev_build_rois, host
code behind the C ABI) with the oracle: ROI records bit for bit, budgets,
offsets, TTC (exact, infinity included), flags, ranks and sweep counts."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import synth
from oracle import policy as P
from test_oracle_policy import POL, as_dicts


@pytest.fixture(scope="module")
def mb():
    from paper_2608_15437_amd import mmbev

    mmbev.load()
    return mmbev


def _both(mb, d, off, e, pol):
    got = mb.build_rois(d, off, e, mb.policy(**pol))
    exp = P.build_rois(*as_dicts(d, off, e), pol)
    return got, exp


def _same(got, exp):
    assert got["roi_offsets"].tolist() == exp["roi_offsets"].tolist()
    assert np.array_equal(got["rois"].view(np.uint32).reshape(-1, 8), exp["rois"].view(np.uint32).reshape(-1, 8))
    assert np.array_equal(got["budgets"], exp["budgets"])
    assert np.array_equal(got["crit"]["ttc"], exp["ttc"])
    assert np.array_equal(got["crit"]["flags"], exp["flags"])
    assert np.array_equal(got["crit"]["rank"], exp["rank"])
    assert np.array_equal(got["sweeps"], exp["sweeps"])


@pytest.mark.parametrize("seed,frames,count,kw", [
    (1, 4, (0, 300), {}),
    (2, 8, (0, 40), {"max_optional": 5}),
    (3, 3, (100, 400), {"dense_count": 200}),
    (4, 16, (0, 12), {"dt": 0.1, "margin": 0.3, "r_coll": 3.5}),
    (5, 2, [0, 0], {}),
    (6, 2, [0, 7], {"fallback_length": 0.0}),
    (7, 5, (0, 60), {"theta_max_deg": 45.0, "theta_min_deg": 45.0, "speed_wide": 10.0, "speed_narrow": 10.0}),
])
def test_random_caches_match_oracle(mb, seed, frames, count, kw):
    d, off, e = synth.detections(seed, frames, count=count)
    _same(*_both(mb, d, off, e, dict(POL, **kw)))


def test_ties_and_exact_boundaries(mb):
    """Equal TTC and distance (order by input), objects on the cone edge and at the braking distance."""
    d = np.zeros(6, dtype=synth.DETECTION_DTYPE)
    d["length"], d["width"], d["cls"] = 4.0, 2.0, 1
    d["x"] = [10.0, 10.0, 18.75, 30.0, 30.0, 0.0]
    d["y"] = [0.0, 0.0, 0.0, 0.0, 0.0, 3.0]
    e = np.zeros(1, dtype=synth.EGO_DTYPE)
    e["speed"] = 15.0
    _same(*_both(mb, d, np.array([0, 6], np.int32), e, dict(POL)))


def test_rejects_bad_arguments(mb):
    d, off, e = synth.detections(9, 2, count=(3, 5))
    L = mb.load()
    for bad in ({"dt": 0.0}, {"r_coll": -1.0}, {"a_brake": 0.0}, {"theta_max_deg": 91.0},
                {"theta_min_deg": 70.0}, {"speed_wide": 40.0}, {"n_full": 256}, {"n_reduced": 11},
                {"n_reduced": 0}, {"max_optional": -1}, {"margin": float("nan")}):
        with pytest.raises(mb.MmbevError):
            mb.build_rois(d, off, e, mb.policy(**dict(POL, **bad)))
    bad_cls = d.copy()
    bad_cls["cls"][0] = 3
    bad_res = d.copy()
    bad_res["reserved"][1] = 1
    bad_nan = d.copy()
    bad_nan["vx"][2] = np.inf
    for dd in (bad_cls, bad_res, bad_nan):
        with pytest.raises(mb.MmbevError):
            mb.build_rois(dd, off, e, mb.policy(**POL))
    for oo in (np.array([1, off[1], off[2]], np.int32), np.array([0, off[2], off[1]], np.int32)):
        with pytest.raises(mb.MmbevError):
            mb.build_rois(d, oo, e, mb.policy(**POL))
    assert L.mmbev_build_rois(None, off.ctypes.data, 2, e.ctypes.data, ctypes.byref(mb.policy(**POL)), None, None,
                              None, None, None) == mb.ERR_INVALID_ARG
