"""Pins of the oracle's out-of-ROI keep rate (Alg. 1: points outside every
ROI are kept with probability rho_out).

The draw is SplitMix64 (Steele, Lea and Flood, OOPSLA 2014; Vigna's
public-domain reference code): point i is kept when the top 24 bits of the
generator's (i + 1)-th output, state seeded with `seed`, lie below
round(rho_out * 2^24).  The generator is pinned to its published outputs;
the rest to closed forms (rate 0 and 1), a binomial bound, and the
counter-based property (a point's draw depends on nothing but the seed and
its index).
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import synth
from common import case_from_workload, records

MASK64 = (1 << 64) - 1


def splitmix64_py(seed: int, n: int) -> int:
    """The same generator in Python's unbounded integers, reduced mod 2^64."""
    z = (seed + n * 0x9E3779B97F4A7C15) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def test_splitmix64_published_outputs():
    # the first three outputs of the reference generator with state 0
    expected = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [oracle.splitmix64(0, n) for n in (1, 2, 3)] == expected
    assert [splitmix64_py(0, n) for n in (1, 2, 3)] == expected


def test_splitmix64_wraps_like_unbounded_integers():
    rng = np.random.default_rng(5)
    for _ in range(200):
        seed = int(rng.integers(0, 2 ** 63)) * 2 + int(rng.integers(0, 2))
        n = int(rng.integers(1, 2 ** 40))
        assert oracle.splitmix64(seed, n) == splitmix64_py(seed, n)


def test_background_threshold():
    assert oracle.background_threshold(0.0) == 0
    assert oracle.background_threshold(-0.5) == 0
    assert oracle.background_threshold(float("nan")) == 0
    assert oracle.background_threshold(1.0) == 1 << 24
    assert oracle.background_threshold(7.0) == 1 << 24
    assert oracle.background_threshold(0.5) == 1 << 23
    assert oracle.background_threshold(0.25) == 1 << 22
    # round to nearest: the fp32 value of 0.1 times 2^24
    assert oracle.background_threshold(0.1) == round(float(np.float32(0.1)) * 2 ** 24)


def _keep(case, rho, seed, rois=None, budgets=None):
    return oracle.keep(case.feat, case.frame_offsets, case.sweep_ids, case.poses,
                       case.rois if rois is None else rois, case.roi_offsets,
                       case.budgets if budgets is None else budgets, case.ogrid(), rho, seed)


def _all_covering(case):
    """One ROI per frame covering the whole grid, admitting every sweep."""
    B = case.B
    rois = records([[0, 0, 1, 0, 1e6, 1e6]] * B)
    return rois, np.arange(B + 1, dtype=np.int32), np.full(B, 255, dtype=np.uint8)


def test_rate_one_keeps_every_point_in_range():
    case = case_from_workload(synth.small(3, frames=2))
    rois, roff, bud = _all_covering(case)
    k1, i1 = _keep(case, 1.0, 9)
    case2 = case_from_workload(synth.small(3, frames=2), rois=rois)
    case2.roi_offsets, case2.budgets = roff, bud
    k2, i2 = case2.oracle_keep()
    assert np.array_equal(i1, i2) and np.array_equal(k1, k2)
    assert len(i1) > len(case.oracle_keep()[1])


def test_rate_zero_is_the_roi_only_path():
    case = case_from_workload(synth.small(4, frames=3))
    k0, i0 = _keep(case, 0.0, 1234)
    k, i = case.oracle_keep()
    assert np.array_equal(i0, i) and np.array_equal(k0, k)


def test_background_matches_independent_draw():
    case = case_from_workload(synth.small(6, frames=2))
    rho, seed = 0.37, 0xDEADBEEF12345678
    thr = oracle.background_threshold(rho)
    _, roi_idx = case.oracle_keep()
    _, all_idx = _keep(case, 1.0, seed)  # every point in range with a valid sweep
    expected = set(roi_idx.tolist())
    for i in all_idx.tolist():
        if (splitmix64_py(seed, i + 1) >> 40) < thr:
            expected.add(i)
    _, got = _keep(case, rho, seed)
    assert got.tolist() == sorted(expected)


def test_background_fraction_is_binomial():
    case = case_from_workload(synth.c2())
    rho, seed = 0.3, 77
    _, roi_idx = case.oracle_keep()
    _, all_idx = _keep(case, 1.0, seed)
    outside = np.setdiff1d(all_idx, roi_idx)
    _, got = _keep(case, rho, seed)
    bg = np.setdiff1d(got, roi_idx)
    assert np.all(np.isin(bg, outside))
    n = len(outside)
    p = oracle.background_threshold(rho) / 2 ** 24
    sigma = math.sqrt(n * p * (1 - p))
    assert n > 10000
    assert abs(len(bg) - n * p) < 6 * sigma


def test_draw_depends_only_on_seed_and_index():
    case = case_from_workload(synth.small(8, frames=2))
    rho = 0.5
    _, roi_idx = case.oracle_keep()
    _, with_rois = _keep(case, rho, 42)
    empty = np.zeros(0, dtype=oracle.ROI_DTYPE)
    _, no_rois = oracle.keep(case.feat, case.frame_offsets, case.sweep_ids, case.poses, empty,
                             np.zeros(case.B + 1, dtype=np.int32), np.zeros(0, dtype=np.uint8), case.ogrid(),
                             rho, 42)
    # outside the ROIs, a point's draw is the same whatever the ROIs are
    assert np.array_equal(np.setdiff1d(with_rois, roi_idx), np.setdiff1d(no_rois, roi_idx))
    _, other_seed = _keep(case, rho, 43)
    assert not np.array_equal(with_rois, other_seed)


@pytest.mark.parametrize("rho", [0.05, 0.5])
def test_background_voxels_cover_roi_voxels(rho):
    # keeping more points never removes a voxel or a point of a voxel below the cap
    wl = synth.small(2, frames=2, max_voxels=10 ** 6, max_points=64)
    case = case_from_workload(wl)
    a = case.run_oracle()
    b = oracle.roi_voxelize(case.feat, case.frame_offsets, case.sweep_ids, case.poses, case.rois,
                            case.roi_offsets, case.budgets, case.ogrid(), rho, 5)
    ka = {tuple(r) for r in a["coords"].tolist()}
    kb = {tuple(r) for r in b["coords"].tolist()}
    assert ka <= kb and len(kb) > len(ka)
