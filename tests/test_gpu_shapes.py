"""Parity with the oracle at shapes the ABI accepts that select other code
paths of the HIP library:

* record widths: C = 3 (one 16-byte record word), C = 6 and 7 (two), C = 8
  (a third word), on small scenes and on the 347,200-point frame;
* frames with more ROIs than the filter stages in LDS (300, 700 and 1024),
  and more sweeps than it stages (S = 80 and S = 255, budgets spanning
  them): the filter's instance that reads its tables from global memory;
* keys of the full 32 bits (a grid of exactly 2^32 voxels: four radix
  passes of 8 bits);
* strided rows (point-by-point loads) together with an out-of-ROI keep rate;
* the limits up to which the point filter builds its frames' tables itself
  with several ROI words per cell (frames per call, cell words per frame).

The steps are those of Alg. 1 (keep loop, Voxelize, feature encoder) and
Eq. 6/7; structure bit for bit, features within 1e-5.
"""
import numpy as np
import pytest

import synth
from common import assert_same_voxels, case_from_workload
from test_gpu_parity import FEAT_TOL, check

pytestmark = pytest.mark.gpu


def _with_features(wl, C, seed):
    """The workload's points with C features: x, y, z, then seeded values
    (every passthrough column distinct, so a misplaced record word shows)."""
    N = wl.num_points
    rng = np.random.default_rng(seed)
    extra = rng.uniform(-100.0, 100.0, (max(C - 3, 0), N)).astype(np.float32)
    feat = np.ascontiguousarray(np.concatenate([wl.feat[:3], extra], 0))
    case = case_from_workload(wl)
    case.feat = feat
    return case


@pytest.mark.parametrize("C", [3, 6, 7, 8])
def test_feature_counts_small(gpu_lib, C):
    wl = synth.small(90 + C, frames=3, max_points=5, max_voxels=300)
    check(gpu_lib, _with_features(wl, C, C), label=f"small C={C}", desc=wl.roi_desc)


@pytest.mark.parametrize("C", [3, 8])
def test_feature_counts_full_frame(gpu_lib, C):
    wl = synth.c2()
    print(f"[shapes] c2 with C={C}", flush=True)
    check(gpu_lib, _with_features(wl, C, 100 + C), label=f"c2 C={C}", desc=wl.roi_desc)


def _random_rois(rng, n, extent):
    """Descriptor rows (cx, cy, length, width, yaw, margin)."""
    return np.column_stack([rng.uniform(-extent, extent, n), rng.uniform(-extent, extent, n),
                            rng.uniform(1.0, 6.0, n), rng.uniform(0.8, 3.0, n), rng.uniform(0, 2 * np.pi, n),
                            np.full(n, 0.3)])


@pytest.mark.parametrize("nroi", [300, 700, 1024])
def test_many_rois_per_frame(gpu_lib, nroi):
    """More ROIs per frame than the filter stages in LDS (256)."""
    import oracle

    wl = synth.small(120 + nroi % 97, frames=2, beams=8, azimuths=96, sweeps=4)
    rng = np.random.default_rng(nroi)
    B = wl.num_frames
    counts = [nroi, nroi // 3]
    desc = _random_rois(rng, sum(counts), 16.0)
    case = case_from_workload(wl, rois=oracle.make_rois(desc))
    case.roi_offsets = np.array([0, counts[0], counts[0] + counts[1]], dtype=np.int32)
    case.budgets = rng.integers(0, 5, sum(counts)).astype(np.uint8)
    assert B == 2
    vz, exp = check(gpu_lib, case, label=f"{nroi} rois", desc=desc)
    assert int(exp["voxel_offsets"][-1]) > 0


def test_many_rois_on_the_full_frame(gpu_lib):
    """The 347,200-point frame with 1,024 ROIs over the whole grid."""
    import oracle

    wl = synth.c2()
    rng = np.random.default_rng(5)
    desc = _random_rois(rng, 1024, 54.0)
    case = case_from_workload(wl, rois=oracle.make_rois(desc))
    case.roi_offsets = np.array([0, 1024], dtype=np.int32)
    case.budgets = rng.integers(1, 11, 1024).astype(np.uint8)
    print("[shapes] c2 with 1024 ROIs", flush=True)
    check(gpu_lib, case, label="c2 1024 rois", desc=desc)


@pytest.mark.parametrize("frames,nroi", [(16, 128), (17, 128), (16, 129)])
def test_frame_tables_built_by_the_filter_at_their_limits(gpu_lib, frames, nroi):
    """A 1440 x 1440 grid (45 x 45 coarse cells) with several ROI words per
    cell: at 16 frames and 128 ROIs (four words, 8,100 cell words) the point
    filter builds every frame's tables in LDS itself; one frame more, or one
    ROI word more (10,125 cell words), and the staging kernel builds them."""
    import oracle

    wl = synth.small(170 + frames + nroi, frames=frames, beams=6, azimuths=48, sweeps=3, dims=(1440, 1440, 16),
                     max_voxels=600, max_points=5)
    rng = np.random.default_rng(frames * 1000 + nroi)
    counts = [nroi] + list(rng.integers(0, nroi + 1, frames - 1))
    desc = _random_rois(rng, sum(counts), 13.0)
    case = case_from_workload(wl, rois=oracle.make_rois(desc))
    case.roi_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    case.budgets = rng.integers(1, 4, sum(counts)).astype(np.uint8)
    vz, exp = check(gpu_lib, case, label=f"{frames} frames x {nroi} rois", desc=desc)
    assert int(exp["voxel_offsets"][-1]) > 0


@pytest.mark.parametrize("S", [80, 255])
def test_many_sweeps(gpu_lib, S):
    """More sweeps than the filter stages in LDS (64), budgets from 1 to S."""
    wl = synth.small(140 + S, frames=2, beams=2, azimuths=24, sweeps=S, rois=8, budget=(1, S), max_voxels=2000)
    case = case_from_workload(wl)
    vz, exp = check(gpu_lib, case, label=f"S={S}", desc=wl.roi_desc)
    assert int(exp["voxel_offsets"][-1]) > 0


def test_full_32_bit_keys(gpu_lib):
    """A grid of exactly 2^32 voxels (65536 x 65536 x 1): keys use all 32 bits."""
    wl = synth.small(150, frames=2, beams=8, azimuths=64, sweeps=2, dims=(65536, 65536, 1), voxel=0.0005,
                     max_voxels=5000)
    case = case_from_workload(wl)
    # the grid is 32.768 m wide around the ego: move it so that it covers the points
    case.grid = dict(case.grid, range_min=[-16.384, -16.384, -4.0], voxel_size=[0.0005, 0.0005, 8.0])
    vz, exp = check(gpu_lib, case, label="2^32 keys", desc=wl.roi_desc)
    V = int(exp["voxel_offsets"][-1])
    assert V > 0 and int(exp["coords"][:V, 3].max()) > 32768 and int(exp["coords"][:V, 2].max()) > 32768


@pytest.mark.parametrize("rho", [0.3, 1.0])
@pytest.mark.parametrize("rois", [6, 40])
def test_strided_rows_with_background(gpu_lib, rho, rois):
    """A row stride that forbids 16-byte loads (point-by-point loads) with a
    nonzero out-of-ROI keep rate, with one ROI word per cell (6 ROIs) and
    with two (40 ROIs, whose cell words the filter keeps in LDS)."""
    import torch

    wl = synth.small(160, frames=3, beams=7, azimuths=61, sweeps=3, rois=rois)
    case = case_from_workload(wl)
    N = case.feat.shape[1]
    wide = np.zeros((case.feat.shape[0], N + 1), dtype=np.float32)
    wide[:, :N] = case.feat
    g = case.grid
    grid = gpu_lib.grid_params(g["range_min"], g["voxel_size"], g["dims"], g["max_points"], g["max_voxels"],
                               g["num_sweeps"], g["num_frames"])
    vz = gpu_lib.Voxelizer(case.feat, case.frame_offsets, case.sweep_ids, case.poses, gpu_lib.make_rois(wl.roi_desc),
                           case.roi_offsets, case.budgets, grid, int(np.max(np.diff(case.roi_offsets))), "cuda:0",
                           rho_out=rho, seed=31)
    vz.feat = torch.as_tensor(wide).cuda()[:, :N]
    vz.run()
    exp = case.run_oracle(rho, 31)
    assert vz.fault() == 0
    assert_same_voxels(vz.result(), exp, feat_atol=FEAT_TOL, label=f"stride rho={rho}")
