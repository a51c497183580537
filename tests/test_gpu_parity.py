"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Structure (voxel coordinates, order, counts, kept point indices, frame
offsets) must match bit for bit; mean features within 1e-5 absolute, the
stated tolerance for the fp32 means (both sides sum the same fp32 values in
double in the same order, so in practice they agree exactly).
"""
import numpy as np
import pytest

import synth
from common import Case, assert_same_voxels, case_from_workload, load_golden, records

pytestmark = pytest.mark.gpu
FEAT_TOL = 1e-5


def run_gpu(mb, case: Case, device="cuda:0", gpu_rois=None, rho_out=0.0, seed=0):
    """Run the HIP path; ROI records are the case's own (hand-made) or gpu_rois
    (built by the library's mmbev_make_rois from the same descriptors).
    rho_out, seed: the out-of-ROI keep rate and its seed."""
    g = case.grid
    grid = mb.grid_params(g["range_min"], g["voxel_size"], g["dims"], g["max_points"], g["max_voxels"],
                          g["num_sweeps"], g["num_frames"])
    mr = int(np.max(np.diff(case.roi_offsets))) if len(case.roi_offsets) > 1 else 0
    rois = case.rois if gpu_rois is None else gpu_rois
    vz = mb.Voxelizer(case.feat, case.frame_offsets, case.sweep_ids, case.poses, rois, case.roi_offsets,
                      case.budgets, grid, max(mr, 1), device, rho_out, seed)
    vz.run()
    return vz


def check(mb, case: Case, label="", desc=None, rho_out=0.0, seed=0):
    """Oracle vs GPU.  With `desc` (ROI descriptors) each side builds its own records."""
    exp = case.run_oracle(rho_out, seed)
    vz = run_gpu(mb, case, gpu_rois=None if desc is None else mb.make_rois(desc), rho_out=rho_out, seed=seed)
    got = vz.result()
    assert vz.fault() == 0, f"{label}: device fault {vz.fault()}"
    assert_same_voxels(got, exp, feat_atol=FEAT_TOL, label=label)
    # rows past V untouched in every output (canary -7 written at allocation)
    V = int(exp["voxel_offsets"][-1])
    for name in ("out_coords", "out_counts", "out_feats", "out_point_idx"):
        rest = getattr(vz, name)[V:]
        assert bool((rest == -7).all().item()), f"{label}: {name} rows past V were written"
    return vz, exp


def test_golden_hand_two_frames(gpu_lib):
    case, exp = load_golden("hand_two_frames.json")
    vz = run_gpu(gpu_lib, case)
    assert vz.fault() == 0
    assert_same_voxels(vz.result(), exp, feat_atol=0.0, label="golden")


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_configs_match_oracle(gpu_lib, name):
    wl = synth.CONFIGS[name]()
    case = case_from_workload(wl)
    vz, exp = check(gpu_lib, case, label=name, desc=wl.roi_desc)
    h = vz.header()
    keys, _ = case.oracle_keep()
    assert h["kept"] == len(keys), "kept-point count differs from the oracle's"


@pytest.mark.parametrize("seed,frames,cap,M,budget", [
    (1, 1, 1000, 4, (1, 3)), (2, 2, 25, 2, (1, 3)), (3, 3, 7, 1, (0, 3)), (4, 4, 1, 3, (1, 3)),
    (5, 5, 50, 8, (2, 3)), (6, 2, 3, 64, (1, 3)), (7, 7, 400, 5, (1, 2))])
def test_small_scenes_match_oracle(gpu_lib, seed, frames, cap, M, budget):
    wl = synth.small(seed, frames=frames, max_voxels=cap, max_points=M, budget=budget)
    check(gpu_lib, case_from_workload(wl), label=f"small{seed}", desc=wl.roi_desc)


def test_ragged_tail_and_scalar_loads(gpu_lib):
    """N not a multiple of 4 and a row stride that forbids 16-byte loads."""
    wl = synth.small(21, frames=1, beams=7, azimuths=61, sweeps=3)
    case = case_from_workload(wl)
    N = case.feat.shape[1]
    assert N % 4 != 0
    check(gpu_lib, case, label="ragged", desc=wl.roi_desc)
    # stride N+1 (scalar path): embed the SoA rows in a wider array
    import torch
    wide = np.zeros((case.feat.shape[0], N + 1), dtype=np.float32)
    wide[:, :N] = case.feat
    g = case.grid
    grid = gpu_lib.grid_params(g["range_min"], g["voxel_size"], g["dims"], g["max_points"], g["max_voxels"],
                               g["num_sweeps"], g["num_frames"])
    vz = gpu_lib.Voxelizer(case.feat, case.frame_offsets, case.sweep_ids, case.poses, gpu_lib.make_rois(wl.roi_desc),
                           case.roi_offsets, case.budgets, grid, int(np.max(np.diff(case.roi_offsets))), "cuda:0")
    vz.feat = torch.as_tensor(wide).cuda()[:, :N]
    vz.run()
    assert_same_voxels(vz.result(), case.run_oracle(), feat_atol=FEAT_TOL, label="stride")


def test_wide_keys_need_frame_lookup(gpu_lib):
    """A 2048 x 2048 x 64 grid (28 key bits, four radix passes) over 33
    frames: each frame is sorted inside its own range of the pair arrays, so
    the keys carry no frame bits however many frames there are."""
    wl = synth.small(31, frames=33, beams=4, azimuths=32, sweeps=2, dims=(2048, 2048, 64), voxel=0.02,
                     max_voxels=60)
    case = case_from_workload(wl)
    check(gpu_lib, case, label="wide", desc=wl.roi_desc)


def test_edge_cases(gpu_lib):
    case, _ = load_golden("hand_two_frames.json")
    # every budget 0: nothing kept
    check(gpu_lib, Case(**{**case.__dict__, "budgets": np.zeros_like(case.budgets)}), label="budget0")
    # one frame with no ROI
    check(gpu_lib, Case(**{**case.__dict__, "rois": case.rois[:2], "budgets": case.budgets[:2],
                           "roi_offsets": np.array([0, 2, 2], dtype=np.int32)}), label="no-roi frame")
    # sweep ids past num_sweeps
    check(gpu_lib, Case(**{**case.__dict__, "sweep_ids": np.full_like(case.sweep_ids, 9)}), label="sweep>=S")
    # non-finite coordinates
    feat = case.feat.copy()
    feat[0, 0], feat[1, 5], feat[2, 12] = np.nan, np.inf, -np.inf
    check(gpu_lib, Case(**{**case.__dict__, "feat": feat}), label="nonfinite")
    # a single point, and an empty frame in the middle
    one = Case(feat=case.feat[:, :1].copy(), sweep_ids=case.sweep_ids[:1], frame_offsets=np.array([0, 1]),
               poses=case.poses[:1], rois=case.rois[:2], roi_offsets=np.array([0, 2], dtype=np.int32),
               budgets=case.budgets[:2], grid=dict(case.grid, num_frames=1))
    check(gpu_lib, one, label="one point")
    wl = synth.small(41, frames=3)
    c3 = case_from_workload(wl)
    fo = c3.frame_offsets.copy()
    keep = np.r_[0:fo[1], fo[2]:fo[3]]
    empty_mid = Case(feat=np.ascontiguousarray(c3.feat[:, keep]), sweep_ids=c3.sweep_ids[keep],
                     frame_offsets=np.array([0, fo[1], fo[1], fo[1] + fo[3] - fo[2]]), poses=c3.poses, rois=c3.rois,
                     roi_offsets=c3.roi_offsets, budgets=c3.budgets, grid=c3.grid)
    check(gpu_lib, empty_mid, label="empty middle frame", desc=wl.roi_desc)


@pytest.mark.parametrize("frames", [255, 256, 2047, 2100, 4100])
def test_many_small_frames(gpu_lib, frames):
    """Frame counts on both sides of the point filter's own layout of the
    call (up to 255 frames of at most 32 ROIs, one frame per thread; beyond,
    the staging kernel lays it out), of the stage's LDS copy of the chunk
    starts (up to 2,047 frames; beyond, each frame's thread writes its filter
    workgroups' frame itself) and of the segments' per-frame tables in LDS
    (up to 4,096 frames; beyond, in the workspace), with every seventh frame
    emptied."""
    wl = synth.small(51, frames=frames, beams=2, azimuths=16, sweeps=1, rois=4)
    c = case_from_workload(wl)
    fo = c.frame_offsets
    keep = np.concatenate([np.arange(fo[f], fo[f + 1]) for f in range(frames) if f % 7 != 3])
    counts = np.array([0 if f % 7 == 3 else fo[f + 1] - fo[f] for f in range(frames)])
    sparse = Case(feat=np.ascontiguousarray(c.feat[:, keep]), sweep_ids=c.sweep_ids[keep],
                  frame_offsets=np.concatenate([[0], np.cumsum(counts)]), poses=c.poses, rois=c.rois,
                  roi_offsets=c.roi_offsets, budgets=c.budgets, grid=c.grid)
    check(gpu_lib, sparse, label=f"{frames} frames", desc=wl.roi_desc)


def test_zero_points(gpu_lib):
    case, _ = load_golden("hand_two_frames.json")
    z = Case(feat=np.zeros((4, 0), np.float32), sweep_ids=np.zeros(0, np.uint8), frame_offsets=np.array([0, 0, 0]),
             poses=case.poses, rois=case.rois, roi_offsets=case.roi_offsets, budgets=case.budgets, grid=case.grid)
    vz = run_gpu(gpu_lib, z)
    assert vz.result()["voxel_offsets"].tolist() == [0, 0, 0]
    assert vz.fault() == 0


def test_repeat_calls_are_bit_identical_and_workspace_reusable(gpu_lib):
    import torch

    wl = synth.c2()
    vz = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
    vz.run()
    a = vz.result()
    for _ in range(3):
        vz.run()
    torch.cuda.synchronize()
    b = vz.result()
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert vz.header()["epoch"] == 4


def test_device_fault_word_reports_bad_offsets(gpu_lib):
    import torch

    case, _ = load_golden("hand_two_frames.json")
    vz = run_gpu(gpu_lib, case)
    vz.frame_offsets = torch.tensor([0, 12, 18], dtype=torch.int64, device="cuda:0")  # off[B] != N
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() & gpu_lib.FAULT_POINT_OFFSETS
    vz.frame_offsets = torch.tensor([0, 12, 19], dtype=torch.int64, device="cuda:0")
    vz.roi_frame_offsets = torch.tensor([0, 3, 4], dtype=torch.int32, device="cuda:0")  # 3 > max_rois_per_frame
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() & gpu_lib.FAULT_ROI_OFFSETS


@pytest.mark.parametrize("frames", [200, 300])
def test_fault_word_reports_offsets_of_late_frames(gpu_lib, frames):
    """Offsets that break the contract only in frame 150 of 200 (the point
    filter lays out the call) or of 300 (the staging kernel does): waves past
    the first check them, after the fault word is cleared.  Decreasing point
    offsets make the call keep nothing (frames would overlap); every kernel
    still runs to its end."""
    import torch

    wl = synth.small(81, frames=frames, beams=2, azimuths=16, sweeps=1, rois=4)
    vz = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() == 0 and int(vz.result()["voxel_offsets"][-1]) > 0
    fo = wl.frame_offsets.copy()
    fo[150] = fo[151] + 5  # off[150] > off[151]
    vz.frame_offsets = torch.as_tensor(fo).cuda()
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() == gpu_lib.FAULT_POINT_OFFSETS
    assert vz.result()["voxel_offsets"].tolist() == [0] * (frames + 1)
    vz.frame_offsets = torch.as_tensor(wl.frame_offsets).cuda()
    ro = wl.roi_offsets.copy()
    ro[150] = ro[151] + 1  # decreasing ROI offsets
    vz.roi_frame_offsets = torch.as_tensor(ro).cuda()
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() == gpu_lib.FAULT_ROI_OFFSETS
    vz.roi_frame_offsets = torch.as_tensor(wl.roi_offsets).cuda()
    vz.run()
    torch.cuda.synchronize()
    assert vz.fault() == 0


def test_throughput_batch_full_size(gpu_lib):
    """The benchmark's batched workload, every frame checked against the oracle."""
    wl = synth.throughput(16)
    check(gpu_lib, case_from_workload(wl), label="c2x16", desc=wl.roi_desc)


def test_throughput_batch_128_frames_two_tile_chunks(gpu_lib):
    """The benchmark's own 128-frame call (2.75M kept pairs): one-tile pair
    chunks would overflow one round of the scatter's resident workgroups, so
    the chunks take at least two tiles; every output checked against the
    oracle."""
    wl = synth.throughput(128)
    vz, exp = check(gpu_lib, case_from_workload(wl), label="c2x128", desc=wl.roi_desc)
    h = vz.header()
    K = int(h["kept"])
    assert K > 2048 * (1024 - 128), K  # one-tile chunks would not fit one round of 1,024 workgroups
    assert 0 < h["pair_chunks"] <= 1024, h
    assert K / h["pair_chunks"] > 2048, (K, h["pair_chunks"])  # chunks longer than one 2,048-pair tile


def test_capped_frame_tables_in_workspace(gpu_lib):
    """A frame over max_voxels whose first-place bitmap does not fit LDS (more
    than 16,384 words: over 524,288 kept pairs), so the cap keeps its tables
    in the workspace: 700,000 points spread over a 256 x 256 x 16 grid, one ROI
    over all of it, about 490,000 voxels capped to 150,000."""
    rng = np.random.default_rng(77)
    N = 700_000
    mn, voxel, dims = (-25.6, -25.6, -2.0), (0.2, 0.2, 0.25), (256, 256, 16)
    cols = [rng.uniform(mn[d], mn[d] + dims[d] * voxel[d], N) for d in range(3)]
    feat = np.ascontiguousarray(np.stack(cols + [rng.random(N)]).astype(np.float32))
    poses = np.array([1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 1, 0], np.float32).reshape(1, 1, 12)
    grid = dict(range_min=list(mn), voxel_size=list(voxel), dims=list(dims), max_points=4, max_voxels=150_000,
                num_sweeps=1, num_frames=1)
    case = Case(feat=feat, sweep_ids=np.zeros(N, np.uint8), frame_offsets=np.array([0, N]), poses=poses,
                rois=records([[0.0, 0.0, 1.0, 0.0, 100.0, 100.0]]), roi_offsets=np.array([0, 1], np.int32),
                budgets=np.array([1], np.uint8), grid=grid)
    vz, exp = check(gpu_lib, case, label="cap-workspace")
    assert int(exp["voxel_offsets"][-1]) == 150_000
    h = vz.header()
    assert h["kept"] > 524_288 and h["capped_voxels"] > 150_000, h


def test_capped_frame_too_large_to_share(gpu_lib):
    """A frame over max_voxels with more kept pairs than a shared cap takes
    (48 steps of 32,768 slots): one workgroup caps it alone, its tables in the
    workspace.  1,700,000 points over a 512 x 512 x 16 grid, one ROI over all
    of it, capped to 200,000 voxels."""
    rng = np.random.default_rng(78)
    N = 1_700_000
    mn, voxel, dims = (-51.2, -51.2, -2.0), (0.2, 0.2, 0.25), (512, 512, 16)
    cols = [rng.uniform(mn[d], mn[d] + dims[d] * voxel[d], N) for d in range(3)]
    feat = np.ascontiguousarray(np.stack(cols + [rng.random(N)]).astype(np.float32))
    poses = np.array([1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 1, 0], np.float32).reshape(1, 1, 12)
    grid = dict(range_min=list(mn), voxel_size=list(voxel), dims=list(dims), max_points=2, max_voxels=200_000,
                num_sweeps=1, num_frames=1)
    case = Case(feat=feat, sweep_ids=np.zeros(N, np.uint8), frame_offsets=np.array([0, N]), poses=poses,
                rois=records([[0.0, 0.0, 1.0, 0.0, 200.0, 200.0]]), roi_offsets=np.array([0, 1], np.int32),
                budgets=np.array([1], np.uint8), grid=grid)
    vz, exp = check(gpu_lib, case, label="cap-unshared")
    assert int(exp["voxel_offsets"][-1]) == 200_000
    h = vz.header()
    assert h["kept"] > 48 * 32_768 and h["capped_voxels"] > 200_000, h


def test_capped_frame_beside_larger_uncapped_frame(gpu_lib):
    """The frame with the most pairs is not over max_voxels (200,000 points in
    a 32 x 32 x 8 block of voxels) while the next frame is (100,000 points
    spread over a 256 x 256 x 16 grid, about 95,000 voxels capped to 40,000):
    the capped frame is capped by its own workgroup and numbered by whole-frame
    prefixes, beside a frame whose cap would have been shared."""
    rng = np.random.default_rng(79)
    mn, voxel, dims = (-25.6, -25.6, -2.0), (0.2, 0.2, 0.25), (256, 256, 16)
    n0, n1 = 200_000, 100_000
    dense = [rng.uniform(0.0, 32 * voxel[d] if d < 2 else 8 * voxel[d], n0) + (0.0 if d < 2 else mn[2]) for d in range(3)]
    spread = [rng.uniform(mn[d], mn[d] + dims[d] * voxel[d], n1) for d in range(3)]
    cols = [np.concatenate([dense[d], spread[d]]) for d in range(3)]
    N = n0 + n1
    feat = np.ascontiguousarray(np.stack(cols + [rng.random(N)]).astype(np.float32))
    poses = np.tile(np.array([1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 1, 0], np.float32), (2, 1)).reshape(2, 1, 12)
    grid = dict(range_min=list(mn), voxel_size=list(voxel), dims=list(dims), max_points=3, max_voxels=40_000,
                num_sweeps=1, num_frames=2)
    case = Case(feat=feat, sweep_ids=np.zeros(N, np.uint8), frame_offsets=np.array([0, n0, N]), poses=poses,
                rois=records([[0.0, 0.0, 1.0, 0.0, 100.0, 100.0]] * 2), roi_offsets=np.array([0, 1, 2], np.int32),
                budgets=np.array([1, 1], np.uint8), grid=grid)
    vz, exp = check(gpu_lib, case, label="cap-beside-larger")
    off = exp["voxel_offsets"]
    assert int(off[1]) < 40_000 and int(off[2] - off[1]) == 40_000, off
    h = vz.header()
    assert h["capped_voxels"] > 40_000 and h["most_frame"] == 0 and h["most_pairs"] == n0, h


def _face_lattice_case(pose_rows, voxel=(0.1, 0.15, 0.3), mn=(-3.7, -2.9, -1.3), dims=(60, 40, 10)):
    """Points on voxel faces (and one ulp either side) of a non-dyadic grid,
    all inside one ROI covering the grid: the voxel index of every point is
    decided by the rounding of (p - min) / v, and every tile queues far more
    candidates than one segment holds."""
    f32 = np.float32
    faces = []
    for d in range(3):
        k = np.arange(-1, dims[d] + 2, dtype=np.float64)
        base = (f32(mn[d]) + k * f32(voxel[d])).astype(f32)
        faces.append(np.unique(np.concatenate([base, np.nextafter(base, f32(np.inf)),
                                               np.nextafter(base, f32(-np.inf))])))
    zc = (f32(mn[2]) + (np.arange(dims[2]) + f32(0.5)) * f32(voxel[2])).astype(f32)
    X, Y = np.meshgrid(faces[0], faces[1], indexing="ij")
    xy = np.stack([X.ravel(), Y.ravel()], 0)
    z = np.resize(np.concatenate([zc, faces[2]]), xy.shape[1]).astype(f32)
    feat = np.ascontiguousarray(np.concatenate([xy, z[None], np.ones((1, xy.shape[1]), f32)], 0).astype(f32))
    N = feat.shape[1]
    cx = mn[0] + voxel[0] * dims[0] / 2
    cy = mn[1] + voxel[1] * dims[1] / 2
    rois = records([[cx, cy, 1.0, 0.0, 50.0, 50.0]])
    poses = np.asarray(pose_rows, np.float32).reshape(1, 1, 12)
    grid = dict(range_min=list(mn), voxel_size=list(voxel), dims=list(dims), max_points=3, max_voxels=100000,
                num_sweeps=1, num_frames=1)
    return Case(feat=feat, sweep_ids=np.zeros(N, np.uint8), frame_offsets=np.array([0, N]), poses=poses, rois=rois,
                roi_offsets=np.array([0, 1], np.int32), budgets=np.array([1], np.uint8), grid=grid)


def test_points_on_voxel_faces_and_full_queues(gpu_lib):
    ident = [1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 1, 0]
    case = _face_lattice_case(ident)
    assert case.feat.shape[1] > 8 * 1024
    _, exp = check(gpu_lib, case, label="faces")
    assert int(exp["voxel_offsets"][-1]) > 1000
    # a translation by a non-dyadic offset moves the faces off the lattice
    shifted = _face_lattice_case([1, 0, 0, 0.05, 0, 1, 0, -0.075, 0, 0, 1, 0.15])
    check(gpu_lib, shifted, label="faces shifted")
