"""Parity of the connected-component proposer (mmbev_voxel_clusters, through
the C ABI) with the oracle's flood fill: clusters, frame offsets and voxel
labels bit for bit (every field is an integer)."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from common import case_from_workload
from test_gpu_parity import run_gpu
from test_oracle_clusters import _grid_voxels

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "clusters_hand.json")


def _gpu(mb, coords, counts, voff, dims, frames, cap, prm, proposer=None, check_rest=True):
    """Upload voxel rows padded to frames * cap rows and run the proposer; labels past
    voxel_offsets[B] must stay untouched (check_rest)."""
    import torch

    rows = frames * cap
    dc = torch.full((rows, 4), -9, dtype=torch.int32, device="cuda:0")
    dn = torch.full((rows,), 1000, dtype=torch.int32, device="cuda:0")
    V = len(coords)
    if V:
        dc[:V] = torch.from_numpy(np.ascontiguousarray(coords, dtype=np.int32)).cuda()
        dn[:V] = torch.from_numpy(np.ascontiguousarray(counts, dtype=np.int32)).cuda()
    dv = torch.from_numpy(np.asarray(voff, dtype=np.int64)).cuda()
    grid = mb.grid_params((0.0, 0.0, 0.0), (1.0, 1.0, 1.0), dims, 1, cap, 1, frames)
    p = proposer or mb.ClusterProposer(grid, prm, "cuda:0")
    p.run(dc, dn, dv)
    torch.cuda.synchronize()
    res = p.result(V)
    if check_rest:
        rest = p.labels[int(voff[-1]):].cpu().numpy()
        assert np.all(rest == -7), "labels past the voxel rows were written"
    return res, p


def _same(got, exp, label=""):
    assert got["cluster_offsets"].tolist() == exp["cluster_offsets"].tolist(), label
    g, e = got["clusters"], exp["clusters"]
    assert len(g) == len(e), label
    for f in ("frame", "root", "cells", "voxels", "points", "x0", "y0", "x1", "y1", "sum_x", "sum_y"):
        assert np.array_equal(g[f], e[f]), (label, f)
    assert np.array_equal(got["voxel_labels"], exp["voxel_labels"]), label


@pytest.mark.parametrize("k", range(4))
def test_golden_hand_fixture(gpu_lib, k):
    g = json.load(open(GOLDEN))
    c = g["cases"][k]
    prm = gpu_lib.cluster_params(c["z_min"], c["z_max"], c["cell_shift"], c["connectivity"], c["min_cells"])
    res, p = _gpu(gpu_lib, np.array(g["coords"]), np.array(g["counts"]), g["voxel_offsets"], g["dims"],
                  g["num_frames"], 10, prm)
    assert p.fault() == 0
    rows = [[int(x[f]) for f in ("frame", "root", "cells", "voxels", "points", "x0", "y0", "x1", "y1", "sum_x",
                                 "sum_y")] for x in res["clusters"]]
    assert rows == c["clusters"]
    assert res["cluster_offsets"].tolist() == c["cluster_offsets"]
    assert res["voxel_labels"].tolist() == c["voxel_labels"]


def _frames(seed, shapes, density, layers=3):
    rng = np.random.default_rng(seed)
    coords, voff = [], [0]
    Dy = max(s[0] for s in shapes)
    Dx = max(s[1] for s in shapes)
    for b, (h, w) in enumerate(shapes):
        occ = np.zeros((Dy, Dx), bool)
        occ[:h, :w] = rng.random((h, w)) < density
        c = _grid_voxels(occ, rng, layers)
        c[:, 0] = b
        coords.append(c)
        voff.append(voff[-1] + len(c))
    coords = np.concatenate(coords)
    counts = rng.integers(1, 11, size=len(coords)).astype(np.int32)
    return coords, counts, np.array(voff), (Dx, Dy, layers)


@pytest.mark.parametrize("conn", [4, 8])
@pytest.mark.parametrize("seed,shapes,density,shift,min_cells,band", [
    (1, [(40, 37)], 0.3, 0, 1, (0, 3)),
    (2, [(64, 64), (64, 64), (10, 3)], 0.55, 0, 2, (1, 3)),
    (3, [(9, 120), (120, 9)], 0.45, 1, 1, (0, 2)),
    (4, [(200, 300)], 0.5, 0, 1, (0, 3)),       # near the percolation threshold: large tangled components
    (5, [(257, 255), (1, 1)], 0.6, 2, 3, (0, 3)),
    (6, [(33, 1), (1, 50)], 0.5, 0, 1, (2, 3)),
])
def test_random_grids_match_oracle(gpu_lib, conn, seed, shapes, density, shift, min_cells, band):
    coords, counts, voff, dims = _frames(seed, shapes, density)
    B = len(shapes)
    cap = int(np.max(np.diff(voff))) + 3
    prm = gpu_lib.cluster_params(band[0], band[1], shift, conn, min_cells)
    res, p = _gpu(gpu_lib, coords, counts, voff, dims, B, cap, prm)
    assert p.fault() == 0
    exp = oracle.clusters(coords, counts, voff, dims, B, band[0], band[1], shift, conn, min_cells)
    _same(res, exp, f"seed{seed}")


def test_one_giant_component_and_a_serpentine(gpu_lib):
    """A fully occupied 1024 x 1024 frame (one cluster of 2^20 cells) and a serpentine path (long chains)."""
    full = np.ones((1024, 1024), bool)
    snake = np.zeros((301, 301), bool)
    snake[::2, :] = True
    snake[1::4, -1] = True
    snake[3::4, 0] = True
    rng = np.random.default_rng(0)
    parts = []
    for b, occ in enumerate([full, np.pad(snake, ((0, 1024 - 301), (0, 1024 - 301)))]):
        c = _grid_voxels(occ, rng, 1)
        c[:, 0] = b
        parts.append(c)
    coords = np.concatenate(parts)
    counts = np.ones(len(coords), np.int32)
    voff = np.array([0, len(parts[0]), len(coords)])
    for conn in (4, 8):
        prm = gpu_lib.cluster_params(0, 1, 0, conn, 1)
        res, p = _gpu(gpu_lib, coords, counts, voff, (1024, 1024, 1), 2, 1024 * 1024, prm)
        exp = oracle.clusters(coords, counts, voff, (1024, 1024, 1), 2, 0, 1, 0, conn, 1)
        _same(res, exp, f"conn{conn}")
        assert len(res["clusters"]) == 2 and res["clusters"]["cells"][0] == 1 << 20


@pytest.mark.parametrize("name,band,shift", [("c2", (18, 40), 1), ("c4", (12, 40), 2), ("c5", (18, 40), 0)])
def test_path_then_clusters_match_oracle(gpu_lib, name, band, shift):
    """Voxelise on the GPU, cluster on the GPU; the oracle does both on the CPU."""
    wl = synth.CONFIGS[name]()
    case = case_from_workload(wl)
    exp_v = case.run_oracle()
    vz = run_gpu(gpu_lib, case, gpu_rois=gpu_lib.make_rois(wl.roi_desc))
    prm = gpu_lib.cluster_params(band[0], band[1], shift, 8, 2)
    p = vz.clusters(prm)
    import torch

    torch.cuda.synchronize()
    assert p.fault() == 0
    V = int(exp_v["voxel_offsets"][-1])
    res = p.result(V)
    exp = oracle.clusters(exp_v["coords"][:V], exp_v["counts"][:V], exp_v["voxel_offsets"], wl.grid.dims,
                          wl.grid.num_frames, band[0], band[1], shift, 8, 2)
    assert len(exp["clusters"]) > 5
    _same(res, exp, name)


def test_batched_frames_and_repeat_calls(gpu_lib):
    """The 16-frame batch, twice through the same workspace (no initialisation between calls)."""
    import torch

    wl = synth.throughput(16)
    case = case_from_workload(wl)
    exp_v = case.run_oracle()
    vz = run_gpu(gpu_lib, case, gpu_rois=gpu_lib.make_rois(wl.roi_desc))
    prm = gpu_lib.cluster_params(18, 40, 1, 8, 1)
    V = int(exp_v["voxel_offsets"][-1])
    exp = oracle.clusters(exp_v["coords"][:V], exp_v["counts"][:V], exp_v["voxel_offsets"], wl.grid.dims, 16,
                          18, 40, 1, 8, 1)
    p = vz.clusters(prm)
    for _ in range(3):
        torch.cuda.synchronize()
        _same(p.result(V), exp, "c2x16")
        vz.clusters(prm, proposer=p)


def test_contract_breaks_set_the_fault_bit(gpu_lib):
    coords, counts, voff, dims = _frames(7, [(30, 30), (30, 30)], 0.4)
    B, cap = 2, int(np.max(np.diff(voff))) + 5
    prm = gpu_lib.cluster_params(0, 3, 0, 8, 1)
    res, p = _gpu(gpu_lib, coords, counts, voff, dims, B, cap, prm)
    assert p.fault() == 0
    outside = coords.copy()
    outside[5, 3] = dims[0]
    other = coords.copy()
    other[3, 0] = 1
    for bad in (outside, other):
        _, p = _gpu(gpu_lib, bad, counts, voff, dims, B, cap, prm)
        assert p.fault() == gpu_lib.FAULT_VOXELS
    for bad_off in ([1, voff[1], voff[2]], [0, voff[2], voff[1]], [0, voff[1], B * cap + 1]):
        # labels cover rows [0, off[B]) clamped to the arrays, whatever the offsets hold
        _, p = _gpu(gpu_lib, coords, counts, np.array(bad_off), dims, B, cap, prm, check_rest=False)
        assert p.fault() == gpu_lib.FAULT_VOXELS, bad_off
