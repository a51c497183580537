"""Parity of ScatterToBEV (mmbev_scatter_to_bev, through the C ABI) with the
oracle's map: every element bit for bit at sizes whose map the host holds
easily, and at the 8-frame 2160 x 2160 x 40 size (a 29.9 GB map) the values
at every voxel plus the count of nonzero elements, which together fix the
whole map."""
import json
import os

import numpy as np
import pytest

import oracle
import synth
from common import case_from_workload
from test_gpu_parity import run_gpu

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bev_hand.json")


def _grid(mb, dims, frames, cap):
    return mb.grid_params((0.0, 0.0, 0.0), (1.0, 1.0, 1.0), dims, 1, cap, 1, frames)


def _gpu_map(mb, coords, feats, voff, grid, fault=True, poison=True):
    """Upload voxel rows (padded to num_frames * max_voxels rows) and scatter them."""
    import torch

    rows = grid.num_frames * grid.max_voxels
    C = feats.shape[1]
    dc = torch.full((rows, 4), -9, dtype=torch.int32, device="cuda:0")
    df = torch.full((rows, C), 77.0, dtype=torch.float32, device="cuda:0")
    V = len(coords)
    if V:
        dc[:V] = torch.from_numpy(np.ascontiguousarray(coords, dtype=np.int32)).cuda()
        df[:V] = torch.from_numpy(np.ascontiguousarray(feats, dtype=np.float32)).cuda()
    dv = torch.from_numpy(np.asarray(voff, dtype=np.int64)).cuda()
    shape = mb.bev_map_shape(grid, C)
    out = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda:0") if poison else \
        torch.empty(shape, dtype=torch.float32, device="cuda:0")
    fw = torch.zeros(1, dtype=torch.int32, device="cuda:0") if fault else None
    mb.scatter_to_bev(dc, df, dv, grid, out, fw)
    torch.cuda.synchronize()
    return out, (int(fw.item()) if fault else 0)


def test_golden_hand_map(gpu_lib):
    g = json.load(open(GOLDEN))
    grid = _grid(gpu_lib, g["dims"], g["num_frames"], 2)
    m, fault = _gpu_map(gpu_lib, np.array(g["coords"]), np.array(g["feats"], np.float32), g["voxel_offsets"], grid)
    assert fault == 0
    flat = m.cpu().numpy().reshape(-1)
    seen = np.zeros(flat.size, dtype=bool)
    for e in g["expected"]:
        assert flat[e["flat"]] == e["value"]
        seen[e["flat"]] = True
    assert np.all(flat[~seen] == 0.0)


def _random_voxels(seed, dims, frames, counts, C):
    """Sorted unique voxels per frame, drawn from the whole grid (dense where counts are large)."""
    rng = np.random.default_rng(seed)
    Dx, Dy, Dz = dims
    cells = Dx * Dy * Dz
    coords, feats, voff = [], [], [0]
    for b in range(frames):
        k = np.sort(rng.choice(cells, size=counts[b], replace=False))
        coords.append(np.stack([np.full(len(k), b), k // (Dx * Dy), (k // Dx) % Dy, k % Dx], 1))
        feats.append(rng.standard_normal((len(k), C)).astype(np.float32))
        voff.append(voff[-1] + len(k))
    return np.concatenate(coords).astype(np.int32), np.concatenate(feats), np.array(voff, np.int64)


@pytest.mark.parametrize("dims,frames,counts,C", [
    ((64, 64, 16), 2, (300, 0), 5),          # one tile per plane, an empty frame
    ((300, 130, 2), 3, (9000, 77800, 5), 4),  # three tiles per plane (last partial), one frame full
    ((333, 61, 3), 2, (4000, 60939), 3),     # plane not a multiple of 4: element stores; full frame
    ((37, 23, 5), 1, (1,), 8),               # tiny plane, one voxel
    ((1, 1, 1), 2, (1, 0), 1),
    ((128, 128, 1), 2, (16384, 100), 6),     # pillar map, one frame dense
])
def test_random_voxels_match_oracle(gpu_lib, dims, frames, counts, C):
    coords, feats, voff = _random_voxels(sum(counts) + C, dims, frames, counts, C)
    cap = max(max(counts), 1)
    grid = _grid(gpu_lib, dims, frames, cap)
    m, fault = _gpu_map(gpu_lib, coords, feats, voff, grid)
    assert fault == 0
    exp = oracle.scatter_to_bev(coords, feats, voff, dims, frames)
    got = m.cpu().numpy()
    assert got.shape == exp.shape
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))


def _path_map(mb, wl):
    case = case_from_workload(wl)
    exp = case.run_oracle()
    vz = run_gpu(mb, case, gpu_rois=mb.make_rois(wl.roi_desc))
    import torch

    fw = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    poisoned = torch.full(mb.bev_map_shape(vz.grid, vz.out_feats.shape[1]), float("nan"), dtype=torch.float32,
                          device="cuda:0")
    m = vz.scatter_to_bev(poisoned, fault=fw)
    torch.cuda.synchronize()
    assert int(fw.item()) == 0
    return m, exp


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_path_then_scatter_matches_oracle(gpu_lib, name):
    """Voxelise on the GPU, scatter on the GPU; the oracle does both on the CPU."""
    wl = synth.CONFIGS[name]()
    m, exp = _path_map(gpu_lib, wl)
    V = int(exp["voxel_offsets"][-1])
    ref = oracle.scatter_to_bev(exp["coords"][:V], exp["feats"][:V], exp["voxel_offsets"], wl.grid.dims,
                                wl.grid.num_frames)
    got = m.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_small_scenes_path_then_scatter(gpu_lib):
    for seed in (1, 2, 3):
        wl = synth.small(seed, frames=3, max_voxels=50 + 400 * (seed - 1), dims=(48, 40, 6))
        m, exp = _path_map(gpu_lib, wl)
        V = int(exp["voxel_offsets"][-1])
        ref = oracle.scatter_to_bev(exp["coords"][:V], exp["feats"][:V], exp["voxel_offsets"], wl.grid.dims,
                                    wl.grid.num_frames)
        assert np.array_equal(m.cpu().numpy().view(np.uint32), ref.view(np.uint32)), seed


def test_full_size_batched_map_by_properties(gpu_lib):
    """8 frames of 2160 x 2160 x 40 (29.9 GB map): values at every voxel, and no other nonzero element."""
    import torch

    wl = synth.c5()
    m, exp = _path_map(gpu_lib, wl)
    V = int(exp["voxel_offsets"][-1])
    co = torch.from_numpy(exp["coords"][:V].astype(np.int64)).cuda()
    fe = exp["feats"][:V]
    Dz = wl.grid.dims[2]
    nonzero = 0
    for c in range(fe.shape[1]):
        got = m[co[:, 0], c * Dz + co[:, 1], co[:, 2], co[:, 3]].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), fe[:, c].view(np.uint32)), c
        nonzero += int(np.count_nonzero(fe[:, c]))
    total = sum(int(torch.count_nonzero(m[b]).item()) for b in range(m.shape[0]))
    assert total == nonzero


def test_unwritten_canvas_is_fully_overwritten_twice(gpu_lib):
    """A second call into the same map (different voxels) leaves nothing of the first."""
    import torch

    dims, frames, C = (300, 130, 2), 2, 3
    grid = _grid(gpu_lib, dims, frames, 20000)
    a = _random_voxels(5, dims, frames, (20000, 3), C)
    b = _random_voxels(6, dims, frames, (7, 19000), C)
    rows = frames * 20000
    out = torch.empty(gpu_lib.bev_map_shape(grid, C), dtype=torch.float32, device="cuda:0")
    for coords, feats, voff in (a, b):
        dc = torch.zeros((rows, 4), dtype=torch.int32, device="cuda:0")
        df = torch.zeros((rows, C), dtype=torch.float32, device="cuda:0")
        dc[:len(coords)] = torch.from_numpy(coords).cuda()
        df[:len(coords)] = torch.from_numpy(feats).cuda()
        gpu_lib.scatter_to_bev(dc, df, torch.from_numpy(voff).cuda(), grid, out)
    torch.cuda.synchronize()
    exp = oracle.scatter_to_bev(*b, dims, frames)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), exp.view(np.uint32))


def test_contract_breaks_set_the_fault_bit(gpu_lib):
    """Rows out of order, outside the grid, of another frame, or bad offsets: the fault bit is set
    (the map is unspecified then, and every access stays inside the buffers)."""
    dims, frames, C = (40, 30, 4), 2, 3
    coords, feats, voff = _random_voxels(9, dims, frames, (500, 400), C)
    grid = _grid(gpu_lib, dims, frames, 600)
    _, fault = _gpu_map(gpu_lib, coords, feats, voff, grid)
    assert fault == 0
    swapped = coords.copy()
    swapped[[10, 11]] = swapped[[11, 10]]
    outside = coords.copy()
    outside[700, 3] = 40
    other = coords.copy()
    other[3, 0] = 1
    huge = coords.copy()
    huge[450] = [1, 2 ** 31 - 1, -2 ** 31, 2 ** 31 - 1]
    for bad in (swapped, outside, other, huge):
        _, fault = _gpu_map(gpu_lib, bad, feats, voff, grid)
        assert fault == gpu_lib.FAULT_VOXELS
    for bad_off in ([1, 500, 900], [0, 900, 500], [0, 500, 1300], [0, 650, 900]):
        _, fault = _gpu_map(gpu_lib, coords, feats, np.array(bad_off), grid)
        assert fault == gpu_lib.FAULT_VOXELS, bad_off
