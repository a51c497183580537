"""Pins of the oracle's voxel-grid connected-component proposer (robot
deployment, Sec. VI: object clusters found on the voxel grid, used by the
adaptive scheduler's cluster-shift trigger).

Reading: a bird's-eye-view cell (ix >> s, iy >> s) is occupied when a voxel
of a layer in [z_min, z_max) lies in it; clusters are the 4- or 8-connected
components of occupied cells with at least min_cells cells, listed per frame
by their smallest cell index.  Pinned to a hand-derived fixture, to
scipy.ndimage.label (a different algorithm) on random occupancy grids, and
to invariants on the path's own voxels.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
from scipy import ndimage

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "clusters_hand.json")
FIELDS = ["frame", "root", "cells", "voxels", "points", "x0", "y0", "x1", "y1", "sum_x", "sum_y"]


def _rows(cl):
    return [[int(c[f]) for f in FIELDS] for c in cl]


@pytest.mark.parametrize("k", range(4))
def test_hand_fixture(k):
    g = json.load(open(GOLDEN))
    case = g["cases"][k]
    r = oracle.clusters(g["coords"], g["counts"], g["voxel_offsets"], g["dims"], g["num_frames"], case["z_min"],
                        case["z_max"], case["cell_shift"], case["connectivity"], case["min_cells"])
    assert _rows(r["clusters"]) == case["clusters"]
    assert r["cluster_offsets"].tolist() == case["cluster_offsets"]
    assert r["voxel_labels"].tolist() == case["voxel_labels"]


def _grid_voxels(occ, rng, layers=3):
    """Voxels (one frame, sorted by key) whose column set is the occupied cells of occ [Dy][Dx]."""
    Dy, Dx = occ.shape
    keys = []
    for y, x in zip(*np.nonzero(occ)):
        for z in rng.choice(layers, size=rng.integers(1, layers + 1), replace=False):
            keys.append((int(z) * Dy + int(y)) * Dx + int(x))
    keys = np.sort(np.array(keys, dtype=np.int64))
    coords = np.stack([np.zeros(len(keys)), keys // (Dx * Dy), (keys // Dx) % Dy, keys % Dx], 1).astype(np.int32)
    return coords


@pytest.mark.parametrize("conn", [4, 8])
@pytest.mark.parametrize("seed,shape,density", [(1, (40, 37), 0.3), (2, (64, 64), 0.55), (3, (9, 120), 0.45),
                                                (4, (1, 50), 0.6), (5, (33, 1), 0.5)])
def test_partition_matches_scipy_label(conn, seed, shape, density):
    rng = np.random.default_rng(seed)
    occ = rng.random(shape) < density
    coords = _grid_voxels(occ, rng)
    counts = rng.integers(1, 10, size=len(coords)).astype(np.int32)
    Dy, Dx = shape
    r = oracle.clusters(coords, counts, [0, len(coords)], (Dx, Dy, 3), 1, 0, 3, 0, conn, 1)
    structure = ndimage.generate_binary_structure(2, 1 if conn == 4 else 2)
    lab, n = ndimage.label(occ, structure=structure)
    cl = r["clusters"]
    assert len(cl) == n
    # the same partition: a bijection between scipy's labels and the clusters
    ours = np.full(shape, -1)
    for y, x, v in zip(coords[:, 2], coords[:, 3], r["voxel_labels"]):
        ours[y, x] = v
    pairs = set(zip(lab[occ].tolist(), ours[occ].tolist()))
    assert len(pairs) == n and len({a for a, _ in pairs}) == n and len({b for _, b in pairs}) == n
    # sizes, roots, boxes and sums per cluster
    for k, c in enumerate(cl):
        ys, xs = np.nonzero(ours == k)
        assert c["cells"] == len(ys)
        assert c["root"] == int(np.min(ys * Dx + xs))
        assert (c["x0"], c["y0"], c["x1"], c["y1"]) == (xs.min(), ys.min(), xs.max(), ys.max())
        assert (c["sum_x"], c["sum_y"]) == (xs.sum(), ys.sum())
    # clusters listed by smallest cell
    assert np.all(np.diff(cl["root"]) > 0)
    assert int(cl["voxels"].sum()) == len(coords) and int(cl["points"].sum()) == int(counts.sum())


def test_min_cells_drops_small_components():
    rng = np.random.default_rng(9)
    occ = rng.random((50, 50)) < 0.35
    coords = _grid_voxels(occ, rng)
    counts = np.ones(len(coords), np.int32)
    lab, n = ndimage.label(occ, structure=np.ones((3, 3)))
    sizes = np.bincount(lab[occ])
    for m in (1, 2, 5, 20):
        r = oracle.clusters(coords, counts, [0, len(coords)], (50, 50, 3), 1, 0, 3, 0, 8, m)
        assert len(r["clusters"]) == int(np.sum(sizes[1:] >= m))
        assert np.all(r["clusters"]["cells"] >= m)


def test_cell_shift_equals_coarsened_columns():
    """Cells of 2^s x 2^s columns: the same clusters as shift 0 on coordinates divided by 2^s."""
    rng = np.random.default_rng(12)
    occ = rng.random((60, 70)) < 0.08
    coords = _grid_voxels(occ, rng)
    counts = rng.integers(1, 5, size=len(coords)).astype(np.int32)
    for s in (1, 2, 3):
        a = oracle.clusters(coords, counts, [0, len(coords)], (70, 60, 3), 1, 0, 3, s, 8, 1)
        cc = coords.copy()
        cc[:, 2] >>= s
        cc[:, 3] >>= s
        W = ((70 + (1 << s) - 1) >> s, (60 + (1 << s) - 1) >> s, 3)
        key = (cc[:, 1].astype(np.int64) * W[1] + cc[:, 2]) * W[0] + cc[:, 3]
        order = np.argsort(key, kind="stable")
        b = oracle.clusters(cc[order], counts[order], [0, len(cc)], W, 1, 0, 3, 0, 8, 1)
        for f in ("root", "cells", "voxels", "points", "x0", "y0", "x1", "y1", "sum_x", "sum_y"):
            assert np.array_equal(a["clusters"][f], b["clusters"][f]), (s, f)


def test_on_the_paths_voxels():
    """Frames of the 8-frame workload: every in-band voxel labelled with a cluster containing its cell."""
    wl = synth.c5(frames=2)
    r = oracle.run_workload(wl)
    V = int(r["voxel_offsets"][-1])
    coords, counts = r["coords"][:V], r["counts"][:V]
    dims = wl.grid.dims
    res = oracle.clusters(coords, counts, r["voxel_offsets"], dims, 2, 18, 40, 1, 8, 3)
    cl, lab = res["clusters"], res["voxel_labels"]
    assert len(cl) > 10
    inband = (coords[:, 1] >= 18) & (coords[:, 1] < 40)
    assert np.all(lab[~inband] == -1)
    for k in np.unique(lab[lab >= 0]):
        sel = lab == k
        c = cl[k]
        assert np.all(coords[sel, 0] == c["frame"])
        x, y = coords[sel, 3] >> 1, coords[sel, 2] >> 1
        assert x.min() >= c["x0"] and x.max() <= c["x1"] and y.min() >= c["y0"] and y.max() <= c["y1"]
        assert sel.sum() == c["voxels"] and counts[sel].sum() == c["points"]
    for b in range(2):
        fr = cl[res["cluster_offsets"][b]:res["cluster_offsets"][b + 1]]
        assert np.all(fr["frame"] == b) and np.all(np.diff(fr["root"]) > 0)


def test_rejects_bad_arguments():
    g = json.load(open(GOLDEN))
    for kw in ({"connectivity": 6}, {"min_cells": 0}, {"cell_shift": 9}):
        args = dict(z_min=1, z_max=3, cell_shift=0, connectivity=8, min_cells=1)
        args.update(kw)
        with pytest.raises(ValueError):
            oracle.clusters(g["coords"], g["counts"], g["voxel_offsets"], g["dims"], g["num_frames"], **args)
    bad = np.array(g["coords"])
    bad[2, 3] = 8
    with pytest.raises(ValueError):
        oracle.clusters(bad, g["counts"], g["voxel_offsets"], g["dims"], g["num_frames"], 1, 3)
