"""Pins of the oracle's ScatterToBEV (Alg. 1's return value; Sec. IV-F: the
voxel features written into a zero-initialised bird's-eye-view map by voxel
coordinate, the map shaped like a dense pipeline's).

Reading: the height axis is folded into channels, map[b][c*Dz + iz][iy][ix]
= feature c of voxel (b, iz, iy, ix).  Pinned to a hand-derived fixture, to
the dense-tensor route a dense pipeline takes ([B][C][Dz][Dy][Dx] viewed as
[B][C*Dz][Dy][Dx]), to the pillar map when Dz = 1, and to round-trip and
count invariants on voxels from the whole path.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bev_hand.json")


def _hand():
    g = json.load(open(GOLDEN))
    return g, oracle.scatter_to_bev(np.array(g["coords"]), np.array(g["feats"], np.float32), g["voxel_offsets"],
                                    g["dims"], g["num_frames"])


def test_hand_fixture():
    g, m = _hand()
    Dx, Dy, Dz = g["dims"]
    assert m.shape == (g["num_frames"], 3 * Dz, Dy, Dx)
    flat = m.reshape(-1)
    seen = np.zeros(flat.size, dtype=bool)
    for e in g["expected"]:
        assert m[e["b"], e["channel"], e["y"], e["x"]] == e["value"]
        assert flat[e["flat"]] == e["value"]
        seen[e["flat"]] = True
    assert np.all(flat[~seen] == 0.0)


def _voxels(wl):
    r = oracle.run_workload(wl)
    V = int(r["voxel_offsets"][-1])
    return r["coords"][:V], r["feats"][:V], r["voxel_offsets"]


def test_matches_dense_tensor_view():
    """The dense pipeline's route: a [B][C][Dz][Dy][Dx] tensor viewed with the height folded into channels."""
    wl = synth.small(5, frames=3, max_voxels=10 ** 5, max_points=8)
    coords, feats, voff = _voxels(wl)
    Dx, Dy, Dz = wl.grid.dims
    B, C = wl.grid.num_frames, feats.shape[1]
    idx = []
    vals = []
    for c in range(C):
        idx.append(np.stack([coords[:, 0], np.full(len(coords), c), coords[:, 1], coords[:, 2], coords[:, 3]]))
        vals.append(feats[:, c])
    dense = torch.sparse_coo_tensor(torch.from_numpy(np.concatenate(idx, axis=1)).long(),
                                    torch.from_numpy(np.concatenate(vals)), (B, C, Dz, Dy, Dx)).to_dense()
    m = oracle.scatter_to_bev(coords, feats, voff, (Dx, Dy, Dz), B)
    assert np.array_equal(dense.reshape(B, C * Dz, Dy, Dx).numpy(), m)


def test_pillar_map_when_height_is_one():
    rng = np.random.default_rng(3)
    B, C, Dx, Dy = 2, 4, 7, 5
    cells = [rng.choice(Dx * Dy, size=n, replace=False) for n in (9, 4)]
    coords = np.concatenate([np.stack([np.full(len(q), b), np.zeros(len(q), int), q // Dx, q % Dx], 1)
                             for b, q in enumerate(cells)]).astype(np.int32)
    feats = rng.standard_normal((len(coords), C)).astype(np.float32)
    voff = np.array([0, 9, 13])
    m = oracle.scatter_to_bev(coords, feats, voff, (Dx, Dy, 1), B)
    assert m.shape == (B, C, Dy, Dx)
    pil = m.reshape(B, C, Dy * Dx)
    for v, (b, _, y, x) in enumerate(coords):
        assert np.array_equal(pil[b, :, y * Dx + x], feats[v])
    assert np.count_nonzero(m) == np.count_nonzero(feats)


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_round_trip_and_counts(name):
    wl = synth.CONFIGS[name]()
    coords, feats, voff = _voxels(wl)
    Dx, Dy, Dz = wl.grid.dims
    B, C = wl.grid.num_frames, feats.shape[1]
    m = oracle.scatter_to_bev(coords, feats, voff, (Dx, Dy, Dz), B)
    for c in range(C):
        got = m[coords[:, 0], c * Dz + coords[:, 1], coords[:, 2], coords[:, 3]]
        assert np.array_equal(got, feats[:, c])
        # the channel block c*Dz .. c*Dz + Dz - 1 holds feature c of every voxel and nothing else
        blk = m[:, c * Dz:(c + 1) * Dz]
        assert np.count_nonzero(blk) == np.count_nonzero(feats[:, c])
        assert np.sum(blk, dtype=np.float64) == pytest.approx(np.sum(feats[:, c], dtype=np.float64), rel=1e-12)


def test_rejects_coordinates_outside_the_grid_or_frame():
    g, _ = _hand()
    feats = np.array(g["feats"], np.float32)
    for bad in ([0, 2, 0, 0], [0, 0, 3, 0], [0, 0, 0, 4], [1, 0, 0, 0], [0, -1, 0, 0]):
        coords = np.array(g["coords"])
        coords[0] = bad
        with pytest.raises(ValueError):
            oracle.scatter_to_bev(coords, feats, g["voxel_offsets"], g["dims"], g["num_frames"])


def test_empty_frames_give_zero_maps():
    m = oracle.scatter_to_bev(np.zeros((0, 4), np.int32), np.zeros((0, 5), np.float32), [0, 0, 0], (6, 4, 3), 2)
    assert m.shape == (2, 15, 4, 6) and not m.any()
