"""Shared test utilities: golden fixtures, brute-force checkers, comparisons.

The brute-force checkers here are independent of the oracle's code: the keep
test and quantisation are redone in float64 (decisions compared only where a
point is further than ``tol`` from every ROI edge and voxel face, where fp32
and float64 must agree), and grouping, caps and means are redone with Python
dicts and ``math.fsum``.
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@dataclass
class Case:
    """Raw inputs in the form both sides accept (ROI records given directly)."""
    feat: np.ndarray          # float32 [C][N]
    sweep_ids: np.ndarray     # uint8 [N]
    frame_offsets: np.ndarray  # int64 [B+1]
    poses: np.ndarray         # float32 [B][S][12]
    rois: np.ndarray          # oracle.ROI_DTYPE [R]
    roi_offsets: np.ndarray   # int32 [B+1]
    budgets: np.ndarray       # uint8 [R]
    grid: dict

    @property
    def B(self):
        return len(self.frame_offsets) - 1

    def ogrid(self):
        g = self.grid
        return oracle.make_grid(g["range_min"], g["voxel_size"], g["dims"], g["max_points"], g["max_voxels"],
                                g["num_sweeps"], g["num_frames"])

    def run_oracle(self, rho_out=0.0, seed=0):
        return oracle.roi_voxelize(self.feat, self.frame_offsets, self.sweep_ids, self.poses, self.rois,
                                   self.roi_offsets, self.budgets, self.ogrid(), rho_out, seed)

    def oracle_keep(self, rho_out=0.0, seed=0):
        return oracle.keep(self.feat, self.frame_offsets, self.sweep_ids, self.poses, self.rois,
                           self.roi_offsets, self.budgets, self.ogrid(), rho_out, seed)


def records(rows) -> np.ndarray:
    """ROI records from rows (cx, cy, cos_yaw, sin_yaw, ext_x, ext_y)."""
    rows = np.asarray(rows, dtype=np.float32).reshape(-1, 6)
    out = np.zeros(len(rows), dtype=oracle.ROI_DTYPE)
    for k, name in enumerate(["cx", "cy", "cos_yaw", "sin_yaw", "ext_x", "ext_y"]):
        out[name] = rows[:, k]
    return out


def load_golden(name: str):
    with open(os.path.join(GOLDEN, name)) as f:
        g = json.load(f)
    pts = np.asarray(g["points"], dtype=np.float64)
    feat = np.ascontiguousarray(pts[:, 1:].T.astype(np.float32))
    case = Case(feat=feat, sweep_ids=pts[:, 0].astype(np.uint8),
                frame_offsets=np.asarray(g["frame_offsets"], dtype=np.int64),
                poses=np.asarray(g["poses"], dtype=np.float32),
                rois=records(g["rois"]), roi_offsets=np.asarray(g["roi_offsets"], dtype=np.int32),
                budgets=np.asarray(g["budgets"], dtype=np.uint8), grid=g["grid"])
    return case, g["expected"]


def case_from_workload(wl, rois=None) -> Case:
    gr = wl.grid
    return Case(feat=wl.feat, sweep_ids=wl.sweep_ids, frame_offsets=wl.frame_offsets, poses=wl.poses,
                rois=oracle.make_rois(wl.roi_desc) if rois is None else rois, roi_offsets=wl.roi_offsets,
                budgets=wl.budgets,
                grid=dict(range_min=gr.range_min, voxel_size=gr.voxel_size, dims=gr.dims,
                          max_points=gr.max_points, max_voxels=gr.max_voxels, num_sweeps=gr.num_sweeps,
                          num_frames=gr.num_frames))


# --------------------------------------------------------- float64 checker
def f64_keep(case: Case, tol: float = 5e-5):
    """Keep decision and voxel indices per point, in float64.

    Returns (keep bool[N], ijk int64[N,3], ambiguous bool[N], p64 float64[N,3]).
    A point is ambiguous when it lies within ``tol`` metres of an admitting
    ROI's edge or of a voxel face; elsewhere fp32 and float64 must agree.
    """
    g = case.grid
    S = g["num_sweeps"]
    N = case.feat.shape[1]
    keep = np.zeros(N, dtype=bool)
    amb = np.zeros(N, dtype=bool)
    ijk = np.full((N, 3), -1, dtype=np.int64)
    p64 = np.full((N, 3), np.nan)
    x, y, z = (case.feat[d].astype(np.float64) for d in range(3))
    mn = np.asarray(g["range_min"], dtype=np.float32).astype(np.float64)
    vs = np.asarray(g["voxel_size"], dtype=np.float32).astype(np.float64)
    D = np.asarray(g["dims"], dtype=np.int64)
    for b in range(case.B):
        lo, hi = int(case.frame_offsets[b]), int(case.frame_offsets[b + 1])
        if hi <= lo:
            continue
        s = case.sweep_ids[lo:hi].astype(np.int64)
        valid = s < S
        P = case.poses[b].astype(np.float64)[np.minimum(s, S - 1)]
        xs, ys, zs = x[lo:hi], y[lo:hi], z[lo:hi]
        p = np.stack([P[:, 4 * r] * xs + P[:, 4 * r + 1] * ys + P[:, 4 * r + 2] * zs + P[:, 4 * r + 3]
                      for r in range(3)], axis=1)
        p64[lo:hi] = p
        inroi = np.zeros(hi - lo, dtype=bool)
        amb_r = np.zeros(hi - lo, dtype=bool)
        for j in range(int(case.roi_offsets[b]), int(case.roi_offsets[b + 1])):
            r = case.rois[j]
            c, sn = float(r["cos_yaw"]), float(r["sin_yaw"])
            dx, dy = p[:, 0] - float(r["cx"]), p[:, 1] - float(r["cy"])
            lx, ly = c * dx + sn * dy, c * dy - sn * dx
            slack = np.minimum(float(r["ext_x"]) - np.abs(lx), float(r["ext_y"]) - np.abs(ly))
            admit = s < int(case.budgets[j])
            inroi |= admit & (slack >= 0)
            amb_r |= admit & (np.abs(slack) < tol)
        with np.errstate(invalid="ignore"):
            f = (p - mn) / vs
            inrange = np.all((f >= 0) & (f < D), axis=1)
            frac = f - np.floor(f)
            near = np.any(np.minimum(frac, 1.0 - frac) * vs < tol, axis=1)
        k = valid & inroi & inrange
        keep[lo:hi] = k
        amb[lo:hi] = valid & (amb_r | (near & inroi))
        ii = np.where(k[:, None], np.floor(np.nan_to_num(f, nan=-1.0)), -1).astype(np.int64)
        ijk[lo:hi] = ii
    return keep, ijk, amb, p64


def key_of(b, ijk, dims):
    Dx, Dy, Dz = (int(d) for d in dims)
    return ((b * Dz + int(ijk[2])) * Dy + int(ijk[1])) * Dx + int(ijk[0])


# ------------------------------------------------------ grouping checker
def dict_voxelize(case: Case, kept_idx, kept_key, values):
    """Steps after the keep test, by brute force.

    kept_idx: ascending point indices kept; kept_key: their voxel keys;
    values: float64 [N, C] feature values per point (p' for c < 3).
    """
    g = case.grid
    M, cap, C = g["max_points"], g["max_voxels"], case.feat.shape[0]
    Dx, Dy, Dz = g["dims"]
    out = {"coords": [], "counts": [], "feats": [], "point_idx": [], "voxel_offsets": [0]}
    fo = case.frame_offsets
    for b in range(case.B):
        groups = {}
        for i, k in zip(kept_idx, kept_key):
            if fo[b] <= i < fo[b + 1]:
                groups.setdefault(int(k), []).append(int(i))
        keys = sorted(groups)
        if len(keys) > cap:
            keys = sorted(sorted(keys, key=lambda kk: groups[kk][0])[:cap])
        for k in keys:
            pts = groups[k][:M]
            ix, rest = k % Dx, k // Dx
            iy, rest = rest % Dy, rest // Dy
            iz = rest % Dz
            out["coords"].append([b, iz, iy, ix])
            out["counts"].append(len(pts))
            out["point_idx"].append(pts + [-1] * (M - len(pts)))
            out["feats"].append([math.fsum(values[i, c] for i in pts) / len(pts) for c in range(C)])
        out["voxel_offsets"].append(out["voxel_offsets"][-1] + len(keys))
    return {
        "coords": np.asarray(out["coords"], dtype=np.int64).reshape(-1, 4),
        "counts": np.asarray(out["counts"], dtype=np.int64),
        "feats": np.asarray(out["feats"], dtype=np.float64).reshape(-1, C),
        "point_idx": np.asarray(out["point_idx"], dtype=np.int64).reshape(-1, M),
        "voxel_offsets": np.asarray(out["voxel_offsets"], dtype=np.int64),
    }


def assert_same_voxels(got, exp, feat_atol=1e-5, label=""):
    """Bit-exact structure, features within feat_atol."""
    np.testing.assert_array_equal(np.asarray(got["voxel_offsets"]), np.asarray(exp["voxel_offsets"]),
                                  err_msg=f"{label} voxel_offsets")
    V = int(np.asarray(exp["voxel_offsets"])[-1])
    for name in ("coords", "counts", "point_idx"):
        np.testing.assert_array_equal(np.asarray(got[name])[:V], np.asarray(exp[name])[:V],
                                      err_msg=f"{label} {name}")
    np.testing.assert_allclose(np.asarray(got["feats"], dtype=np.float64)[:V],
                               np.asarray(exp["feats"], dtype=np.float64)[:V], rtol=0, atol=feat_atol,
                               err_msg=f"{label} feats")
