"""CPU oracle for ROI-aware multi-sweep voxelisation -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (the HIP library and its
binding) never imports, loads or calls it, and the two share no code.

The arithmetic lives in ``oracle.c`` (plain C, single-threaded, built with
``-O2 -ffp-contract=off``); this file only marshals numpy arrays.  The
definition it follows is spelled out in ``oracle.h``: Eq. 6/7 motion
compensation, the Alg. 1 keep test against the Eq. 1 ROI union (with an
optional out-of-ROI keep rate drawn from SplitMix64), quantisation, sort by (key, point index), max_points and
max_voxels caps, fp64 mean pooling, the scatter of the voxel features into a
dense bird's-eye-view map, and the voxel-grid connected-component proposer.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")


class OracleRoi(ctypes.Structure):
    _fields_ = [("cx", ctypes.c_float), ("cy", ctypes.c_float), ("cos_yaw", ctypes.c_float),
                ("sin_yaw", ctypes.c_float), ("ext_x", ctypes.c_float), ("ext_y", ctypes.c_float),
                ("unused0", ctypes.c_float), ("unused1", ctypes.c_float)]


class OracleGrid(ctypes.Structure):
    _fields_ = [("range_min", ctypes.c_float * 3), ("voxel_size", ctypes.c_float * 3),
                ("dims", ctypes.c_int32 * 3), ("max_points", ctypes.c_int32), ("max_voxels", ctypes.c_int32),
                ("num_sweeps", ctypes.c_int32), ("num_frames", ctypes.c_int32)]


ROI_DTYPE = np.dtype([("cx", "<f4"), ("cy", "<f4"), ("cos_yaw", "<f4"), ("sin_yaw", "<f4"),
                      ("ext_x", "<f4"), ("ext_y", "<f4"), ("unused0", "<f4"), ("unused1", "<f4")])

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_LIB_PATH)
        p = ctypes.c_void_p
        L.oracle_make_roi.argtypes = [ctypes.c_double] * 6 + [p]
        L.oracle_make_roi.restype = None
        L.oracle_compensate.argtypes = [p, ctypes.c_float, ctypes.c_float, ctypes.c_float, p]
        L.oracle_compensate.restype = None
        L.oracle_inside.argtypes = [p, ctypes.c_float, ctypes.c_float]
        L.oracle_inside.restype = ctypes.c_int32
        L.oracle_quantize.argtypes = [p, p, p]
        L.oracle_quantize.restype = ctypes.c_int32
        args = [p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64, p, p, p, p, p, p, p]
        L.oracle_keep.argtypes = args + [p, p]
        L.oracle_keep.restype = ctypes.c_int64
        L.oracle_roi_voxelize.argtypes = args + [p, p, p, p, p]
        L.oracle_roi_voxelize.restype = ctypes.c_int64
        bg = [ctypes.c_float, ctypes.c_uint64]
        L.oracle_keep_bg.argtypes = args + bg + [p, p]
        L.oracle_keep_bg.restype = ctypes.c_int64
        L.oracle_roi_voxelize_bg.argtypes = args + bg + [p, p, p, p, p]
        L.oracle_roi_voxelize_bg.restype = ctypes.c_int64
        L.oracle_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_splitmix64.restype = ctypes.c_uint64
        L.oracle_background_threshold.argtypes = [ctypes.c_float]
        L.oracle_background_threshold.restype = ctypes.c_uint32
        L.oracle_background_keep.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64]
        L.oracle_background_keep.restype = ctypes.c_int32
        L.oracle_scatter_to_bev.argtypes = [p, p, p, ctypes.c_int32, ctypes.c_int32, p, p]
        L.oracle_scatter_to_bev.restype = ctypes.c_int32
        L.oracle_clusters.argtypes = [p, p, p, ctypes.c_int32, p, p, p, p, p]
        L.oracle_clusters.restype = ctypes.c_int64
        _lib = L
    return _lib


def make_grid(range_min, voxel_size, dims, max_points, max_voxels, num_sweeps, num_frames) -> OracleGrid:
    g = OracleGrid()
    for d in range(3):
        g.range_min[d] = float(range_min[d])
        g.voxel_size[d] = float(voxel_size[d])
        g.dims[d] = int(dims[d])
    g.max_points, g.max_voxels = int(max_points), int(max_voxels)
    g.num_sweeps, g.num_frames = int(num_sweeps), int(num_frames)
    return g


def grid_of(wl) -> OracleGrid:
    gr = wl.grid
    return make_grid(gr.range_min, gr.voxel_size, gr.dims, gr.max_points, gr.max_voxels, gr.num_sweeps,
                     gr.num_frames)


def make_rois(desc: np.ndarray) -> np.ndarray:
    """ROI records (structured array, 32 B each) from descriptor rows
    (cx, cy, length, width, yaw, margin)."""
    desc = np.asarray(desc, dtype=np.float64).reshape(-1, 6)
    out = np.zeros(len(desc), dtype=ROI_DTYPE)
    L = lib()
    for k, d in enumerate(desc):
        r = OracleRoi()
        L.oracle_make_roi(*[float(x) for x in d], ctypes.byref(r))
        out[k] = (r.cx, r.cy, r.cos_yaw, r.sin_yaw, r.ext_x, r.ext_y, r.unused0, r.unused1)
    return out


def compensate(pose12, x: float, y: float, z: float) -> np.ndarray:
    pose = np.ascontiguousarray(pose12, dtype=np.float32).reshape(12)
    out = np.zeros(3, dtype=np.float32)
    lib().oracle_compensate(pose.ctypes.data, x, y, z, out.ctypes.data)
    return out


def inside(roi_record: np.ndarray, x: float, y: float) -> bool:
    r = np.ascontiguousarray(np.asarray(roi_record, dtype=ROI_DTYPE).reshape(1))
    return bool(lib().oracle_inside(r.ctypes.data, x, y))


def quantize(grid: OracleGrid, p) -> tuple | None:
    p = np.ascontiguousarray(p, dtype=np.float32).reshape(3)
    ijk = np.zeros(3, dtype=np.int32)
    ok = lib().oracle_quantize(ctypes.byref(grid), p.ctypes.data, ijk.ctypes.data)
    return tuple(int(v) for v in ijk) if ok else None


def _common(feat, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets):
    feat = np.ascontiguousarray(feat, dtype=np.float32)
    C, N = feat.shape
    fo = np.ascontiguousarray(frame_offsets, dtype=np.int64)
    sw = np.ascontiguousarray(sweep_ids, dtype=np.uint8)
    po = np.ascontiguousarray(poses, dtype=np.float32)
    ro = np.ascontiguousarray(rois, dtype=ROI_DTYPE)
    rf = np.ascontiguousarray(roi_offsets, dtype=np.int32)
    bu = np.ascontiguousarray(budgets, dtype=np.uint8)
    keep_alive = (feat, fo, sw, po, ro, rf, bu)
    args = [feat.ctypes.data, N, C, N, fo.ctypes.data, sw.ctypes.data, po.ctypes.data,
            ro.ctypes.data if len(ro) else None, rf.ctypes.data, bu.ctypes.data if len(bu) else None]
    return C, N, args, keep_alive


def splitmix64(seed: int, n: int) -> int:
    """n-th output (n >= 1) of SplitMix64 seeded with seed."""
    return int(lib().oracle_splitmix64(seed, n))


def background_threshold(rho: float) -> int:
    return int(lib().oracle_background_threshold(rho))


def keep(feat, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets, grid: OracleGrid,
         rho_out: float = 0.0, seed: int = 0):
    """Kept (key, point index) pairs in point order (steps 1-4)."""
    C, N, args, _ka = _common(feat, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets)
    keys = np.zeros(max(N, 1), dtype=np.uint64)
    idx = np.zeros(max(N, 1), dtype=np.int64)
    K = lib().oracle_keep_bg(*args, ctypes.byref(grid), rho_out, seed, keys.ctypes.data, idx.ctypes.data)
    if K < 0:
        raise ValueError("oracle_keep: bad argument")
    return keys[:K].copy(), idx[:K].copy()


def roi_voxelize(feat, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets, grid: OracleGrid,
                 rho_out: float = 0.0, seed: int = 0):
    """The whole path.  Returns a dict of numpy arrays trimmed to V rows."""
    C, N, args, _ka = _common(feat, frame_offsets, sweep_ids, poses, rois, roi_offsets, budgets)
    B, M, cap = grid.num_frames, grid.max_points, grid.max_voxels
    rows = max(B * cap, 1)
    coords = np.zeros((rows, 4), dtype=np.int32)
    counts = np.zeros(rows, dtype=np.int32)
    feats = np.zeros((rows, C), dtype=np.float32)
    pidx = np.zeros((rows, M), dtype=np.int32)
    voff = np.zeros(B + 1, dtype=np.int64)
    V = lib().oracle_roi_voxelize_bg(*args, ctypes.byref(grid), rho_out, seed, coords.ctypes.data,
                                     counts.ctypes.data, feats.ctypes.data, pidx.ctypes.data, voff.ctypes.data)
    if V < 0:
        raise ValueError("oracle_roi_voxelize: bad argument")
    return {"coords": coords[:V].copy(), "counts": counts[:V].copy(), "feats": feats[:V].copy(),
            "point_idx": pidx[:V].copy(), "voxel_offsets": voff}


def run_workload(wl, rho_out: float = 0.0, seed: int = 0):
    """Oracle output for a synth workload (records built by the oracle's own make_rois)."""
    return roi_voxelize(wl.feat, wl.frame_offsets, wl.sweep_ids, wl.poses, make_rois(wl.roi_desc),
                        wl.roi_offsets, wl.budgets, grid_of(wl), rho_out, seed)


def scatter_to_bev(coords, feats, voxel_offsets, dims, num_frames: int) -> np.ndarray:
    """ScatterToBEV (Alg. 1's return value; Sec. IV-F): the fp32 map
    [num_frames][C*Dz][Dy][Dx] with map[b][c*Dz + iz][iy][ix] = feats[v][c]
    for every voxel v = (b, iz, iy, ix) of frame b (rows voxel_offsets[b] ..
    voxel_offsets[b+1]), zero elsewhere."""
    coords = np.ascontiguousarray(coords, dtype=np.int32).reshape(-1, 4)
    feats = np.ascontiguousarray(feats, dtype=np.float32)
    feats = feats.reshape(len(coords), -1) if len(coords) else feats.reshape(0, max(feats.shape[-1], 1))
    voff = np.ascontiguousarray(voxel_offsets, dtype=np.int64)
    Dx, Dy, Dz = (int(d) for d in dims)
    C = int(feats.shape[1])
    d = np.array([Dx, Dy, Dz], dtype=np.int32)
    out = np.empty((num_frames, C * Dz, Dy, Dx), dtype=np.float32)
    L = lib()
    rc = L.oracle_scatter_to_bev(coords.ctypes.data, feats.ctypes.data, voff.ctypes.data, num_frames, C,
                                 d.ctypes.data, out.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_scatter_to_bev: bad sizes or voxel coordinates")
    return out


CLUSTER_DTYPE = np.dtype([("frame", "<i4"), ("root", "<i4"), ("cells", "<i4"), ("voxels", "<i4"), ("points", "<i4"),
                          ("x0", "<i4"), ("y0", "<i4"), ("x1", "<i4"), ("y1", "<i4"), ("unused", "<i4"),
                          ("sum_x", "<i8"), ("sum_y", "<i8")])


class OracleCCParams(ctypes.Structure):
    _fields_ = [("z_min", ctypes.c_int32), ("z_max", ctypes.c_int32), ("cell_shift", ctypes.c_int32),
                ("connectivity", ctypes.c_int32), ("min_cells", ctypes.c_int32), ("reserved", ctypes.c_int32)]


def clusters(coords, counts, voxel_offsets, dims, num_frames: int, z_min: int, z_max: int, cell_shift: int = 0,
             connectivity: int = 8, min_cells: int = 1) -> dict:
    """The voxel-grid connected-component proposer (robot deployment, Sec. VI):
    connected components (4- or 8-neighbourhood) of the bird's-eye-view
    cells (ix >> s, iy >> s) holding a voxel of a layer in [z_min, z_max),
    at least min_cells cells each, per frame in order of their smallest cell
    index.  Returns the clusters (CLUSTER_DTYPE), cluster_offsets [B+1] and
    voxel_labels (cluster index per voxel row, -1 if none)."""
    coords = np.ascontiguousarray(coords, dtype=np.int32).reshape(-1, 4)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    voff = np.ascontiguousarray(voxel_offsets, dtype=np.int64)
    d = np.array([int(x) for x in dims], dtype=np.int32)
    prm = OracleCCParams(int(z_min), int(z_max), int(cell_shift), int(connectivity), int(min_cells), 0)
    rows = max(len(coords), 1)
    out = np.zeros(rows, dtype=CLUSTER_DTYPE)
    coff = np.zeros(num_frames + 1, dtype=np.int64)
    labels = np.full(rows, -1, dtype=np.int32)
    n = lib().oracle_clusters(coords.ctypes.data, counts.ctypes.data, voff.ctypes.data, num_frames, d.ctypes.data,
                              ctypes.byref(prm), out.ctypes.data, coff.ctypes.data, labels.ctypes.data)
    if n < 0:
        raise ValueError("oracle_clusters: bad arguments or voxel coordinates")
    return {"clusters": out[:n], "cluster_offsets": coff, "voxel_labels": labels[:len(coords)]}
