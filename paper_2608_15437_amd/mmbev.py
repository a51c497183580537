"""Python binding of libmmbev (ctypes): argument marshalling only.

The names mirror include/mmbev.h.  PyTorch supplies device memory and the
current stream; every step of the voxelisation runs in the HIP kernels of
libmmbev.so.  There is no fallback: if the library or a GPU is missing, the
calls raise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmmbev.so")

OK, ERR_INVALID_ARG, ERR_WORKSPACE, ERR_UNSUPPORTED, ERR_HIP = 0, -1, -2, -3, -4
FAULT_POINT_OFFSETS, FAULT_ROI_OFFSETS, FAULT_INTERNAL, FAULT_VOXELS = 1, 2, 4, 8

ROI_DTYPE = np.dtype([("cx", "<f4"), ("cy", "<f4"), ("cos_yaw", "<f4"), ("sin_yaw", "<f4"),
                      ("ext_x", "<f4"), ("ext_y", "<f4"), ("reserved0", "<f4"), ("reserved1", "<f4")])


class mmbev_points_t(ctypes.Structure):
    _fields_ = [("feat", ctypes.c_void_p), ("stride", ctypes.c_int64), ("num_features", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("num_points", ctypes.c_int64), ("frame_offsets", ctypes.c_void_p)]


class mmbev_rois_t(ctypes.Structure):
    _fields_ = [("boxes", ctypes.c_void_p), ("frame_offsets", ctypes.c_void_p), ("num_rois", ctypes.c_int32),
                ("max_rois_per_frame", ctypes.c_int32)]


class mmbev_grid_t(ctypes.Structure):
    _fields_ = [("range_min", ctypes.c_float * 3), ("voxel_size", ctypes.c_float * 3),
                ("dims", ctypes.c_int32 * 3), ("max_points", ctypes.c_int32), ("max_voxels", ctypes.c_int32),
                ("num_sweeps", ctypes.c_int32), ("num_frames", ctypes.c_int32)]


class mmbev_options_t(ctypes.Structure):
    _fields_ = [("out_of_roi_keep_rate", ctypes.c_float), ("reserved", ctypes.c_uint32), ("seed", ctypes.c_uint64)]


class mmbev_cluster_params_t(ctypes.Structure):
    _fields_ = [("z_min", ctypes.c_int32), ("z_max", ctypes.c_int32), ("cell_shift", ctypes.c_int32),
                ("connectivity", ctypes.c_int32), ("min_cells", ctypes.c_int32), ("reserved", ctypes.c_int32)]


CLUSTER_DTYPE = np.dtype([("frame", "<i4"), ("root", "<i4"), ("cells", "<i4"), ("voxels", "<i4"), ("points", "<i4"),
                          ("x0", "<i4"), ("y0", "<i4"), ("x1", "<i4"), ("y1", "<i4"), ("reserved", "<i4"),
                          ("sum_x", "<i8"), ("sum_y", "<i8")])


DETECTION_DTYPE = np.dtype([("x", "<f8"), ("y", "<f8"), ("yaw", "<f8"), ("length", "<f8"), ("width", "<f8"),
                            ("vx", "<f8"), ("vy", "<f8"), ("cls", "<i4"), ("reserved", "<i4")])
EGO_DTYPE = np.dtype([("speed", "<f8"), ("dx", "<f8"), ("dy", "<f8"), ("dyaw", "<f8")])
CRIT_DTYPE = np.dtype([("ttc", "<f8"), ("flags", "<i4"), ("rank", "<i4")])
CLASS_VRU, CLASS_MOTORIZED, CLASS_STATIC = 0, 1, 2
CRIT_GEOM, CRIT_SAFETY, CRIT_MANDATORY, CRIT_DROPPED = 1, 2, 4, 8


class mmbev_policy_t(ctypes.Structure):
    _fields_ = [("dt", ctypes.c_double), ("margin", ctypes.c_double), ("a_brake", ctypes.c_double),
                ("d_min", ctypes.c_double), ("theta_max_deg", ctypes.c_double), ("theta_min_deg", ctypes.c_double),
                ("speed_wide", ctypes.c_double), ("speed_narrow", ctypes.c_double), ("tau_vru", ctypes.c_double),
                ("tau_motorized", ctypes.c_double), ("r_coll", ctypes.c_double), ("slow_speed", ctypes.c_double),
                ("dense_count", ctypes.c_int32), ("n_full", ctypes.c_int32), ("n_reduced", ctypes.c_int32),
                ("max_optional", ctypes.c_int32), ("reserved", ctypes.c_int32), ("_pad", ctypes.c_int32),
                ("fallback_length", ctypes.c_double), ("fallback_width", ctypes.c_double)]


# Paper values: cone bounds 60 / 15 degrees, TTC thresholds 1.5 s / 2.5 s,
# sweep counts 10 / 5 (Sec. IV-C, IV-G); the rest are deployment choices.
DEFAULT_POLICY = dict(dt=0.5, margin=0.5, a_brake=6.0, d_min=10.0, theta_max_deg=60.0, theta_min_deg=15.0,
                      speed_wide=5.0, speed_narrow=30.0, tau_vru=1.5, tau_motorized=2.5, r_coll=2.0, slow_speed=5.0,
                      dense_count=64, n_full=10, n_reduced=5, max_optional=64, fallback_length=108.0,
                      fallback_width=108.0)


def policy(**kw) -> mmbev_policy_t:
    v = dict(DEFAULT_POLICY)
    v.update(kw)
    return mmbev_policy_t(**{k: v[k] for k in DEFAULT_POLICY}, reserved=0)


class MmbevError(RuntimeError):
    pass


_lib = None


def load() -> ctypes.CDLL:
    """Load libmmbev.so (built in-tree by build.py); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MmbevError(f"{LIB_PATH} is missing: build it with paper_2608_15437_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        p = ctypes.c_void_p
        L.mmbev_abi_version.argtypes = []
        L.mmbev_abi_version.restype = ctypes.c_int32
        L.mmbev_status_string.argtypes = [ctypes.c_int32]
        L.mmbev_status_string.restype = ctypes.c_char_p
        L.mmbev_roi_voxelize_workspace_bytes.argtypes = [ctypes.POINTER(mmbev_grid_t), ctypes.c_int64,
                                                         ctypes.c_int32, ctypes.c_int32]
        L.mmbev_roi_voxelize_workspace_bytes.restype = ctypes.c_size_t
        L.mmbev_workspace_init.argtypes = [p, ctypes.c_size_t, p]
        L.mmbev_workspace_init.restype = ctypes.c_int32
        L.mmbev_make_rois.argtypes = [p, ctypes.c_int64, p]
        L.mmbev_make_rois.restype = ctypes.c_int32
        L.mmbev_roi_voxelize.argtypes = [ctypes.POINTER(mmbev_points_t), p, p, ctypes.POINTER(mmbev_rois_t), p,
                                         ctypes.POINTER(mmbev_grid_t), p, p, p, p, p, p, ctypes.c_size_t, p]
        L.mmbev_roi_voxelize.restype = ctypes.c_int32
        L.mmbev_roi_voxelize_profiled.argtypes = L.mmbev_roi_voxelize.argtypes + [p, ctypes.c_int32, p]
        L.mmbev_roi_voxelize_profiled.restype = ctypes.c_int32
        a = L.mmbev_roi_voxelize.argtypes
        L.mmbev_roi_voxelize_ex.argtypes = a[:6] + [ctypes.POINTER(mmbev_options_t)] + a[6:] + [p, ctypes.c_int32, p]
        L.mmbev_roi_voxelize_ex.restype = ctypes.c_int32
        L.mmbev_roi_voxelize_noalloc.argtypes = a[:11] + [p, p]
        L.mmbev_roi_voxelize_noalloc.restype = ctypes.c_int32
        L.mmbev_scatter_to_bev.argtypes = [p, p, p, ctypes.c_int32, ctypes.POINTER(mmbev_grid_t), p, p, p]
        L.mmbev_scatter_to_bev.restype = ctypes.c_int32
        L.mmbev_voxel_clusters_workspace_bytes.argtypes = [ctypes.POINTER(mmbev_grid_t),
                                                           ctypes.POINTER(mmbev_cluster_params_t)]
        L.mmbev_voxel_clusters_workspace_bytes.restype = ctypes.c_size_t
        L.mmbev_voxel_clusters.argtypes = [p, p, p, ctypes.POINTER(mmbev_grid_t),
                                           ctypes.POINTER(mmbev_cluster_params_t), p, p, p, p, ctypes.c_size_t, p]
        L.mmbev_voxel_clusters.restype = ctypes.c_int32
        L.mmbev_build_rois.argtypes = [p, p, ctypes.c_int32, p, ctypes.POINTER(mmbev_policy_t), p, p, p, p, p]
        L.mmbev_build_rois.restype = ctypes.c_int32
        _lib = L
    return _lib


def _check(status: int, what: str) -> None:
    if status != OK:
        msg = load().mmbev_status_string(status).decode()
        raise MmbevError(f"{what}: {msg} ({status})")


def abi_version() -> int:
    return int(load().mmbev_abi_version())


def grid_params(range_min, voxel_size, dims, max_points, max_voxels, num_sweeps, num_frames) -> mmbev_grid_t:
    g = mmbev_grid_t()
    for d in range(3):
        g.range_min[d] = float(range_min[d])
        g.voxel_size[d] = float(voxel_size[d])
        g.dims[d] = int(dims[d])
    g.max_points, g.max_voxels = int(max_points), int(max_voxels)
    g.num_sweeps, g.num_frames = int(num_sweeps), int(num_frames)
    return g


def roi_voxelize_workspace_bytes(grid: mmbev_grid_t, num_points: int, num_features: int,
                                 max_rois_per_frame: int) -> int:
    return int(load().mmbev_roi_voxelize_workspace_bytes(ctypes.byref(grid), int(num_points), int(num_features),
                                                         int(max_rois_per_frame)))


def _ptr(t) -> int | None:
    if t is None:
        return None
    return int(t.data_ptr()) if t.numel() > 0 else None


def _stream(stream) -> int | None:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) or None


def workspace_init(workspace, stream=None) -> None:
    _check(load().mmbev_workspace_init(_ptr(workspace), workspace.numel() * workspace.element_size(),
                                       _stream(stream)), "mmbev_workspace_init")


def make_rois(desc) -> np.ndarray:
    """ROI records (host) from descriptor rows (cx, cy, length, width, yaw, margin)."""
    desc = np.ascontiguousarray(desc, dtype=np.float64).reshape(-1, 6)
    out = np.zeros(len(desc), dtype=ROI_DTYPE)
    _check(load().mmbev_make_rois(desc.ctypes.data if len(desc) else None, len(desc),
                                  out.ctypes.data if len(desc) else None), "mmbev_make_rois")
    return out


def roi_voxelize(feat, frame_offsets, sweep_ids, sweep_poses, rois, roi_frame_offsets, roi_sweep_budget,
                 grid: mmbev_grid_t, out_coords, out_counts, out_feats, out_point_idx, out_voxel_offsets,
                 workspace, max_rois_per_frame: int, stream=None, events=None, rho_out: float = 0.0,
                 seed: int = 0) -> int:
    """Enqueue one call of mmbev_roi_voxelize on `stream` (torch tensors on the GPU).

    feat: float32 [C][stride] (SoA); frame_offsets: int64 [B+1]; sweep_ids: uint8 [N];
    sweep_poses: float32 [B][S][12]; rois: float32 [R][8] (mmbev_roi_t records);
    roi_frame_offsets: int32 [B+1]; roi_sweep_budget: uint8 [R]; outputs as in mmbev.h.
    rho_out, seed: the out-of-ROI keep rate and its seed; either nonzero selects
    mmbev_roi_voxelize_ex.
    """
    C = int(feat.shape[0])
    N = int(sweep_ids.numel())
    pts = mmbev_points_t(feat=_ptr(feat), stride=int(feat.stride(0)) if feat.dim() == 2 else N,
                         num_features=C, reserved=0, num_points=N, frame_offsets=_ptr(frame_offsets))
    if N > 0 and feat.dim() == 2 and feat.stride(1) != 1:
        raise MmbevError("feat rows must be contiguous")
    R = int(rois.shape[0])
    rr = mmbev_rois_t(boxes=_ptr(rois), frame_offsets=_ptr(roi_frame_offsets), num_rois=R,
                      max_rois_per_frame=int(max_rois_per_frame))
    args = [ctypes.byref(pts), _ptr(sweep_ids), _ptr(sweep_poses), ctypes.byref(rr), _ptr(roi_sweep_budget),
            ctypes.byref(grid), _ptr(out_coords), _ptr(out_counts), _ptr(out_feats), _ptr(out_point_idx),
            _ptr(out_voxel_offsets), _ptr(workspace), workspace.numel() * workspace.element_size(),
            _stream(stream)]
    if rho_out != 0.0 or seed != 0:
        opt = mmbev_options_t(out_of_roi_keep_rate=float(rho_out), reserved=0, seed=int(seed) & ((1 << 64) - 1))
        evs = events or []
        handles = (ctypes.c_void_p * max(len(evs), 1))(*[int(e.cuda_event) for e in evs])
        used = ctypes.c_int32(0)
        _check(load().mmbev_roi_voxelize_ex(*args[:6], ctypes.byref(opt), *args[6:], handles if evs else None,
                                            len(evs), ctypes.byref(used)), "mmbev_roi_voxelize_ex")
        return int(used.value)
    if events is None:
        _check(load().mmbev_roi_voxelize(*args), "mmbev_roi_voxelize")
        return 0
    # events: torch.cuda.Event objects (timing enabled) that have been recorded once
    handles = (ctypes.c_void_p * len(events))(*[int(e.cuda_event) for e in events])
    used = ctypes.c_int32(0)
    _check(load().mmbev_roi_voxelize_profiled(*args, handles, len(events), ctypes.byref(used)),
           "mmbev_roi_voxelize_profiled")
    return int(used.value)


def roi_voxelize_noalloc(feat, frame_offsets, sweep_ids, sweep_poses, rois, roi_frame_offsets, roi_sweep_budget,
                         grid: mmbev_grid_t, out_coords, out_counts, out_feats, out_point_idx, out_voxel_offsets,
                         max_rois_per_frame: int, out_fault=None, stream=None) -> None:
    """Enqueue mmbev_roi_voxelize_noalloc on `stream`: the same call as
    roi_voxelize, with the library's own per-device scratch as its workspace
    (nothing allocated).  out_fault: optional int32 tensor of one element that
    receives the call's fault word."""
    C = int(feat.shape[0])
    N = int(sweep_ids.numel())
    if N > 0 and feat.dim() == 2 and feat.stride(1) != 1:
        raise MmbevError("feat rows must be contiguous")
    pts = mmbev_points_t(feat=_ptr(feat), stride=int(feat.stride(0)) if feat.dim() == 2 else N,
                         num_features=C, reserved=0, num_points=N, frame_offsets=_ptr(frame_offsets))
    rr = mmbev_rois_t(boxes=_ptr(rois), frame_offsets=_ptr(roi_frame_offsets), num_rois=int(rois.shape[0]),
                      max_rois_per_frame=int(max_rois_per_frame))
    _check(load().mmbev_roi_voxelize_noalloc(ctypes.byref(pts), _ptr(sweep_ids), _ptr(sweep_poses), ctypes.byref(rr),
                                             _ptr(roi_sweep_budget), ctypes.byref(grid), _ptr(out_coords),
                                             _ptr(out_counts), _ptr(out_feats), _ptr(out_point_idx),
                                             _ptr(out_voxel_offsets), _ptr(out_fault), _stream(stream)),
           "mmbev_roi_voxelize_noalloc")


def bev_map_shape(grid: mmbev_grid_t, num_features: int) -> tuple:
    """Shape of the ScatterToBEV map: [num_frames][C*Dz][Dy][Dx]."""
    Dx, Dy, Dz = grid.dims[0], grid.dims[1], grid.dims[2]
    return (grid.num_frames, int(num_features) * Dz, Dy, Dx)


def scatter_to_bev(coords, feats, voxel_offsets, grid: mmbev_grid_t, bev_map, fault=None, stream=None) -> None:
    """Enqueue mmbev_scatter_to_bev on `stream` (torch tensors on the GPU).

    coords int32 [rows][4], feats fp32 [rows][C], voxel_offsets int64 [B+1]
    (as written by mmbev_roi_voxelize); bev_map fp32 of bev_map_shape(grid, C),
    every element written; fault: optional int32 tensor of one element that
    receives MMBEV_FAULT_VOXELS when the rows break the contract.
    """
    C = int(feats.shape[1])
    if tuple(bev_map.shape) != bev_map_shape(grid, C) or not bev_map.is_contiguous():
        raise MmbevError(f"bev_map must be a contiguous tensor of shape {bev_map_shape(grid, C)}")
    if not (coords.is_contiguous() and feats.is_contiguous()):
        raise MmbevError("coords and feats must be contiguous")
    _check(load().mmbev_scatter_to_bev(_ptr(coords), _ptr(feats), _ptr(voxel_offsets), C, ctypes.byref(grid),
                                       _ptr(bev_map), _ptr(fault), _stream(stream)), "mmbev_scatter_to_bev")


def build_rois(dets, det_offsets, ego, pol: mmbev_policy_t) -> dict:
    """mmbev_build_rois on host arrays: dets DETECTION_DTYPE [D], det_offsets
    int32 [B+1], ego EGO_DTYPE [B].  Returns ROI records (ROI_DTYPE), budgets
    uint8, roi_offsets int32 [B+1], crit (CRIT_DTYPE, input order) and the
    sweep count of each frame."""
    dets = np.ascontiguousarray(dets, dtype=DETECTION_DTYPE)
    det_offsets = np.ascontiguousarray(det_offsets, dtype=np.int32)
    ego = np.ascontiguousarray(ego, dtype=EGO_DTYPE)
    B = len(det_offsets) - 1
    D = int(det_offsets[-1])
    cap = 2 * D + B
    rois = np.zeros(max(cap, 1), dtype=ROI_DTYPE)
    budgets = np.zeros(max(cap, 1), dtype=np.uint8)
    roff = np.zeros(B + 1, dtype=np.int32)
    crit = np.zeros(max(D, 1), dtype=CRIT_DTYPE)
    sweeps = np.zeros(max(B, 1), dtype=np.int32)
    _check(load().mmbev_build_rois(dets.ctypes.data if D else None, det_offsets.ctypes.data, B, ego.ctypes.data,
                                   ctypes.byref(pol), rois.ctypes.data, budgets.ctypes.data, roff.ctypes.data,
                                   crit.ctypes.data, sweeps.ctypes.data), "mmbev_build_rois")
    R = int(roff[-1])
    return {"rois": rois[:R], "budgets": budgets[:R], "roi_offsets": roff, "crit": crit[:D], "sweeps": sweeps[:B]}


def cluster_params(z_min: int, z_max: int, cell_shift: int = 0, connectivity: int = 8,
                   min_cells: int = 1) -> mmbev_cluster_params_t:
    return mmbev_cluster_params_t(int(z_min), int(z_max), int(cell_shift), int(connectivity), int(min_cells), 0)


def voxel_clusters_workspace_bytes(grid: mmbev_grid_t, params: mmbev_cluster_params_t) -> int:
    return int(load().mmbev_voxel_clusters_workspace_bytes(ctypes.byref(grid), ctypes.byref(params)))


def voxel_clusters(coords, counts, voxel_offsets, grid: mmbev_grid_t, params: mmbev_cluster_params_t,
                   out_clusters, out_offsets, out_labels, workspace, stream=None) -> None:
    """Enqueue mmbev_voxel_clusters (torch tensors on the GPU).  out_clusters:
    any contiguous tensor of rows * 56 bytes (rows = num_frames * max_voxels);
    out_offsets int64 [B+1]; out_labels int32 [rows]."""
    _check(load().mmbev_voxel_clusters(_ptr(coords), _ptr(counts), _ptr(voxel_offsets), ctypes.byref(grid),
                                       ctypes.byref(params), _ptr(out_clusters), _ptr(out_offsets), _ptr(out_labels),
                                       _ptr(workspace), workspace.numel() * workspace.element_size(),
                                       _stream(stream)), "mmbev_voxel_clusters")


class ClusterProposer:
    """Owns the outputs and workspace of mmbev_voxel_clusters for one grid."""

    def __init__(self, grid: mmbev_grid_t, params: mmbev_cluster_params_t, device):
        import torch

        self.grid, self.params, self.device = grid, params, torch.device(device)
        rows = grid.num_frames * grid.max_voxels
        nbytes = voxel_clusters_workspace_bytes(grid, params)
        if nbytes == 0:
            raise MmbevError("invalid sizes for mmbev_voxel_clusters_workspace_bytes")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.out = torch.zeros(rows * CLUSTER_DTYPE.itemsize // 8, dtype=torch.int64, device=self.device)
        self.offsets = torch.zeros(grid.num_frames + 1, dtype=torch.int64, device=self.device)
        self.labels = torch.full((rows,), -7, dtype=torch.int32, device=self.device)

    def run(self, coords, counts, voxel_offsets, stream=None) -> None:
        voxel_clusters(coords, counts, voxel_offsets, self.grid, self.params, self.out, self.offsets, self.labels,
                       self.workspace, stream)

    def fault(self) -> int:
        return int(self.workspace[:4].cpu().numpy().view(np.int32)[0])

    def result(self, num_voxels: int) -> dict:
        """Clusters (CLUSTER_DTYPE), offsets [B+1] and the labels of the first num_voxels rows (synchronises)."""
        off = self.offsets.cpu().numpy()
        n = int(off[-1])
        cl = self.out[:n * CLUSTER_DTYPE.itemsize // 8].cpu().numpy().view(CLUSTER_DTYPE)
        return {"clusters": cl, "cluster_offsets": off, "voxel_labels": self.labels[:num_voxels].cpu().numpy()}


class Voxelizer:
    """Owns device inputs, outputs and workspace for repeated calls on one batch shape.

    All buffers are torch tensors on `device`; `run()` enqueues one call on the
    current stream and returns without waiting.
    """

    def __init__(self, feat, frame_offsets, sweep_ids, sweep_poses, rois, roi_frame_offsets, roi_sweep_budget,
                 grid: mmbev_grid_t, max_rois_per_frame: int, device, rho_out: float = 0.0, seed: int = 0):
        import torch

        self.device = torch.device(device)
        dev = self.device

        def up(a, dtype):
            return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).to(dev)

        self.feat = up(feat, torch.float32)
        self.frame_offsets = up(frame_offsets, torch.int64)
        self.sweep_ids = up(sweep_ids, torch.uint8)
        self.sweep_poses = up(sweep_poses, torch.float32)
        rois = np.ascontiguousarray(rois)
        rec = rois.view(np.float32).reshape(-1, 8) if rois.dtype.fields else np.asarray(rois, np.float32)
        self.rois = up(rec.reshape(-1, 8), torch.float32)
        self.roi_frame_offsets = up(roi_frame_offsets, torch.int32)
        self.roi_sweep_budget = up(roi_sweep_budget, torch.uint8)
        self.grid = grid
        self.max_rois = int(max_rois_per_frame)
        self.rho_out, self.seed = float(rho_out), int(seed)
        B, cap, M, C = grid.num_frames, grid.max_voxels, grid.max_points, int(self.feat.shape[0])
        rows = B * cap
        self.out_coords = torch.full((rows, 4), -7, dtype=torch.int32, device=dev)
        self.out_counts = torch.full((rows,), -7, dtype=torch.int32, device=dev)
        self.out_feats = torch.full((rows, C), -7.0, dtype=torch.float32, device=dev)
        self.out_point_idx = torch.full((rows, M), -7, dtype=torch.int32, device=dev)
        self.out_voxel_offsets = torch.zeros(B + 1, dtype=torch.int64, device=dev)
        nbytes = roi_voxelize_workspace_bytes(grid, int(self.sweep_ids.numel()), C, self.max_rois)
        if nbytes == 0:
            raise MmbevError("invalid sizes for mmbev_roi_voxelize_workspace_bytes")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        workspace_init(self.workspace)

    def run(self, stream=None, events=None) -> int:
        return roi_voxelize(self.feat, self.frame_offsets, self.sweep_ids, self.sweep_poses, self.rois,
                            self.roi_frame_offsets, self.roi_sweep_budget, self.grid, self.out_coords,
                            self.out_counts, self.out_feats, self.out_point_idx, self.out_voxel_offsets,
                            self.workspace, self.max_rois, stream, events, self.rho_out, self.seed)

    def scatter_to_bev(self, bev_map=None, fault=None, stream=None):
        """ScatterToBEV of this Voxelizer's outputs into bev_map (allocated when None); returns the map."""
        import torch

        if bev_map is None:
            bev_map = torch.empty(bev_map_shape(self.grid, self.out_feats.shape[1]), dtype=torch.float32,
                                  device=self.device)
        scatter_to_bev(self.out_coords, self.out_feats, self.out_voxel_offsets, self.grid, bev_map, fault, stream)
        return bev_map

    def clusters(self, params: mmbev_cluster_params_t, proposer=None, stream=None) -> "ClusterProposer":
        """The connected-component proposer over this Voxelizer's outputs (enqueued; returns the proposer)."""
        if proposer is None:
            proposer = ClusterProposer(self.grid, params, self.device)
        proposer.run(self.out_coords, self.out_counts, self.out_voxel_offsets, stream)
        return proposer

    def fault(self) -> int:
        """Device fault word of the last completed call (synchronises)."""
        return int(self.workspace[:4].cpu().numpy().view(np.int32)[0])

    def header(self) -> dict:
        """Per-call counters of the last completed call (synchronises)."""
        h = self.workspace[:64].cpu().numpy().view(np.uint32)
        return {"fault": int(h[0]), "epoch": int(h[1]), "kept": int(h[2]), "voxels": int(h[3]),
                "capped_voxels": int(h[4]), "any_capped": int(h[5]), "filter_chunks": int(h[6]),
                "pair_chunks": int(h[7]), "voxel_tiles": int(h[8]), "most_frame": int(h[9]), "most_pairs": int(h[10])}

    def result(self) -> dict:
        """Outputs of the last completed call as numpy arrays trimmed to V rows (synchronises)."""
        off = self.out_voxel_offsets.cpu().numpy()
        V = int(off[-1])
        return {"coords": self.out_coords[:V].cpu().numpy(), "counts": self.out_counts[:V].cpu().numpy(),
                "feats": self.out_feats[:V].cpu().numpy(), "point_idx": self.out_point_idx[:V].cpu().numpy(),
                "voxel_offsets": off}


def voxelizer_for_workload(wl, device, rois=None, rho_out: float = 0.0, seed: int = 0) -> Voxelizer:
    """A Voxelizer for a synth workload; ROI records from the library's mmbev_make_rois."""
    gr = wl.grid
    g = grid_params(gr.range_min, gr.voxel_size, gr.dims, gr.max_points, gr.max_voxels, gr.num_sweeps,
                    gr.num_frames)
    recs = make_rois(wl.roi_desc) if rois is None else rois
    return Voxelizer(wl.feat, wl.frame_offsets, wl.sweep_ids, wl.poses, recs, wl.roi_offsets, wl.budgets, g,
                     max(wl.max_rois_per_frame, 1), device, rho_out, seed)


def roi_voxelize_workload(wl, device) -> dict:
    vz = voxelizer_for_workload(wl, device)
    vz.run()
    return vz.result()
