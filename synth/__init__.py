"""Seeded synthetic inputs for ROI-aware multi-sweep voxelisation.

This module only builds inputs (points, sweep ids, per-sweep ego poses, ROI
descriptors, sweep budgets, grid parameters).  It holds none of the
voxelisation arithmetic and imports neither the GPU library nor the oracle;
both consume what it returns.

Recipes mirror the five workloads the method is measured on:

* ``c1`` tiny single sweep: 32 beams x 625 columns = 20,000 points, 4 ROIs;
* ``c2`` nuScenes-shaped frame: 10 sweeps x 32 x 1085 = 347,200 points,
  30 obstacles, 32 ROIs (30 footprints + 2 motion-extrapolated copies);
* ``c3`` the ``c2`` points with one all-covering ROI (dense voxelisation);
* ``c4`` Ouster-128-shaped frame: 3 sweeps x 128 x 1024 = 393,216 points;
* ``c5`` batch of 8 ``c2``-shaped frames with 256 ROIs each;
* ``throughput(F)`` F ``c2``-shaped frames (seeds 22 + 1000 f) in one batch.
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")


class SceneT(ctypes.Structure):
    _fields_ = [
        ("beams", ctypes.c_int32),
        ("azimuths", ctypes.c_int32),
        ("elev_lo_deg", ctypes.c_double),
        ("elev_hi_deg", ctypes.c_double),
        ("sensor_h", ctypes.c_double),
        ("range_sigma", ctypes.c_double),
        ("r_max", ctypes.c_double),
        ("num_sweeps", ctypes.c_int32),
        ("num_features", ctypes.c_int32),
        ("sweep_dt", ctypes.c_double),
        ("speed_lo", ctypes.c_double),
        ("speed_hi", ctypes.c_double),
        ("yawrate_lo", ctypes.c_double),
        ("yawrate_hi", ctypes.c_double),
        ("num_obstacles", ctypes.c_int32),
        ("axis_aligned", ctypes.c_int32),
        ("obs_len", ctypes.c_double),
        ("obs_wid", ctypes.c_double),
        ("obs_hgt", ctypes.c_double),
        ("obs_jitter", ctypes.c_double),
        ("obs_r_lo", ctypes.c_double),
        ("obs_r_hi", ctypes.c_double),
    ]


class RoiRecipeT(ctypes.Structure):
    _fields_ = [
        ("num_on_obstacles", ctypes.c_int32),
        ("num_extrapolated", ctypes.c_int32),
        ("num_random", ctypes.c_int32),
        ("num_overlapping", ctypes.c_int32),
        ("extrap_speed", ctypes.c_double),
        ("extrap_dt", ctypes.c_double),
        ("rand_extent", ctypes.c_double),
        ("rand_len", ctypes.c_double),
        ("rand_wid", ctypes.c_double),
        ("margin", ctypes.c_double),
        ("budget_lo", ctypes.c_int32),
        ("budget_hi", ctypes.c_int32),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        _lib = ctypes.CDLL(_LIB_PATH)
        p = ctypes.c_void_p
        _lib.synth_obstacles.argtypes = [ctypes.POINTER(SceneT), ctypes.c_uint64, p]
        _lib.synth_obstacles.restype = ctypes.c_int64
        _lib.synth_frame.argtypes = [ctypes.POINTER(SceneT), ctypes.c_uint64, p, ctypes.c_int64,
                                     p, ctypes.c_int64, ctypes.c_int64, p, p]
        _lib.synth_frame.restype = ctypes.c_int64
        _lib.synth_rois.argtypes = [ctypes.POINTER(RoiRecipeT), ctypes.c_uint64, p, ctypes.c_int64, p, p]
        _lib.synth_rois.restype = ctypes.c_int64
    return _lib


@dataclass
class Grid:
    """Voxel grid of one workload (current-frame BEV + height)."""
    range_min: tuple
    voxel_size: tuple
    dims: tuple  # (Dx, Dy, Dz)
    max_points: int
    max_voxels: int
    num_sweeps: int
    num_frames: int


@dataclass
class Workload:
    """One batch of frames: SoA points, sweep ids, poses, ROI descriptors."""
    name: str
    feat: np.ndarray            # float32 [C][N] (row stride == N)
    sweep_ids: np.ndarray       # uint8 [N]
    frame_offsets: np.ndarray   # int64 [B+1]
    poses: np.ndarray           # float32 [B][S][12], row-major [R | T]
    roi_desc: np.ndarray        # float64 [R][6]: cx, cy, length, width, yaw, margin
    roi_offsets: np.ndarray     # int32 [B+1]
    budgets: np.ndarray         # uint8 [R]
    grid: Grid
    obstacles: list = field(default_factory=list)  # per frame float64 [n][7]

    @property
    def num_points(self) -> int:
        return int(self.feat.shape[1])

    @property
    def num_features(self) -> int:
        return int(self.feat.shape[0])

    @property
    def num_frames(self) -> int:
        return int(self.frame_offsets.shape[0] - 1)

    @property
    def max_rois_per_frame(self) -> int:
        return int(np.max(np.diff(self.roi_offsets))) if self.num_frames else 0


# ----------------------------------------------------------------- scenes
def _scene32(sweeps: int, azimuths: int, nobs: int, axis_aligned: bool, features: int,
             speed=(0.0, 15.0)) -> SceneT:
    return SceneT(beams=32, azimuths=azimuths, elev_lo_deg=-30.0, elev_hi_deg=10.0, sensor_h=1.8,
                  range_sigma=0.02, r_max=100.0, num_sweeps=sweeps, num_features=features,
                  sweep_dt=0.05, speed_lo=speed[0], speed_hi=speed[1], yawrate_lo=-0.3, yawrate_hi=0.3,
                  num_obstacles=nobs, axis_aligned=1 if axis_aligned else 0, obs_len=4.5, obs_wid=1.9,
                  obs_hgt=1.7, obs_jitter=0.0 if axis_aligned else 0.1, obs_r_lo=3.0, obs_r_hi=50.0)


def _scene_ouster() -> SceneT:
    # sensor height 1.0 m and 10 Hz sweeps are assumptions for the robot frame
    return SceneT(beams=128, azimuths=1024, elev_lo_deg=-22.5, elev_hi_deg=22.5, sensor_h=1.0,
                  range_sigma=0.02, r_max=100.0, num_sweeps=3, num_features=5, sweep_dt=0.1,
                  speed_lo=0.0, speed_hi=2.0, yawrate_lo=-0.3, yawrate_hi=0.3, num_obstacles=40,
                  axis_aligned=0, obs_len=4.5, obs_wid=1.9, obs_hgt=1.7, obs_jitter=0.1,
                  obs_r_lo=3.0, obs_r_hi=38.0)


def _recipe(on=0, extrap=0, rand=0, overlap=0, extent=30.0, margin=0.5, budget=(1, 1)) -> RoiRecipeT:
    return RoiRecipeT(num_on_obstacles=on, num_extrapolated=extrap, num_random=rand,
                      num_overlapping=overlap, extrap_speed=5.0, extrap_dt=0.5, rand_extent=extent,
                      rand_len=4.5, rand_wid=1.9, margin=margin, budget_lo=budget[0], budget_hi=budget[1])


def _grid(xy: float, zlo: float, zhi: float, vxy: float, vz: float, dims, m: int, cap: int,
          sweeps: int, frames: int) -> Grid:
    return Grid(range_min=(-xy, -xy, zlo), voxel_size=(vxy, vxy, vz), dims=tuple(dims), max_points=m,
                max_voxels=cap, num_sweeps=sweeps, num_frames=frames)


def _build(name: str, scene: SceneT, recipe: RoiRecipeT | None, seeds, grid: Grid,
           fixed_rois=None) -> Workload:
    L = lib()
    B = len(seeds)
    S = scene.num_sweeps
    per_frame = S * scene.beams * scene.azimuths
    N = B * per_frame
    C = scene.num_features
    feat = np.zeros((C, N), dtype=np.float32)
    sweep_ids = np.zeros(N, dtype=np.uint8)
    poses = np.zeros((B, S, 12), dtype=np.float32)
    descs, budgets, roi_off = [], [], [0]

    def one_frame(f):
        # ctypes releases the GIL: frames are generated in parallel into disjoint ranges
        seed = seeds[f]
        obs = np.zeros((max(scene.num_obstacles, 1), 7), dtype=np.float64)
        nobs = L.synth_obstacles(ctypes.byref(scene), seed, obs.ctypes.data)
        obs = np.ascontiguousarray(obs[:nobs])
        pose_f = np.zeros((S, 12), dtype=np.float32)
        n = L.synth_frame(ctypes.byref(scene), seed, obs.ctypes.data, nobs, feat.ctypes.data, N,
                          f * per_frame, sweep_ids.ctypes.data, pose_f.ctypes.data)
        if n != per_frame:
            raise RuntimeError("synth_frame failed")
        poses[f] = pose_f
        return obs

    workers = min(B, max(1, min(os.cpu_count() or 1, 16)))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        obstacles = list(ex.map(one_frame, range(B)))
    for f, seed in enumerate(seeds):
        obs = obstacles[f]
        nobs = len(obs)
        if fixed_rois is not None:
            d, bud = fixed_rois
            d = np.asarray(d, dtype=np.float64).reshape(-1, 6)
            bud = np.asarray(bud, dtype=np.uint8).reshape(-1)
        else:
            cap = recipe.num_on_obstacles + recipe.num_extrapolated + recipe.num_random
            d = np.zeros((max(cap, 1), 6), dtype=np.float64)
            bud = np.zeros(max(cap, 1), dtype=np.uint8)
            nr = L.synth_rois(ctypes.byref(recipe), seed, obs.ctypes.data, nobs, d.ctypes.data,
                              bud.ctypes.data)
            d, bud = d[:nr], bud[:nr]
        descs.append(d)
        budgets.append(bud)
        roi_off.append(roi_off[-1] + len(d))
    frame_offsets = np.arange(B + 1, dtype=np.int64) * per_frame
    return Workload(name=name, feat=feat, sweep_ids=sweep_ids, frame_offsets=frame_offsets, poses=poses,
                    roi_desc=np.concatenate(descs).reshape(-1, 6),
                    roi_offsets=np.asarray(roi_off, dtype=np.int32),
                    budgets=np.concatenate(budgets).astype(np.uint8), grid=grid, obstacles=obstacles)


def c1(seed: int = 11) -> Workload:
    scene = _scene32(1, 625, 6, True, 4)
    return _build("c1", scene, _recipe(rand=4, extent=30.0, margin=0.5, budget=(1, 1)), [seed],
                  _grid(51.2, -5.0, 3.0, 0.2, 0.2, (512, 512, 40), 10, 20000, 1, 1))


def c2(seed: int = 22) -> Workload:
    scene = _scene32(10, 1085, 30, False, 5)
    return _build("c2", scene, _recipe(on=30, extrap=2, margin=0.5, budget=(1, 10)), [seed],
                  _grid(54.0, -5.0, 3.0, 0.075, 0.2, (1440, 1440, 40), 10, 120000, 10, 1))


def c3(seed: int = 22) -> Workload:
    scene = _scene32(10, 1085, 30, False, 5)
    # one ROI centred on the ego, 120 m x 120 m, no margin, all 10 sweeps
    fixed = ([[0.0, 0.0, 120.0, 120.0, 0.0, 0.0]], [10])
    return _build("c3", scene, None, [seed],
                  _grid(54.0, -5.0, 3.0, 0.075, 0.2, (1440, 1440, 40), 10, 120000, 10, 1), fixed_rois=fixed)


def c4(seed: int = 44) -> Workload:
    return _build("c4", _scene_ouster(), _recipe(on=40, rand=24, extent=40.0, margin=0.3, budget=(1, 3)),
                  [seed], _grid(40.0, -3.0, 3.0, 0.05, 0.15, (1600, 1600, 40), 8, 200000, 3, 1))


def c5(seed: int = 55, frames: int = 8) -> Workload:
    scene = _scene32(10, 1085, 30, False, 5)
    recipe = _recipe(on=30, rand=226, overlap=51, extent=54.0, margin=0.5, budget=(1, 10))
    return _build("c5", scene, recipe, [seed + f for f in range(frames)],
                  _grid(54.0, -5.0, 3.0, 0.05, 0.2, (2160, 2160, 40), 10, 160000, 10, frames))


def throughput(frames: int, seed: int = 22) -> Workload:
    """``frames`` c2-shaped frames (seeds seed + 1000 f) voxelised in one call."""
    scene = _scene32(10, 1085, 30, False, 5)
    return _build(f"c2x{frames}", scene, _recipe(on=30, extrap=2, margin=0.5, budget=(1, 10)),
                  [seed + 1000 * f for f in range(frames)],
                  _grid(54.0, -5.0, 3.0, 0.075, 0.2, (1440, 1440, 40), 10, 120000, 10, frames))


def small(seed: int, beams: int = 8, azimuths: int = 64, sweeps: int = 3, frames: int = 2, rois: int = 6,
          features: int = 5, voxel: float = 0.5, dims=(64, 64, 16), max_points: int = 4,
          max_voxels: int = 1000, budget=(1, 3), xy: float = 16.0) -> Workload:
    """Small multi-frame scenes for parity sweeps (the oracle finishes in ms)."""
    scene = _scene32(sweeps, azimuths, 6, False, features, speed=(0.0, 10.0))
    scene.beams = beams
    scene.obs_r_hi = 12.0
    recipe = _recipe(on=3, rand=max(rois - 3, 0), overlap=min(1, max(rois - 3, 0)), extent=xy,
                     margin=0.3, budget=budget)
    return _build(f"small{seed}", scene, recipe, [seed + 7 * f for f in range(frames)],
                  _grid(xy, -2.0, -2.0 + dims[2] * 0.25, voxel, 0.25, dims, max_points, max_voxels,
                        sweeps, frames))


CONFIGS = {"c1": c1, "c2": c2, "c3": c3, "c4": c4, "c5": c5}


# ------------------------------------------------------------- detections
# The detection cache B^{t-1} of the temporal-ROI selector: boxes with class,
# velocity and the ego state per frame.  Positions: a third of the objects in
# a forward corridor (x in [0, 45] m, |y| < 0.6 x + 2), the rest uniform in
# [-60, 60]^2; classes 30% vulnerable road users (0.8 x 0.8 m, speed U[0, 2]
# m/s, any heading), 50% motorized (4.5 x 1.9 m +-10%, speed U[0, 15] m/s,
# heading along +-x within 20 degrees; a quarter head-on towards the ego),
# 20% static (0.5 x 0.5 m, at rest).  Ego speed U[0, 35] m/s, yaw rate U[-0.3,
# 0.3] rad/s over dt; the frame-to-frame motion moves points back by the
# distance driven.

DETECTION_DTYPE = np.dtype([("x", "<f8"), ("y", "<f8"), ("yaw", "<f8"), ("length", "<f8"), ("width", "<f8"),
                            ("vx", "<f8"), ("vy", "<f8"), ("cls", "<i4"), ("reserved", "<i4")])
EGO_DTYPE = np.dtype([("speed", "<f8"), ("dx", "<f8"), ("dy", "<f8"), ("dyaw", "<f8")])


def detections(seed: int, frames: int, count=(0, 300), dt: float = 0.5, speed=(0.0, 35.0)):
    """Seeded detection caches: (dets [D] DETECTION_DTYPE, det_offsets int32
    [frames+1], ego [frames] EGO_DTYPE).  count: (lo, hi) detections per frame,
    or a list of exact counts."""
    rng = np.random.default_rng(seed)
    counts = list(count) if isinstance(count, list) else [int(rng.integers(count[0], count[1] + 1))
                                                           for _ in range(frames)]
    D = int(sum(counts))
    d = np.zeros(D, dtype=DETECTION_DTYPE)
    corridor = rng.random(D) < 1 / 3
    x = np.where(corridor, rng.uniform(0, 45, D), rng.uniform(-60, 60, D))
    y = np.where(corridor, rng.uniform(-1, 1, D) * (0.6 * x + 2), rng.uniform(-60, 60, D))
    u = rng.random(D)
    cls = np.where(u < 0.3, 0, np.where(u < 0.8, 1, 2)).astype(np.int32)
    heading = np.where(cls == 0, rng.uniform(-np.pi, np.pi, D),
                       rng.uniform(-0.35, 0.35, D) + np.where(rng.random(D) < 0.25, np.pi, 0.0))
    sp = np.where(cls == 0, rng.uniform(0, 2, D), np.where(cls == 1, rng.uniform(0, 15, D), 0.0))
    d["x"], d["y"] = x, y
    d["yaw"] = np.where(cls == 2, rng.uniform(-np.pi, np.pi, D), heading)
    d["length"] = np.where(cls == 0, 0.8, np.where(cls == 1, 4.5 * rng.uniform(0.9, 1.1, D), 0.5))
    d["width"] = np.where(cls == 0, 0.8, np.where(cls == 1, 1.9 * rng.uniform(0.9, 1.1, D), 0.5))
    d["vx"], d["vy"] = sp * np.cos(heading), sp * np.sin(heading)
    d["cls"] = cls
    off = np.zeros(frames + 1, dtype=np.int32)
    off[1:] = np.cumsum(counts)
    ego = np.zeros(frames, dtype=EGO_DTYPE)
    ego["speed"] = rng.uniform(speed[0], speed[1], frames)
    ego["dyaw"] = rng.uniform(-0.3, 0.3, frames) * dt
    ego["dx"] = -ego["speed"] * dt * np.cos(ego["dyaw"])
    ego["dy"] = -ego["speed"] * dt * np.sin(ego["dyaw"])
    return d, off, ego
