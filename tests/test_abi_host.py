"""The C ABI without a GPU: exported symbols, host helpers, argument checks.

Nothing here launches a kernel: every call tested returns before the library
touches the HIP runtime.
"""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mmbev.h")
LIB = os.path.join(ROOT, "paper_2608_15437_amd", "libmmbev.so")


@pytest.fixture(scope="module")
def mb():
    if not os.path.exists(LIB):
        import __graft_entry__ as ge

        ge.build()
    from paper_2608_15437_amd import mmbev

    mmbev.load()
    return mmbev


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mmbev_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_path():
    names = declared_functions()
    for n in ["mmbev_roi_voxelize", "mmbev_roi_voxelize_ex", "mmbev_scatter_to_bev", "mmbev_voxel_clusters",
              "mmbev_build_rois",
              "mmbev_voxel_clusters_workspace_bytes",
              "mmbev_roi_voxelize_workspace_bytes", "mmbev_make_rois",
              "mmbev_workspace_init", "mmbev_abi_version", "mmbev_status_string"]:
        assert n in names


def test_library_exports_every_declared_symbol(mb):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (mmbev_\w+)", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, f"not exported: {missing}"
    lib = ctypes.CDLL(LIB)
    for n in declared_functions():
        getattr(lib, n)


def test_struct_layouts_match_header(mb):
    assert ctypes.sizeof(mb.mmbev_points_t) == 40
    assert ctypes.sizeof(mb.mmbev_rois_t) == 24
    assert ctypes.sizeof(mb.mmbev_grid_t) == 52
    assert ctypes.sizeof(mb.mmbev_options_t) == 16
    assert mb.ROI_DTYPE.itemsize == 32
    assert mb.abi_version() == 7
    assert ctypes.sizeof(mb.mmbev_policy_t) == 136
    assert mb.DETECTION_DTYPE.itemsize == 64 and mb.EGO_DTYPE.itemsize == 32 and mb.CRIT_DTYPE.itemsize == 16
    assert ctypes.sizeof(mb.mmbev_cluster_params_t) == 24
    assert mb.CLUSTER_DTYPE.itemsize == 56


def test_make_rois_matches_oracle_bitwise(mb):
    rng = np.random.default_rng(0)
    desc = np.column_stack([rng.uniform(-60, 60, 300), rng.uniform(-60, 60, 300), rng.uniform(0.5, 10, 300),
                            rng.uniform(0.5, 5, 300), rng.uniform(-7, 7, 300), rng.uniform(0, 1, 300)])
    a = mb.make_rois(desc).view(np.uint32).reshape(-1, 8)[:, :6]
    b = oracle.make_rois(desc).view(np.uint32).reshape(-1, 8)[:, :6]
    assert np.array_equal(a, b)


def test_workspace_bytes_validation(mb):
    g = mb.grid_params((-54, -54, -5), (0.075, 0.075, 0.2), (1440, 1440, 40), 10, 120000, 10, 1)
    n = mb.roi_voxelize_workspace_bytes(g, 347200, 5, 32)
    assert n > 347200 * 24
    assert n % 256 == 0
    assert mb.roi_voxelize_workspace_bytes(g, 347200 * 2, 5, 32) > n
    bad = [dict(max_points=0), dict(max_points=65), dict(max_voxels=0), dict(num_sweeps=0), dict(num_sweeps=256),
           dict(num_frames=0), dict(dims=(0, 10, 10)), dict(voxel_size=(0.0, 1, 1)),
           dict(voxel_size=(float("nan"), 1, 1)), dict(dims=(70000, 70000, 2))]
    base = dict(range_min=(-54, -54, -5), voxel_size=(0.075, 0.075, 0.2), dims=(1440, 1440, 40), max_points=10,
                max_voxels=120000, num_sweeps=10, num_frames=1)
    for b in bad:
        gg = mb.grid_params(**{**base, **b})
        assert mb.roi_voxelize_workspace_bytes(gg, 1000, 5, 32) == 0, b
    assert mb.roi_voxelize_workspace_bytes(g, 1 << 30, 5, 32) == 0
    assert mb.roi_voxelize_workspace_bytes(g, 1000, 5, 1025) == 0
    assert mb.roi_voxelize_workspace_bytes(g, -1, 5, 32) == 0
    assert mb.roi_voxelize_workspace_bytes(g, 1000, 2, 32) == 0
    assert mb.roi_voxelize_workspace_bytes(g, 1000, 9, 32) == 0
    # one record column per feature
    assert mb.roi_voxelize_workspace_bytes(g, 347200, 8, 32) > mb.roi_voxelize_workspace_bytes(g, 347200, 3, 32)


def test_voxelize_rejects_bad_arguments_before_any_launch(mb):
    L = mb.load()
    g = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (16, 16, 4), 2, 3, 2, 1)
    fake = 1 << 40  # never dereferenced: validation fails first
    pts = mb.mmbev_points_t(feat=fake, stride=100, num_features=4, reserved=0, num_points=100, frame_offsets=fake)
    rr = mb.mmbev_rois_t(boxes=fake, frame_offsets=fake, num_rois=2, max_rois_per_frame=2)
    ws_need = mb.roi_voxelize_workspace_bytes(g, 100, 4, 2)

    def call(points=pts, rois=rr, grid=g, sweep=fake, poses=fake, budget=fake, outs=(fake,) * 5, ws=fake,
             ws_bytes=ws_need):
        return L.mmbev_roi_voxelize(ctypes.byref(points), sweep, poses, ctypes.byref(rois), budget,
                                    ctypes.byref(grid), *outs, ws, ws_bytes, None)

    assert call(ws_bytes=ws_need - 1) == mb.ERR_WORKSPACE
    assert call(ws=fake + 8) == mb.ERR_WORKSPACE
    assert call(ws=None) == mb.ERR_WORKSPACE
    assert call(sweep=None) == mb.ERR_INVALID_ARG
    assert call(poses=None) == mb.ERR_INVALID_ARG
    assert call(budget=None) == mb.ERR_INVALID_ARG
    assert call(outs=(fake, fake, None, fake, fake)) == mb.ERR_INVALID_ARG
    bad_c = mb.mmbev_points_t(feat=fake, stride=100, num_features=9, reserved=0, num_points=100,
                              frame_offsets=fake)
    assert call(points=bad_c) == mb.ERR_INVALID_ARG
    bad_stride = mb.mmbev_points_t(feat=fake, stride=99, num_features=4, reserved=0, num_points=100,
                                   frame_offsets=fake)
    assert call(points=bad_stride) == mb.ERR_INVALID_ARG
    too_many = mb.mmbev_rois_t(boxes=fake, frame_offsets=fake, num_rois=2, max_rois_per_frame=2000)
    assert call(rois=too_many) == mb.ERR_UNSUPPORTED
    assert mb.load().mmbev_status_string(mb.ERR_HIP) == b"HIP launch failed"


def test_options_reserved_field_must_be_zero(mb):
    L = mb.load()
    g = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (16, 16, 4), 2, 3, 2, 1)
    fake = 1 << 40  # never dereferenced: validation fails first
    pts = mb.mmbev_points_t(feat=fake, stride=100, num_features=4, reserved=0, num_points=100, frame_offsets=fake)
    rr = mb.mmbev_rois_t(boxes=fake, frame_offsets=fake, num_rois=2, max_rois_per_frame=2)
    ws_need = mb.roi_voxelize_workspace_bytes(g, 100, 4, 2)
    used = ctypes.c_int32(0)

    def call(opt, ws_bytes=ws_need):
        return L.mmbev_roi_voxelize_ex(ctypes.byref(pts), fake, fake, ctypes.byref(rr), fake, ctypes.byref(g),
                                       ctypes.byref(opt), *(fake,) * 5, fake, ws_bytes, None, None, 0,
                                       ctypes.byref(used))

    assert call(mb.mmbev_options_t(out_of_roi_keep_rate=0.5, reserved=1, seed=3)) == mb.ERR_INVALID_ARG
    # a valid options block reaches the workspace check
    assert call(mb.mmbev_options_t(out_of_roi_keep_rate=0.5, reserved=0, seed=3), ws_need - 1) == mb.ERR_WORKSPACE


def test_scatter_to_bev_rejects_bad_arguments_before_any_launch(mb):
    L = mb.load()
    g = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (16, 16, 4), 2, 3, 2, 1)
    fake = 1 << 40  # never dereferenced: validation fails first

    def call(coords=fake, feats=fake, voff=fake, C=5, grid=g, out=fake):
        return L.mmbev_scatter_to_bev(coords, feats, voff, C, ctypes.byref(grid), out, None, None)

    assert call(coords=None) == mb.ERR_INVALID_ARG
    assert call(feats=None) == mb.ERR_INVALID_ARG
    assert call(voff=None) == mb.ERR_INVALID_ARG
    assert call(out=None) == mb.ERR_INVALID_ARG
    assert call(coords=fake + 4) == mb.ERR_INVALID_ARG  # int4 rows need 16-byte alignment
    assert call(C=0) == mb.ERR_INVALID_ARG
    assert call(C=65) == mb.ERR_INVALID_ARG
    bad = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (16, 0, 4), 2, 3, 2, 1)
    assert call(grid=bad) == mb.ERR_INVALID_ARG
    huge = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (1 << 16, 1 << 16, 2), 2, 3, 2, 1)
    assert call(grid=huge) == mb.ERR_UNSUPPORTED


def test_voxel_clusters_validation(mb):
    L = mb.load()
    g = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (16, 16, 4), 2, 3, 2, 2)
    prm = mb.cluster_params(1, 3, 0, 8, 1)
    need = mb.voxel_clusters_workspace_bytes(g, prm)
    assert need > 0
    for bad in (mb.cluster_params(1, 3, 0, 6, 1), mb.cluster_params(1, 3, 9, 8, 1), mb.cluster_params(1, 3, 0, 8, 0)):
        assert mb.voxel_clusters_workspace_bytes(g, bad) == 0
    r = mb.cluster_params(1, 3, 0, 8, 1)
    r.reserved = 1
    assert mb.voxel_clusters_workspace_bytes(g, r) == 0
    big = mb.grid_params((-4, -4, -1), (0.5, 0.5, 0.5), (1 << 15, 1 << 15, 1), 2, 3, 2, 1)
    assert mb.voxel_clusters_workspace_bytes(big, prm) == 0  # 2^30 cells
    assert mb.voxel_clusters_workspace_bytes(big, mb.cluster_params(0, 1, 1, 8, 1)) > 0  # 2^28 cells
    fake = 1 << 40

    def call(coords=fake, out=fake, ws=fake, ws_bytes=need, params=prm):
        return L.mmbev_voxel_clusters(coords, fake, fake, ctypes.byref(g), ctypes.byref(params), out, fake, fake,
                                      ws, ws_bytes, None)

    assert call(coords=None) == mb.ERR_INVALID_ARG
    assert call(coords=fake + 4) == mb.ERR_INVALID_ARG
    assert call(out=fake + 4) == mb.ERR_INVALID_ARG
    assert call(ws=None) == mb.ERR_WORKSPACE
    assert call(ws=fake + 128) == mb.ERR_WORKSPACE
    assert call(ws_bytes=need - 1) == mb.ERR_WORKSPACE
    assert call(params=mb.cluster_params(1, 3, 0, 5, 1)) == mb.ERR_INVALID_ARG


def test_noalloc_rejects_before_any_launch(mb):
    """The no-alloc entry point checks its arguments, and that the sizes fit
    its fixed scratch, before it touches the device."""
    L = mb.load()
    fake = 1 << 40  # never dereferenced: validation fails first
    g = mb.grid_params((-54, -54, -5), (0.075, 0.075, 0.2), (1440, 1440, 40), 10, 120000, 10, 1)
    limit = 64 << 20

    def call(n, sweep=fake, outs=(fake,) * 5):
        pts = mb.mmbev_points_t(feat=fake, stride=n, num_features=5, reserved=0, num_points=n, frame_offsets=fake)
        rr = mb.mmbev_rois_t(boxes=fake, frame_offsets=fake, num_rois=32, max_rois_per_frame=32)
        return L.mmbev_roi_voxelize_noalloc(ctypes.byref(pts), sweep, fake, ctypes.byref(rr), fake,
                                            ctypes.byref(g), *outs, None, None)

    big = 2_000_000
    assert mb.roi_voxelize_workspace_bytes(g, big, 5, 32) > limit
    assert mb.roi_voxelize_workspace_bytes(g, 347200, 5, 32) <= limit
    assert call(big) == mb.ERR_UNSUPPORTED
    assert call(347200, sweep=None) == mb.ERR_INVALID_ARG
    assert call(347200, outs=(fake, fake, None, fake, fake)) == mb.ERR_INVALID_ARG
