"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each step of the oracle (Eq. 6 compensation, the Alg. 1 keep test against the
Eq. 1 ROI union, quantisation, grouping, caps, means) is checked against
something other than itself: a hand-derived worked example, closed forms on
exactly representable inputs, a float64 re-derivation, brute-force grouping
with Python dicts, a library special case (torch.unique), the physical
ghost-collapse property of motion compensation, and metamorphic invariants.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from common import (Case, assert_same_voxels, case_from_workload, dict_voxelize, f64_keep, key_of,
                    load_golden, records)

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

IDENT = np.array([1, 0, 0, 0, 0, 1, 0, 0, 0, 0, 1, 0], dtype=np.float32)


# ------------------------------------------------------------------ golden
def test_golden_hand_two_frames():
    case, exp = load_golden("hand_two_frames.json")
    got = case.run_oracle()
    assert_same_voxels(got, exp, feat_atol=0.0, label="golden")
    _, idx = case.oracle_keep()
    assert idx.tolist() == exp["kept_before_caps"]


# ------------------------------------------------------ Eq. 6 compensation
def test_compensate_identity_is_exact():
    rng = np.random.default_rng(0)
    pts = rng.normal(0, 40, size=(500, 3)).astype(np.float32)
    for p in pts:
        out = oracle.compensate(IDENT, *p)
        assert np.array_equal(out, p)


def test_compensate_dyadic_translation_exact():
    pose = IDENT.copy()
    pose[[3, 7, 11]] = [1.5, -2.25, 0.125]
    rng = np.random.default_rng(1)
    pts = (rng.integers(-4096, 4096, size=(300, 3)) / 256.0).astype(np.float32)
    for p in pts:
        out = oracle.compensate(pose, *p)
        assert np.array_equal(out, p + np.array([1.5, -2.25, 0.125], dtype=np.float32))


@pytest.mark.parametrize("yaw_deg", [90, 180, 270])
def test_compensate_rotation_closed_form(yaw_deg):
    # R = Rz(yaw): a point on the sweep's x axis lands at (cos yaw, sin yaw) in the current frame
    c, s = {90: (0, 1), 180: (-1, 0), 270: (0, -1)}[yaw_deg]
    pose = np.array([c, -s, 0, 0.5, s, c, 0, -0.75, 0, 0, 1, 2.0], dtype=np.float32)
    rng = np.random.default_rng(yaw_deg)
    pts = (rng.integers(-2048, 2048, size=(200, 3)) / 64.0).astype(np.float32)
    for x, y, z in pts:
        out = oracle.compensate(pose, x, y, z)
        exp = np.array([c * x - s * y + 0.5, s * x + c * y - 0.75, z + 2.0], dtype=np.float32)
        assert np.array_equal(out, exp)


def test_compensate_general_pose_vs_float64():
    rng = np.random.default_rng(7)
    for _ in range(50):
        a, b, g = rng.uniform(-math.pi, math.pi, 3)
        Rz = np.array([[math.cos(a), -math.sin(a), 0], [math.sin(a), math.cos(a), 0], [0, 0, 1]])
        Ry = np.array([[math.cos(b), 0, math.sin(b)], [0, 1, 0], [-math.sin(b), 0, math.cos(b)]])
        Rx = np.array([[1, 0, 0], [0, math.cos(g), -math.sin(g)], [0, math.sin(g), math.cos(g)]])
        R = Rz @ Ry @ Rx
        T = rng.uniform(-5, 5, 3)
        pose = np.concatenate([R, T[:, None]], axis=1).astype(np.float32).reshape(12)
        P = pose.astype(np.float64).reshape(3, 4)
        for p in rng.uniform(-60, 60, size=(20, 3)).astype(np.float32):
            out = oracle.compensate(pose, *p)
            exp = P[:, :3] @ p.astype(np.float64) + P[:, 3]
            assert np.max(np.abs(out - exp)) < 2e-5


def test_motion_compensation_collapses_ghosts():
    """Static structure seen from a moving ego lands on one place after Eq. 6.

    One static box, ego at 10 m/s turning at 0.2 rad/s, 10 sweeps 0.05 s
    apart: uncompensated, the box's returns from sweep s sit about 0.5 s metres
    away from it; compensated, every above-ground return lies on its surface.
    """
    scene = synth._scene32(10, 1085, 1, False, 5, speed=(10.0, 10.0))
    scene.yawrate_lo = scene.yawrate_hi = 0.2
    scene.obs_r_lo, scene.obs_r_hi = 8.0, 12.0
    wl = synth._build("ghost", scene, synth._recipe(on=1, margin=0.5, budget=(10, 10)), [5],
                      synth._grid(54.0, -5.0, 3.0, 0.1, 0.2, (1080, 1080, 40), 10, 100000, 10, 1))
    box = wl.obstacles[0][0]
    cx, cy, cz, L, W, H, yaw = box

    def surface_distance(p):
        dx, dy = p[:, 0] - cx, p[:, 1] - cy
        lx = math.cos(yaw) * dx + math.sin(yaw) * dy
        ly = -math.sin(yaw) * dx + math.cos(yaw) * dy
        lz = p[:, 2] - cz
        q = np.abs(np.stack([lx, ly, lz], 1)) - np.array([L / 2, W / 2, H / 2])
        outside = np.linalg.norm(np.maximum(q, 0), axis=1)
        inside = np.minimum(np.max(q, axis=1), 0)
        return np.abs(outside + inside)

    per = 32 * 1085
    for s in range(10):
        sl = slice(s * per, (s + 1) * per)
        raw = wl.feat[:3, sl].T
        # above-ground returns closer than 25 m can only come from the box
        raw = raw[(raw[:, 2] > 0.3) & (np.hypot(raw[:, 0], raw[:, 1]) < 25.0)]
        comp = np.stack([oracle.compensate(wl.poses[0, s], *p) for p in raw])
        assert len(comp) > 50, "box not visible"
        assert np.quantile(surface_distance(comp.astype(np.float64)), 0.99) < 0.1, f"sweep {s} not collapsed"
        if s >= 2:
            uncomp = raw.astype(np.float64)
            assert np.median(surface_distance(uncomp)) > 0.3, "test would not detect a missing compensation"


# ----------------------------------------------------------- ROI keep test
def test_make_roi_closed_form():
    r = oracle.make_rois([[1.5, -2.0, 4.5, 1.9, 0.0, 0.5]])[0]
    assert (r["cx"], r["cy"], r["cos_yaw"], r["sin_yaw"]) == (np.float32(1.5), np.float32(-2.0), 1.0, 0.0)
    assert r["ext_x"] == np.float32(2.25 + 0.5) and r["ext_y"] == np.float32(0.95 + 0.5)
    r = oracle.make_rois([[0.0, 0.0, 2.0, 2.0, math.pi / 2, 0.0]])[0]
    assert abs(float(r["cos_yaw"])) < 1e-7 and r["sin_yaw"] == 1.0


def test_inside_axis_aligned_edges_inclusive():
    roi = records([[2.0, 3.0, 1.0, 0.0, 1.5, 0.75]])[0]
    e = 2.0 ** -10
    assert oracle.inside(roi, 3.5, 3.0) and oracle.inside(roi, 0.5, 3.0)
    assert oracle.inside(roi, 2.0, 3.75) and oracle.inside(roi, 2.0, 2.25)
    assert oracle.inside(roi, 3.5, 3.75) and oracle.inside(roi, 0.5, 2.25)
    assert not oracle.inside(roi, 3.5 + e, 3.0) and not oracle.inside(roi, 0.5 - e, 3.0)
    assert not oracle.inside(roi, 2.0, 3.75 + e) and not oracle.inside(roi, 2.0, 2.25 - e)


def test_inside_rot90_swaps_axes():
    # yaw +90 deg: the box's length runs along world y
    roi = records([[0.0, 0.0, 0.0, 1.0, 2.0, 0.5]])[0]
    assert oracle.inside(roi, 0.0, 2.0) and oracle.inside(roi, 0.0, -2.0)
    assert oracle.inside(roi, 0.5, 0.0) and oracle.inside(roi, -0.5, 0.0)
    assert not oracle.inside(roi, 2.0, 0.0) and not oracle.inside(roi, 1.0, 0.0)
    assert not oracle.inside(roi, 0.0, 2.0 + 2.0 ** -10)
    assert not oracle.inside(roi, 0.5 + 2.0 ** -10, 0.0)


def test_inside_random_vs_float64():
    rng = np.random.default_rng(3)
    desc = np.column_stack([rng.uniform(-20, 20, 40), rng.uniform(-20, 20, 40), rng.uniform(1, 8, 40),
                            rng.uniform(1, 4, 40), rng.uniform(0, 2 * math.pi, 40), rng.uniform(0, 1, 40)])
    rois = oracle.make_rois(desc)
    pts = rng.uniform(-25, 25, size=(400, 2)).astype(np.float32)
    checked = 0
    for r in rois:
        c, s = float(r["cos_yaw"]), float(r["sin_yaw"])
        for x, y in pts:
            dx, dy = float(x) - float(r["cx"]), float(y) - float(r["cy"])
            lx, ly = c * dx + s * dy, c * dy - s * dx
            slack = min(float(r["ext_x"]) - abs(lx), float(r["ext_y"]) - abs(ly))
            if abs(slack) < 1e-4:
                continue
            assert oracle.inside(r, x, y) == (slack >= 0)
            checked += 1
    assert checked > 15000


# --------------------------------------------------------------- quantise
def test_quantize_faces_and_range():
    g = oracle.make_grid((-4, -4, -1), (0.25, 0.25, 0.5), (32, 32, 4), 4, 100, 1, 1)
    e = 2.0 ** -12
    assert oracle.quantize(g, (-4, -4, -1)) == (0, 0, 0)
    assert oracle.quantize(g, (-4 + 5 * 0.25, -4 + 31 * 0.25, -1 + 3 * 0.5)) == (5, 31, 3)
    assert oracle.quantize(g, (-4 + 5 * 0.25 - e, -4 + 7 * 0.25 - e, 0.0 - e)) == (4, 6, 1)
    assert oracle.quantize(g, (4.0, 0.0, 0.0)) is None
    assert oracle.quantize(g, (0.0, 4.0, 0.0)) is None
    assert oracle.quantize(g, (0.0, 0.0, 1.0)) is None
    assert oracle.quantize(g, (4.0 - e, 4.0 - e, 1.0 - e)) == (31, 31, 3)
    assert oracle.quantize(g, (-4.0 - e, 0.0, 0.0)) is None
    for bad in (np.nan, np.inf, -np.inf):
        assert oracle.quantize(g, (bad, 0.0, 0.0)) is None
        assert oracle.quantize(g, (0.0, 0.0, bad)) is None


def test_nonfinite_points_are_dropped():
    case, _ = load_golden("hand_two_frames.json")
    ref = case.run_oracle()
    feat = case.feat.copy()
    # point 4 was dropped anyway; make points 4 and 10 non-finite: nothing changes
    feat[0, 4], feat[2, 10] = np.nan, np.inf
    case2 = Case(**{**case.__dict__, "feat": feat})
    assert_same_voxels(case2.run_oracle(), ref, feat_atol=0.0)


# --------------------------------------------- keep test vs float64 (whole)
@pytest.mark.parametrize("make", [lambda: synth.c1(), lambda: synth.c2(), lambda: synth.small(5),
                                  lambda: synth.small(9, frames=3, budget=(0, 3))])
def test_keep_matches_float64(make):
    wl = make()
    case = case_from_workload(wl)
    keep64, ijk64, amb, _ = f64_keep(case)
    keys, idx = case.oracle_keep()
    keep32 = np.zeros(wl.num_points, dtype=bool)
    keep32[idx] = True
    clear = ~amb
    assert np.array_equal(keep32[clear], keep64[clear])
    fo = case.frame_offsets
    frame = np.searchsorted(fo, idx, side="right") - 1
    for k, i, b in zip(keys, idx, frame):
        if not amb[i]:
            assert int(k) == key_of(int(b), ijk64[i], case.grid["dims"])
    assert keep64.sum() > 0


# ----------------------------------------------- grouping/caps/means brute
@pytest.mark.parametrize("seed,cap,M", [(1, 1000, 4), (2, 25, 2), (4, 7, 1), (6, 1, 3)])
def test_pipeline_matches_dict_bruteforce(seed, cap, M):
    wl = synth.small(seed, frames=3, max_voxels=cap, max_points=M)
    case = case_from_workload(wl)
    keep64, ijk64, amb, p64 = f64_keep(case)
    # where float64 is unambiguous it decides; elsewhere the (separately pinned) fp32 steps do
    keys32, idx32 = case.oracle_keep()
    keep = keep64.copy()
    keep[amb] = False
    keep[idx32[amb[idx32]]] = True
    kept_idx = np.nonzero(keep)[0]
    fo = case.frame_offsets
    key_map = dict(zip(idx32.tolist(), keys32.tolist()))
    kept_key = []
    for i in kept_idx:
        b = int(np.searchsorted(fo, i, side="right") - 1)
        kept_key.append(key_map[int(i)] if amb[i] else key_of(b, ijk64[i], case.grid["dims"]))
    values = np.concatenate([p64, case.feat[3:].T.astype(np.float64)], axis=1)
    exp = dict_voxelize(case, kept_idx, kept_key, values)
    got = case.run_oracle()
    assert_same_voxels(got, exp, feat_atol=2e-5, label=f"seed {seed}")
    if cap < 1000:
        assert np.any(np.diff(got["voxel_offsets"]) == cap), "cap did not bind"


# ---------------------------------------------------- library special case
def test_all_covering_roi_equals_torch_unique():
    """One sweep, identity pose, one ROI covering everything, no cap binding:
    the path reduces to plain voxelisation, i.e. torch.unique over voxel keys
    plus a float64 index_add_ of the features."""
    torch = pytest.importorskip("torch")
    wl = synth.c1()
    case = case_from_workload(wl, rois=records([[0, 0, 1, 0, 1e4, 1e4]]))
    case.budgets = np.array([1], dtype=np.uint8)
    case.grid = dict(case.grid, max_points=64, max_voxels=10 ** 6)
    assert np.array_equal(case.poses[0, 0], IDENT)
    got = case.run_oracle()

    p = torch.from_numpy(case.feat[:3].T.copy())
    mn = torch.tensor(case.grid["range_min"], dtype=torch.float32)
    vs = torch.tensor(case.grid["voxel_size"], dtype=torch.float32)
    D = torch.tensor(case.grid["dims"], dtype=torch.float32)
    f = (p - mn) / vs
    ok = ((f >= 0) & (f < D)).all(dim=1)
    ijk = f[ok].to(torch.int64)
    Dx, Dy, _ = case.grid["dims"]
    keys = (ijk[:, 2] * Dy + ijk[:, 1]) * Dx + ijk[:, 0]
    uniq, inv, counts = torch.unique(keys, sorted=True, return_inverse=True, return_counts=True)
    assert int(counts.max()) <= 64
    vals = torch.from_numpy(case.feat.T.copy()).to(torch.float64)[ok]
    sums = torch.zeros(len(uniq), vals.shape[1], dtype=torch.float64).index_add_(0, inv, vals)
    means = (sums / counts[:, None].to(torch.float64)).to(torch.float32)
    assert np.array_equal(got["counts"], counts.numpy())
    exp_coords = np.stack([np.zeros(len(uniq)), (uniq // (Dx * Dy)).numpy(), ((uniq // Dx) % Dy).numpy(),
                           (uniq % Dx).numpy()], 1)
    assert np.array_equal(got["coords"], exp_coords)
    np.testing.assert_allclose(got["feats"], means.numpy(), rtol=0, atol=1e-5)
    order = torch.argsort(inv, stable=True)
    pid = torch.nonzero(ok).flatten()[order]
    starts = np.concatenate([[0], np.cumsum(counts.numpy())])
    for v in range(len(uniq)):
        row = pid[starts[v]:starts[v + 1]].numpy()
        assert np.array_equal(got["point_idx"][v, :len(row)], row)


# ---------------------------------------------------------- invariants
def _runs(case):
    keys, idx = case.oracle_keep()
    u, c = np.unique(keys, return_counts=True)
    return dict(zip(u.tolist(), c.tolist())), keys, idx


def test_invariants_c2():
    wl = synth.c2()
    case = case_from_workload(wl)
    out = case.run_oracle()
    runs, keys, idx = _runs(case)
    g = case.grid
    Dx, Dy, Dz = g["dims"]
    M = g["max_points"]
    vkeys = ((out["coords"][:, 0].astype(np.int64) * Dz + out["coords"][:, 1]) * Dy
             + out["coords"][:, 2]) * Dx + out["coords"][:, 3]
    assert np.all(np.diff(vkeys) > 0), "keys must strictly increase"
    assert len(vkeys) == len(runs) <= g["max_voxels"]
    assert int(out["counts"].sum()) == sum(min(r, M) for r in runs.values())
    assert np.array_equal(out["counts"], np.minimum([runs[k] for k in vkeys.tolist()], M))
    for row, cnt in zip(out["point_idx"], out["counts"]):
        assert np.all(np.diff(row[:cnt]) > 0) and np.all(row[cnt:] == -1)
    # every kept point lies in an ROI that admits its sweep (float64 check with slack)
    keep64, _, amb, _ = f64_keep(case)
    assert np.all(keep64[idx] | amb[idx])


def test_roi_order_does_not_matter():
    wl = synth.c2()
    case = case_from_workload(wl)
    ref = case.run_oracle()
    perm = np.random.default_rng(0).permutation(len(case.rois))
    case.rois, case.budgets = case.rois[perm], case.budgets[perm]
    assert_same_voxels(case.run_oracle(), ref, feat_atol=0.0)


def test_adding_rois_or_budget_never_removes_voxels():
    wl = synth.small(8, frames=2, max_voxels=10 ** 6)
    case = case_from_workload(wl)
    base = case.run_oracle()
    bigger = Case(**{**case.__dict__, "budgets": np.minimum(case.budgets.astype(int) + 1, 255).astype(np.uint8)})
    more = bigger.run_oracle()

    def keyset(o):
        return set(map(tuple, o["coords"].tolist()))

    assert keyset(base) <= keyset(more)
    assert len(keyset(more)) > len(keyset(base))


def test_frames_are_independent():
    wl = synth.small(11, frames=3, max_voxels=40)
    case = case_from_workload(wl)
    whole = case.run_oracle()
    for b in range(3):
        lo, hi = int(case.frame_offsets[b]), int(case.frame_offsets[b + 1])
        rlo, rhi = int(case.roi_offsets[b]), int(case.roi_offsets[b + 1])
        one = Case(feat=np.ascontiguousarray(case.feat[:, lo:hi]), sweep_ids=case.sweep_ids[lo:hi],
                   frame_offsets=np.array([0, hi - lo]), poses=case.poses[b:b + 1], rois=case.rois[rlo:rhi],
                   roi_offsets=np.array([0, rhi - rlo], dtype=np.int32), budgets=case.budgets[rlo:rhi],
                   grid=dict(case.grid, num_frames=1)).run_oracle()
        v0, v1 = whole["voxel_offsets"][b], whole["voxel_offsets"][b + 1]
        assert v1 - v0 == one["voxel_offsets"][1]
        assert np.array_equal(whole["coords"][v0:v1, 1:], one["coords"][:, 1:])
        assert np.all(whole["coords"][v0:v1, 0] == b)
        assert np.array_equal(whole["point_idx"][v0:v1], np.where(one["point_idx"] >= 0, one["point_idx"] + lo, -1))
        assert np.array_equal(whole["feats"][v0:v1], one["feats"])


def test_degenerate_inputs():
    case, _ = load_golden("hand_two_frames.json")
    # no ROI admits anything: empty output
    none = Case(**{**case.__dict__, "budgets": np.zeros_like(case.budgets)})
    out = none.run_oracle()
    assert out["voxel_offsets"].tolist() == [0, 0, 0]
    # empty ROI set in a frame
    empty = Case(**{**case.__dict__, "rois": case.rois[:2], "budgets": case.budgets[:2],
                    "roi_offsets": np.array([0, 2, 2], dtype=np.int32)})
    out = empty.run_oracle()
    assert out["voxel_offsets"][2] == out["voxel_offsets"][1]
    # sweep ids beyond num_sweeps are dropped
    bad = Case(**{**case.__dict__, "sweep_ids": np.full_like(case.sweep_ids, 7)})
    assert bad.run_oracle()["voxel_offsets"].tolist() == [0, 0, 0]
    # zero points
    z = Case(feat=np.zeros((4, 0), np.float32), sweep_ids=np.zeros(0, np.uint8),
             frame_offsets=np.array([0, 0, 0]), poses=case.poses, rois=case.rois, roi_offsets=case.roi_offsets,
             budgets=case.budgets, grid=case.grid)
    assert z.run_oracle()["voxel_offsets"].tolist() == [0, 0, 0]
