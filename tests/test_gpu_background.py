"""Parity of the out-of-ROI keep rate (Alg. 1, rho_out) on the HIP path.

Points outside every ROI (or whose sweep no ROI admits) are kept when their
SplitMix64 draw lies below round(rho_out * 2^24); both sides draw from the
same published generator, seeded by the caller, so the kept set, and with it
every output, must match the oracle bit for bit.
"""
import numpy as np
import pytest

import synth
from common import case_from_workload
from test_gpu_parity import check, run_gpu

pytestmark = pytest.mark.gpu

SEED_HI = 0xF00DFACE12345678


@pytest.mark.parametrize("name", ["c1", "c2", "c4", "c5"])
@pytest.mark.parametrize("rho,seed", [(0.05, 7), (0.5, SEED_HI), (1.0, 0)])
def test_configs_with_background(gpu_lib, name, rho, seed):
    wl = synth.CONFIGS[name]()
    case = case_from_workload(wl)
    vz, exp = check(gpu_lib, case, label=f"{name} rho={rho}", desc=wl.roi_desc, rho_out=rho, seed=seed)
    keys, _ = case.oracle_keep(rho, seed)
    assert vz.header()["kept"] == len(keys)


@pytest.mark.parametrize("seed,frames,cap,M,rho", [
    (11, 1, 1000, 4, 0.3), (12, 3, 20, 2, 0.9), (13, 5, 1, 8, 0.02), (14, 2, 400, 64, 0.6),
    (15, 4, 9, 3, 1e-7)])
def test_small_scenes_with_background(gpu_lib, seed, frames, cap, M, rho):
    wl = synth.small(seed, frames=frames, max_voxels=cap, max_points=M)
    check(gpu_lib, case_from_workload(wl), label=f"small{seed}", desc=wl.roi_desc, rho_out=rho,
          seed=(1 << 64) - seed)


def test_background_without_rois(gpu_lib):
    """No ROI anywhere: only the draw keeps points."""
    wl = synth.small(16, frames=3, max_voxels=10 ** 5, max_points=16)
    case = case_from_workload(wl)
    B = case.B
    case.rois = case.rois[:0]
    case.budgets = case.budgets[:0]
    case.roi_offsets = np.zeros(B + 1, dtype=np.int32)
    vz, exp = check(gpu_lib, case, label="no rois", rho_out=0.25, seed=99)
    assert int(exp["voxel_offsets"][-1]) > 0


def test_rate_zero_options_match_plain_entry_point(gpu_lib):
    """rho_out = 0 through the options block (a nonzero seed selects it) is the plain call."""
    wl = synth.small(17, frames=2)
    case = case_from_workload(wl)
    rois = gpu_lib.make_rois(wl.roi_desc)
    a = run_gpu(gpu_lib, case, gpu_rois=rois).result()
    for rho in (0.0, -1.0, float("nan")):
        b = run_gpu(gpu_lib, case, gpu_rois=rois, rho_out=rho, seed=5).result()
        for k in a:
            assert np.array_equal(a[k], b[k]), (rho, k)


def test_throughput_batch_with_background(gpu_lib):
    """The benchmark's batched workload at 16 frames with a 10% background rate."""
    wl = synth.throughput(16)
    check(gpu_lib, case_from_workload(wl), label="c2x16 rho=0.1", desc=wl.roi_desc, rho_out=0.1, seed=2024)
