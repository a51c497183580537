"""The temporal-ROI selector feeding the voxelisation: the library's
mmbev_build_rois output drives the HIP path, the oracle's selector output
drives the oracle path, and the voxels must match bit for bit (features
within the path's stated tolerance)."""
import pytest

import synth
from common import Case, assert_same_voxels, case_from_workload
from oracle import policy as P
from test_gpu_parity import FEAT_TOL, run_gpu
from test_oracle_policy import POL, as_dicts

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,seed,count,kw", [
    ("c2", 1, (20, 80), {}),
    ("c5", 2, (0, 150), {"max_optional": 20}),
    ("c4", 3, (40, 60), {"dt": 0.1, "n_full": 3, "n_reduced": 2}),
])
def test_selector_then_voxelize(gpu_lib, name, seed, count, kw):
    wl = synth.CONFIGS[name]()
    pol = dict(POL, **kw)
    d, off, e = synth.detections(seed, wl.num_frames, count=count)
    sel = gpu_lib.build_rois(d, off, e, gpu_lib.policy(**pol))
    ref = P.build_rois(*as_dicts(d, off, e), pol)
    base = case_from_workload(wl)
    gpu_case = Case(**{**base.__dict__, "rois": sel["rois"], "roi_offsets": sel["roi_offsets"],
                       "budgets": sel["budgets"]})
    ora_case = Case(**{**base.__dict__, "rois": ref["rois"], "roi_offsets": ref["roi_offsets"],
                       "budgets": ref["budgets"]})
    exp = ora_case.run_oracle()
    vz = run_gpu(gpu_lib, gpu_case)
    assert vz.fault() == 0
    assert_same_voxels(vz.result(), exp, feat_atol=FEAT_TOL, label=name)
    assert int(exp["voxel_offsets"][-1]) > 0
