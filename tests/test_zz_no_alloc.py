"""mmbev_roi_voxelize_noalloc (the library's own per-device scratch as the
workspace) against mmbev_roi_voxelize with a caller-allocated workspace, on
two calls in a row, the second with a smaller input: structure bit for bit,
features within 1e-5, rows past the voxel count untouched, fault word 0.
Both are also checked against the oracle."""
import numpy as np
import pytest

import synth
from common import assert_same_voxels

pytestmark = pytest.mark.gpu
FEAT_TOL = 1e-5


def _noalloc_outputs(mb, vz):
    """Run the no-alloc entry point on vz's inputs into fresh canary-filled outputs."""
    import torch

    g = vz.grid
    rows = g.num_frames * g.max_voxels
    C, M = int(vz.feat.shape[0]), g.max_points
    out = {"coords": torch.full((rows, 4), -7, dtype=torch.int32, device=vz.device),
           "counts": torch.full((rows,), -7, dtype=torch.int32, device=vz.device),
           "feats": torch.full((rows, C), -7.0, dtype=torch.float32, device=vz.device),
           "point_idx": torch.full((rows, M), -7, dtype=torch.int32, device=vz.device),
           "voxel_offsets": torch.zeros(g.num_frames + 1, dtype=torch.int64, device=vz.device)}
    fault = torch.full((1,), -1, dtype=torch.int32, device=vz.device)
    mb.roi_voxelize_noalloc(vz.feat, vz.frame_offsets, vz.sweep_ids, vz.sweep_poses, vz.rois, vz.roi_frame_offsets,
                            vz.roi_sweep_budget, g, out["coords"], out["counts"], out["feats"], out["point_idx"],
                            out["voxel_offsets"], vz.max_rois, out_fault=fault)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, int(fault.item())


@pytest.mark.parametrize("first,second", [("c2", "small")])
def test_noalloc_matches_workspace_call_twice(gpu_lib, first, second):
    import oracle

    workloads = [synth.c2(), synth.small(71, frames=3, max_voxels=40, max_points=3)]
    assert workloads[1].num_points < workloads[0].num_points
    for wl in workloads:
        print(f"[noalloc] {wl.name}: {wl.num_points} points, {wl.num_frames} frames", flush=True)
        vz = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
        vz.run()
        ref = vz.result()
        assert vz.fault() == 0
        got, fault = _noalloc_outputs(gpu_lib, vz)
        assert fault == 0, f"{wl.name}: fault word {fault}"
        V = int(ref["voxel_offsets"][-1])
        assert V > 0
        assert_same_voxels(got, ref, feat_atol=FEAT_TOL, label=f"noalloc {wl.name}")
        # the same kernels: the means agree bit for bit as well
        assert np.array_equal(got["feats"][:V].view(np.uint32), ref["feats"][:V].view(np.uint32))
        for name in ("coords", "counts", "feats", "point_idx"):
            rest = got[name][V:]
            assert np.all(rest == -7), f"{wl.name}: rows past V of {name} were written"
        assert_same_voxels(got, oracle.run_workload(wl), feat_atol=FEAT_TOL, label=f"noalloc {wl.name} vs oracle")
