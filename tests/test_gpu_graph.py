"""One call of the path captured in a HIP graph and replayed.

The entry point only enqueues kernels on the caller's stream (no allocation,
no host synchronisation, no memset), so a caller can capture it.  The graph
is replayed several times with the program's own eager work (output
scribbles, eager calls, synchronisations) between the replays, and every
replay's outputs must equal the eager call's bit for bit."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu


def _snapshot(vz):
    r = vz.result()
    return {k: np.array(v, copy=True) for k, v in r.items()}


@pytest.mark.parametrize("name", ["small", "c2"])
def test_call_replays_as_a_graph(gpu_lib, name):
    import torch

    wl = synth.small(61, frames=3) if name == "small" else synth.c2()
    vz = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
    vz.run()
    torch.cuda.synchronize()
    ref = _snapshot(vz)
    assert ref["voxel_offsets"][-1] > 0

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        vz.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        vz.run()
    torch.cuda.synchronize()

    for rep in range(3):
        vz.out_coords.fill_(-5)
        vz.out_feats.fill_(7.0)
        vz.out_point_idx.fill_(-9)
        vz.out_counts.fill_(-1)
        graph.replay()
        torch.cuda.synchronize()
        got = _snapshot(vz)
        for k in ref:
            assert np.array_equal(got[k], ref[k]), (name, rep, k)
        assert vz.fault() == 0
        vz.run()  # eager work between the replays
        torch.cuda.synchronize()


def test_two_calls_in_flight_on_two_streams(gpu_lib):
    """Calls alternating between two default-priority streams, each voxelizer
    with its own inputs, workspace and outputs (the bench's two-stream
    measurement): both copies end with the single-stream outputs."""
    import torch

    wl = synth.throughput(16)
    a = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
    b = gpu_lib.voxelizer_for_workload(wl, "cuda:0")
    a.run()
    torch.cuda.synchronize()
    ref = _snapshot(a)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for i in range(8):
        (a, b)[i % 2].run(stream=streams[i % 2])
    torch.cuda.synchronize()
    for vz in (a, b):
        got = _snapshot(vz)
        for k in ref:
            assert np.array_equal(got[k], ref[k]), k
        assert vz.fault() == 0
