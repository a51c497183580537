"""Benchmark: ROI-aware multi-sweep voxelisation on one MI355X.

One step = one call of mmbev_roi_voxelize over one batch of F nuScenes-shaped
frames (10 sweeps x 32 beams x 1085 columns = 347,200 points each, 32 ROIs,
1440 x 1440 x 40 grid, max 10 points per voxel, 120k voxels per frame), inputs
resident in HBM.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--frames F] [--no-cpu-baseline]

HBM traffic of every kernel of the call (the filter's is the `traffic` field
of the roofline object), and LDS bank conflicts:

    rocprofv3 --pmc FETCH_SIZE -f csv -d DIR_F -o run -- python3 bench.py --probe-traffic DIR_F/meta.json
    rocprofv3 --pmc WRITE_SIZE -f csv -d DIR_W -o run -- python3 bench.py --probe-traffic DIR_W/meta.json
    python bench.py --write-traffic DIR_F DIR_W
    rocprofv3 --pmc SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE ... -f csv -d DIR_L -o run -- python3 bench.py --probe-traffic DIR_L/meta.json
    python bench.py --write-lds DIR_L

--probe-traffic runs the batched call a few times and a plain device copy of
COPY_BYTES bytes, and stores the call's sizes (N, K, V, chunk counts) next to
the counters; --write-traffic scales each counter by the known bytes the copy
moved over what the counter read for it, and stores every kernel's HBM bytes
per launch with its ratio to the bytes its job needs, tagged with the hash of
the library's sources (a changed kernel makes the stored figures stale, and
bench.py then reports null).

value = input points per second over the timed steps (Mpoints/s).  The
roofline object reports the dominant kernel (the fused point filter): its
algorithmic bytes per launch over its mean launch duration, taken live from
HIP events the library records between its launches on the bench's stream.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "Mpoints/s ROI-voxelized (10-sweep, 347k pts) + achieved HBM GB/s vs peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "roi_voxelize_c2x128_traffic.json")
LDS_FILE = os.path.join(ROOT, "profiles", "roi_voxelize_c2x128_lds.json")
CSRC = os.path.join("paper_2608_15437_amd", "csrc")
COPY_BYTES = 1 << 30


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def library_sources() -> list:
    d = os.path.join(ROOT, CSRC)
    return [os.path.join(CSRC, f) for f in sorted(os.listdir(d)) if f.endswith((".hip", ".hpp"))]


def source_sha(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def launch_names(vz) -> list:
    """The launch groups of one call, in order (mmbev_roi_voxelize_profiled)."""
    g = vz.grid
    cells = g.dims[0] * g.dims[1] * g.dims[2]
    kb = max(1, (cells - 1).bit_length())
    passes = (kb + 8) // 9  # digits of at most 9 bits; frames are kept apart, not sorted
    return (["stage", "filter", "segments", "compact"] + [f"sort{p}" for p in range(passes)]
            + ["heads", "fincap", "mean"])


def time_calls(vz, steps: int, warmup: int) -> float:
    import torch

    for _ in range(warmup):
        vz.run()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        vz.run()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def time_two_streams(vz_a, vz_b, steps: int, warmup: int) -> float:
    """Mean time per call with two calls in flight: calls alternate between
    two streams, each voxelizer with its own inputs, workspace and outputs,
    so that one call's latency-bound kernels overlap the next call's filter.
    Returns ms per call."""
    import torch

    streams = [torch.cuda.Stream(), torch.cuda.Stream()]  # default priority
    vzs = [vz_a, vz_b]
    torch.cuda.synchronize()
    for i in range(warmup):
        vzs[i % 2].run(stream=streams[i % 2])
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for i in range(steps):
        vzs[i % 2].run(stream=streams[i % 2])
    for s in streams:
        torch.cuda.current_stream().wait_stream(s)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def time_graph_calls(vz, steps: int, warmup: int) -> float:
    """Mean time of one call captured in a HIP graph and replayed (the entry
    point only enqueues kernels, so a caller can capture it)."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        vz.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        vz.run()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        graph.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def time_launches(vz, steps: int) -> dict:
    """Median duration of every launch group of one call, from events recorded between launches."""
    import torch

    names = launch_names(vz)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)] for _ in range(steps)]
    for row in evs:  # materialise the events
        for e in row:
            e.record()
    torch.cuda.synchronize()
    for row in evs:
        used = vz.run(events=row)
        if used != len(names) + 1:
            raise RuntimeError(f"recorded {used} events, expected {len(names) + 1}")
    torch.cuda.synchronize()
    out = {}
    for k, n in enumerate(names):
        out[n] = statistics.median(row[k].elapsed_time(row[k + 1]) for row in evs) * 1e3  # us
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def median_call_ms(run, steps: int, warmup: int) -> float:
    """Median over `steps` calls of one call's duration, each bracketed by HIP
    events on the current stream (after `warmup` calls)."""
    import torch

    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in pairs:
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in pairs)


def alg_bytes(wl, K: int, V: int) -> int:
    """Algorithmic bytes of one call: x, y, z and the sweep id of every point,
    the passthrough features of the kept points, the output rows, the ROI
    records with their budgets, and the poses."""
    C, M = wl.num_features, wl.grid.max_points
    row = 16 + 4 + 4 * C + 4 * M
    return 13 * wl.num_points + 4 * (C - 3) * K + row * V + 33 * len(wl.roi_desc) + 48 * wl.num_frames * wl.grid.num_sweeps


def outputs_match(exp, got) -> tuple:
    """(structure bit for bit, max |feature difference|) of an oracle and a GPU result."""
    import numpy as np

    V = int(exp["voxel_offsets"][-1])
    same = bool(np.array_equal(exp["voxel_offsets"], got["voxel_offsets"]))
    for k in ("coords", "counts", "point_idx"):
        same = same and bool(np.array_equal(np.asarray(exp[k])[:V], np.asarray(got[k])[:V]))
    err = float(np.max(np.abs(np.asarray(got["feats"])[:V].astype(np.float64) - exp["feats"][:V]))) if V and same else 0.0
    return same, err


def time_config(name: str, wl, dev, steps: int, warmup: int, with_oracle: bool) -> dict:
    """One configuration: the median call (events around each call), the
    median replay of a captured call, counts, algorithmic bytes and their rate
    against the HBM peak, and the oracle on the same inputs."""
    import torch

    from paper_2608_15437_amd import mmbev

    vz = mmbev.voxelizer_for_workload(wl, dev)
    ms = median_call_ms(vz.run, steps, warmup)
    msg = time_graph_calls(vz, steps, warmup)
    h = vz.header()
    res = vz.result()
    N, K, V = wl.num_points, h["kept"], int(res["voxel_offsets"][-1])
    alg = alg_bytes(wl, K, V)
    gbs = alg / (ms * 1e-3) / 1e9
    row = {"frames": wl.num_frames, "points": N, "rois": len(wl.roi_desc), "kept": K, "voxels": V,
           "us_median": round(ms * 1e3, 2), "us_graph_mean": round(msg * 1e3, 2),
           "mpoints_s": round(N / (ms * 1e-3) / 1e6, 1), "alg_bytes": alg, "gbps": round(gbs, 1),
           "frac": round(gbs / HBM_PEAK_GBS, 4), "fault": h["fault"]}
    if with_oracle:
        import oracle

        runs = 3 if N > 1_000_000 else 5
        oracle.run_workload(wl)  # warm-up
        times, exp = [], None
        for _ in range(runs):
            t0 = time.perf_counter()
            exp = oracle.run_workload(wl)
            times.append(time.perf_counter() - t0)
        same, err = outputs_match(exp, res)
        row.update({"oracle_ms_median": round(statistics.median(times) * 1e3, 2), "oracle_runs": runs,
                    "matches_oracle": same and err <= 1e-5, "max_feat_diff": err})
    del vz
    torch.cuda.empty_cache()
    return row


def probe_traffic(frames: int, meta_path: str) -> int:
    """The launches whose counters --write-traffic / --write-lds read: batched
    calls, then one plain copy; the call's sizes go to meta_path."""
    import torch

    import synth
    from paper_2608_15437_amd import mmbev

    wl = synth.throughput(frames)
    vz = mmbev.voxelizer_for_workload(wl, torch.device("cuda:0"))
    for _ in range(3):
        vz.run()
    torch.cuda.synchronize()
    h = vz.header()
    res = vz.result()
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    g = wl.grid
    meta = {"frames": frames, "N": wl.num_points, "K": h["kept"], "V": int(res["voxel_offsets"][-1]),
            "K_in_voxels": int(res["counts"].sum()), "C": wl.num_features, "M": g.max_points,
            "R": len(wl.roi_desc), "B": wl.num_frames, "S": g.num_sweeps, "filter_chunks": h["filter_chunks"],
            "pair_chunks": h["pair_chunks"], "voxel_tiles": h["voxel_tiles"],
            "passes": len([n for n in launch_names(vz) if n.startswith("sort")]), "calls": 3,
            "source_sha": source_sha(library_sources())}
    os.makedirs(os.path.dirname(os.path.abspath(meta_path)), exist_ok=True)
    with open(meta_path, "w") as f:
        json.dump(meta, f)
    log(f"[probe] 3 calls on {frames} frames, one copy of {COPY_BYTES} bytes; sizes in {meta_path}")
    return 0


def time_scatter(wl, dev, steps: int, warmup: int) -> dict:
    """ScatterToBEV (mmbev_scatter_to_bev) of one voxelised workload, timed
    with HIP events around `steps` calls; algorithmic bytes = the map written
    once + the voxel rows read (coords 16 B + C features) + the offsets."""
    import torch

    from paper_2608_15437_amd import mmbev

    vz = mmbev.voxelizer_for_workload(wl, dev)
    vz.run()
    V = vz.header()["voxels"]
    C = wl.num_features
    bev_map = torch.empty(mmbev.bev_map_shape(vz.grid, C), dtype=torch.float32, device=dev)
    for _ in range(warmup):
        vz.scatter_to_bev(bev_map)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        vz.scatter_to_bev(bev_map)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / steps * 1e3
    map_bytes = bev_map.numel() * 4
    alg = map_bytes + V * (16 + 4 * C) + 8 * (wl.num_frames + 1)
    gbs = alg / (us * 1e-6) / 1e9
    out = {"workload": f"{wl.num_frames} frames, {wl.grid.dims[0]}x{wl.grid.dims[1]}x{wl.grid.dims[2]} grid, "
                       f"C={C}: map [B][C*Dz][Dy][Dx] fp32",
           "voxels": V, "map_bytes": map_bytes, "us_per_call": round(us, 1),
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                        "kernel": "bev_clear4_kernel + bev_values_kernel", "alg_bytes_per_call": alg}}
    del bev_map, vz
    torch.cuda.empty_cache()
    return out


def time_selector(steps: int) -> dict:
    """The temporal-ROI selector and sweep-count knob (mmbev_build_rois, host
    code) over 128 detection caches of 64 objects each, the default policy;
    wall clock over `steps` calls on one host thread."""
    import synth
    from paper_2608_15437_amd import mmbev

    d, off, e = synth.detections(7, 128, count=[64] * 128)
    pol = mmbev.policy()
    mmbev.build_rois(d, off, e, pol)
    t0 = time.perf_counter()
    for _ in range(max(steps, 1)):
        out = mmbev.build_rois(d, off, e, pol)
    us = (time.perf_counter() - t0) / max(steps, 1) * 1e6
    return {"frames": 128, "detections_per_frame": 64, "rois": int(out["roi_offsets"][-1]),
            "us_per_call": round(us, 1), "us_per_frame": round(us / 128, 2), "where": "host, one thread"}


def time_clusters(vz, steps: int, warmup: int, ouster: bool = False) -> dict:
    """The connected-component proposer (mmbev_voxel_clusters) over a
    Voxelizer's outputs: layers 0.4-4.4 m above the ground plane (above 1.0 m
    below the sensor for the Ouster grid), cells of one voxel column,
    8-neighbourhood, clusters of at least 2 cells; HIP events around `steps`
    calls."""
    import torch

    from paper_2608_15437_amd import mmbev

    vz.run()
    band = (12, 40) if ouster else (18, 40)
    prm = mmbev.cluster_params(band[0], band[1], 0, 8, 2)
    p = vz.clusters(prm)
    for _ in range(warmup):
        vz.clusters(prm, proposer=p)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        vz.clusters(prm, proposer=p)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / steps * 1e3
    g = vz.grid
    return {"frames": g.num_frames, "grid": [g.dims[0], g.dims[1], g.dims[2]], "voxels": vz.header()["voxels"],
            "clusters": int(p.offsets[-1].item()), "layers": list(band), "us_per_call": round(us, 1),
            "us_per_frame": round(us / g.num_frames, 2), "fault": p.fault()}


def kernel_short_name(name: str) -> str:
    import re

    m = re.search(r"(\w+_kernel)", name)
    if m:
        return m.group(1)
    return "copyBuffer" if "copyBuffer" in name else name.split("(")[0][-40:]


def counter_values(run_dir: str, counters) -> dict:
    """Per-dispatch counter values, summed over the counter's instances, per
    short kernel name in dispatch order: {kernel: [{counter: value}, ...]}."""
    import csv
    import glob

    per = {}
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] in counters:
                key = (kernel_short_name(r["Kernel_Name"]), int(r["Dispatch_Id"]))
                d = per.setdefault(key, {})
                d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    out = {}
    for (name, _), d in sorted(per.items(), key=lambda kv: kv[0][1]):
        out.setdefault(name, []).append(d)
    return out


def split_passes(vals: dict, passes: int) -> dict:
    """count_kernel / scatter_kernel dispatches split by radix pass (every call
    launches one of each per pass, in pass order)."""
    out = {}
    for name, rows in vals.items():
        if name in ("count_kernel", "scatter_kernel") and passes > 1:
            for p in range(passes):
                out[f"{name}[pass {p}]"] = rows[p::passes]
        else:
            out[name] = rows
    return out


def kernel_job_bytes(name: str, m: dict):
    """HBM bytes a kernel's job needs in this design (its inputs read once, its
    outputs written once); None for the latency-bound bookkeeping kernels."""
    N, K, V, C, M = m["N"], m["K"], m["V"], m["C"], m["M"]
    RW = (2 + C) & ~1  # record words: index, x', y', z', raw features 3.., rounded up to even
    if name.startswith("filter_kernel"):
        return 13 * N + 33 * m["R"] + 48 * m["B"] * m["S"]  # x, y, z, sweep id; ROI records; poses
    if name == "compact_kernel":
        # kept bitmaps and counts; the kept points' columns and sweep ids; keys and records
        return N // 8 + 4 * m["filter_chunks"] + (4 * C + 1) * K + 4 * K + 4 * RW * K
    if name.startswith("count_kernel"):
        return 4 * K + 4 * 512 * m["pair_chunks"]  # keys; one count row per chunk
    if name.startswith("scatter_kernel"):
        return (12 if name.endswith("[pass 0]") else 16) * K  # pairs read (pass 0: keys only) and written
    if name == "heads_kernel":
        return 4 * K + 12 * V  # keys; each head's pair, place and count
    if name == "mean_kernel":
        # heads' pairs and places, the values and records of the kept points, the rows
        return 8 * V + (4 + 4 * RW) * m["K_in_voxels"] + V * (16 + 4 + 4 * C + 4 * M)
    return None


def write_traffic(fetch_dir: str, write_dir: str) -> int:
    fe, wr = counter_values(fetch_dir, ["FETCH_SIZE"]), counter_values(write_dir, ["WRITE_SIZE"])
    with open(os.path.join(fetch_dir, "meta.json")) as f:
        meta = json.load(f)
    # the copy of COPY_BYTES is the largest copy dispatch (the others upload inputs)
    copy_f = max(r["FETCH_SIZE"] for r in fe["copyBuffer"])
    copy_w = max(r["WRITE_SIZE"] for r in wr["copyBuffer"])
    fetch_scale = COPY_BYTES / (copy_f * 1024.0)
    write_scale = COPY_BYTES / (copy_w * 1024.0)
    fe, wr = split_passes(fe, meta["passes"]), split_passes(wr, meta["passes"])
    kernels = {}
    for name in fe:
        if name == "copyBuffer" or name not in wr:
            continue
        calls = meta["calls"]
        f_rows, w_rows = fe[name][-calls:], wr[name][-calls:]  # the bench call's dispatches (last ones)
        fk = statistics.mean(r["FETCH_SIZE"] for r in f_rows)
        wk = statistics.mean(r["WRITE_SIZE"] for r in w_rows)
        fb, wb = fk * 1024.0 * fetch_scale, wk * 1024.0 * write_scale
        job = kernel_job_bytes(name, meta)
        kernels[name] = {"fetch_kib_per_launch": round(fk, 1), "write_kib_per_launch": round(wk, 1),
                         "fetch_bytes_per_launch": int(fb), "write_bytes_per_launch": int(wb),
                         "bytes_per_launch": int(fb + wb), "job_bytes": job,
                         "ratio_to_job": round((fb + wb) / job, 3) if job else None}
    filt = [k for k in kernels if k.startswith("filter_kernel")]
    out = {"workload": f"{meta['frames']} nuScenes-shaped frames per call", "sizes": meta,
           "source_sha": source_sha(library_sources()), "probe_source_sha": meta["source_sha"],
           "copy_bytes": COPY_BYTES, "copy_fetch_kib": copy_f, "copy_write_kib": copy_w,
           "fetch_scale": fetch_scale, "write_scale": write_scale,
           "filter_bytes_per_launch": kernels[filt[0]]["bytes_per_launch"] if filt else None,
           "kernels": kernels}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))
    return 0


def write_lds(lds_dir: str) -> int:
    """LDS counters per kernel (mean per dispatch of the bench call) and the
    ratio of bank-conflict cycles to indexed-LDS active cycles."""
    with open(os.path.join(lds_dir, "meta.json")) as f:
        meta = json.load(f)
    names = ["SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_ADDR_CONFLICT", "SQ_LDS_UNALIGNED_STALL",
             "SQ_INSTS_LDS", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS", "SQ_INSTS_VALU"]
    vals = split_passes(counter_values(lds_dir, names), meta["passes"])
    kernels = {}
    for name, rows in vals.items():
        if name == "copyBuffer":
            continue
        rows = rows[-meta["calls"]:]
        mean = {c: statistics.mean(r.get(c, 0.0) for r in rows) for c in rows[0]}
        ent = {c: round(v, 1) for c, v in sorted(mean.items())}
        if mean.get("SQ_LDS_IDX_ACTIVE"):
            ent["bank_conflict_per_idx_active"] = round(mean.get("SQ_LDS_BANK_CONFLICT", 0.0)
                                                        / mean["SQ_LDS_IDX_ACTIVE"], 4)
        kernels[name] = ent
    out = {"workload": f"{meta['frames']} nuScenes-shaped frames per call", "sizes": meta,
           "source_sha": source_sha(library_sources()), "probe_source_sha": meta["source_sha"], "kernels": kernels}
    with open(LDS_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--frames", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-two-streams", action="store_true",
                    help="skip the two-calls-in-flight measurement (kernel traces then time each kernel alone)")
    ap.add_argument("--no-configs", action="store_true", help="skip the per-configuration rows (c1..c5)")
    ap.add_argument("--probe-traffic", metavar="META_JSON")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--write-lds", metavar="LDS_DIR")
    args = ap.parse_args()
    if args.write_traffic:
        return write_traffic(args.write_traffic[0], args.write_traffic[1])
    if args.write_lds:
        return write_lds(args.write_lds)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); frames are independent, so "
              "a multi-GPU run would shard the batch by frame with no exchange", file=sys.stderr)
        return 2
    if args.probe_traffic:
        return probe_traffic(args.frames, args.probe_traffic)

    import numpy as np
    import torch

    import synth
    from paper_2608_15437_amd import mmbev

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    F = args.frames

    log(f"[bench] generating {F} frames")
    t0 = time.time()
    wl = synth.throughput(F)
    log(f"[bench] generated {wl.num_points} points in {time.time() - t0:.1f}s; uploading")
    vz = mmbev.voxelizer_for_workload(wl, dev)
    torch.cuda.synchronize()

    log("[bench] timing the batched call")
    ms = time_calls(vz, args.steps, args.warmup)
    h = vz.header()
    res = vz.result()
    N = wl.num_points
    K, V = h["kept"], int(res["voxel_offsets"][-1])
    C = wl.num_features
    R = len(wl.roi_desc)
    B, S, M = wl.num_frames, wl.grid.num_sweeps, wl.grid.max_points
    alg_total = alg_bytes(wl, K, V)
    alg_filter = 13 * N + 33 * R + 48 * B * S

    log("[bench] timing every launch with events")
    per = time_launches(vz, args.steps)
    filt_us = per["filter"]
    achieved = alg_filter / (filt_us * 1e-6) / 1e9

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("source_sha") == source_sha(library_sources()) and tr.get("sizes", {}).get("frames") == F:
            traffic = tr.get("filter_bytes_per_launch")

    two = None
    if not args.no_two_streams:
        log("[bench] two calls in flight on two streams (a second copy of the batch)")
        vz_b = mmbev.voxelizer_for_workload(wl, dev)
        ms2 = time_two_streams(vz, vz_b, args.steps, args.warmup)
        res_b = vz_b.result()
        two_ok = all(np.array_equal(res[k], res_b[k]) for k in ("coords", "counts", "point_idx", "voxel_offsets")) \
            and np.array_equal(res["feats"], res_b["feats"])
        two = {"mpoints_s": round(N / (ms2 * 1e-3) / 1e6, 1), "ms_per_call": round(ms2, 4), "outputs_match": bool(two_ok),
               "note": "two batches in flight on two default-priority streams, separate workspaces"}
        del vz_b
        torch.cuda.empty_cache()

    log("[bench] single-frame latency (one 347,200-point frame)")
    wl1 = synth.c2()
    vz1 = mmbev.voxelizer_for_workload(wl1, dev)
    us1 = time_calls(vz1, max(args.steps, 20), args.warmup) * 1e3
    us1g = time_graph_calls(vz1, max(args.steps, 20), args.warmup) * 1e3
    del vz1

    configs = {}
    if not args.no_configs:
        for name in ("c1", "c2", "c3", "c4", "c5"):
            log(f"[bench] config {name}: median of {max(args.steps, 100)} calls, oracle beside it")
            configs[name] = time_config(name, synth.CONFIGS[name](), dev, max(args.steps, 100), args.warmup,
                                        not args.no_cpu_baseline)
        c2r, c3r = configs["c2"], configs["c3"]
        configs["roi_speedup_c3_over_c2"] = {
            "time": round(c3r["us_median"] / c2r["us_median"], 3),
            "voxels": round(c3r["voxels"] / max(c2r["voxels"], 1), 2),
            "kept": round(c3r["kept"] / max(c2r["kept"], 1), 2),
            "note": "the same 347,200 points with one all-covering ROI (dense) against 32 temporal ROIs"}

    log("[bench] temporal-ROI selector (host) on 128 detection caches")
    selector = time_selector(args.steps)

    log("[bench] connected-component proposer on the batch's voxels")
    clusters = time_clusters(vz, args.steps, args.warmup)
    log("[bench] connected-component proposer on one Ouster-shaped frame")
    clusters1 = time_clusters(mmbev.voxelizer_for_workload(synth.c4(), dev), args.steps, args.warmup, ouster=True)

    log("[bench] ScatterToBEV of the 8-frame 2160x2160x40 workload (29.9 GB map)")
    bev = time_scatter(synth.c5(), dev, args.steps, args.warmup)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        log("[bench] oracle (single-threaded C) on the same batch")
        times = []
        t_start = time.time()
        exp = None
        while len(times) < 3 and (time.time() - t_start) < 15.0:
            t0 = time.perf_counter()
            exp = oracle.run_workload(wl)
            times.append(time.perf_counter() - t0)
        t_med = statistics.median(times)
        cpu = {"value": round(N / t_med / 1e6, 3), "unit": "Mpoints/s", "cores": 1, "kind": "oracle",
               "sample": f"the full {F}-frame batch ({N} points), {len(times)} run(s), median; "
                         f"CPU {cpu_model()}, nproc {os.cpu_count()}"}
        same, err = outputs_match(exp, res)
        if not same or err > 1e-5:
            log("[bench] WARNING: GPU output differs from the oracle")
        cpu["gpu_output_matches"] = bool(same and err <= 1e-5)
        cpu["max_feat_diff"] = err

    out = {
        "metric": METRIC,
        "value": round(N / (ms * 1e-3) / 1e6, 1),
        "unit": "Mpoints/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{F} nuScenes-shaped frames per call (10 sweeps x 34,720 points, 5 features, "
                               f"32 ROIs, 1440x1440x40 grid, M=10, cap 120k/frame)",
                   "frames": F, "points": N, "kept": K, "voxels": V},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "kernel": "filter_kernel", "kernel_us": round(filt_us, 2),
                     "alg_bytes_per_launch": alg_filter},
        "path_roofline": {"bound": "hbm", "achieved": round(alg_total / (ms * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                          "unit": "GB/s", "frac": round(alg_total / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "alg_bytes_per_call": alg_total,
                          "note": "the whole call: 13 N + 4 (C-3) K + row V + 33 R + 48 B S bytes over ms_per_step"},
        "two_streams": two,
        "launch_us": {k: round(v, 2) for k, v in per.items()},
        "single_frame": {"points": wl1.num_points, "us_per_call": round(us1, 2),
                         "mpoints_s": round(wl1.num_points / (us1 * 1e-6) / 1e6, 1),
                         "us_per_call_graph": round(us1g, 2)},
        "configs": configs,
        "scatter_to_bev": bev,
        "voxel_clusters": {"batch": clusters, "single_ouster_frame": clusters1},
        "roi_selector": selector,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
