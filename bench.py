"""Benchmark: fused-tile (MAFAT) execution of YOLOv2 layers 0-15 on one GPU.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--graph]

Default workload: 608x608x3, bf16 activations/weights with fp32 accumulate,
two groups -- layers 0-7 on a 5x5 tile grid, layers 8-15 on 2x2
("5x5/8/2x2"), batch 1.  Inputs are seeded synthetic tensors already resident
in device memory; one step is one pass of the whole stack (both groups).

Prints ONE JSON line: frames/s (value), executed/useful TFLOP/s and their
fraction of the bf16 (or fp32) matrix-core peak, per-group and per-stage
times from HIP events recorded on the launch stream, the roofline of the
dominant stage kernel, peak device memory against the untiled layer-by-layer
baseline, and the CPU oracle's rate on a bounded sample (baseline only).
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "frames/s + TFLOP/s (frac of MFMA peak), YOLOv2 L0-15 608² 2-group tiled"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # MI355X dense matrix-core peaks
# MI355X vector-ALU peak: 256 CUs x 4 SIMDs x 16 lanes x 2 multiply-adds
# (bf16 packed dot product, or packed fp32 FMA) x 2 flop x 2.4 GHz.
PEAK_VALU_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded."""

    def __init__(self):
        self.rt = ctypes.CDLL("libamdhip64.so.7")   # already loaded by torch: same runtime
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.rt.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            assert self.rt.hipEventCreate(ctypes.byref(e)) == 0
            out.append(e.value)
        return out

    def record(self, e, stream):
        assert self.rt.hipEventRecord(ctypes.c_void_p(e), ctypes.c_void_p(stream.cuda_stream)) == 0

    def ms(self, a, b):
        f = ctypes.c_float()
        assert self.rt.hipEventSynchronize(b) == 0
        assert self.rt.hipEventElapsedTime(ctypes.byref(f), a, b) == 0
        return f.value

    def destroy(self, evs):
        for e in evs:
            self.rt.hipEventDestroy(e)


def stage_flops(plan, g):
    """Executed FLOPs (2 * MAC, halo recompute included) of every stage of
    group g for one frame, from the plan's region table."""
    first, nl, nt = plan.group(g)
    R = plan.regions(g)
    out = []
    for (a, b) in plan.stages(g):
        L = plan.layers[a]
        if L["op"] != "conv":
            out.append(0)
            continue
        d = plan.shape(a)
        per = d[5] * L["f"] * L["f"] * d[2]
        k = a - first
        area = sum(int(R[t, k, 5] - R[t, k, 4]) * int(R[t, k, 7] - R[t, k, 6]) for t in range(nt))
        out.append(2 * area * per)
    return out


def stage_io_bytes(plan, g, esz):
    """Algorithmic HBM bytes of every stage of group g for one frame, as
    (read, written, weights): each tile's input region (halo included) read
    once, each tile's output rectangle written once, the weights (and
    scale, bias) once."""
    first, nl, nt = plan.group(g)
    R = plan.regions(g)
    out = []
    for (a, b) in plan.stages(g):
        da, db = plan.shape(a), plan.shape(b)
        ka, kb = a - first, b - first
        rd = sum(int(R[t, ka, 1] - R[t, ka, 0]) * int(R[t, ka, 3] - R[t, ka, 2]) for t in range(nt)) * da[2] * esz
        wr = sum(int(R[t, kb, 5] - R[t, kb, 4]) * int(R[t, kb, 7] - R[t, kb, 6]) for t in range(nt)) * db[5] * esz
        L = plan.layers[a]
        w = (da[5] * L["f"] * L["f"] * da[2] * esz + 8 * da[5]) if L["op"] == "conv" else 0
        out.append((rd, wr, w))
    return out


def launch_bytes(io, launch):
    """Algorithmic bytes of one kernel launch running the stages `launch`
    (a fused pair keeps its intermediate on chip): the first stage's input,
    the last stage's output, every stage's weights."""
    return io[launch[0]][0] + io[launch[-1]][1] + sum(io[s][2] for s in launch)


def bench_network(M, wl, params):
    """The plan and device network bench.py times for workload wl: its
    tiling, batch and dtype, bf16 3x3 weights packed once for the patch
    kernels (MAFAT_PLAN_PACKED_WEIGHTS).  The full-size parity tests build
    their network with this same function."""
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling, packed_weights=True)
    return plan, M.Network(plan, params, wl.batch, wl.dtype)


def untiled_groups(layers):
    """Every stage its own group on a 1x1 grid: the untiled layer-by-layer
    execution with the same kernels (a conv and its following pool fused)."""
    starts, l = [], 0
    while l < len(layers):
        starts.append(l)
        l += 2 if (layers[l]["op"] == "conv" and l + 1 < len(layers) and layers[l + 1]["op"] == "max") else 1
    return starts, [1] * len(starts), [1] * len(starts)


def measure_peak_memory(M, layers, hwc, tiling, params, batch, dtype, x_np, runs=2, part=False, packed=False,
                        tile_batch=0, bounds=None, reuse=False):
    """Peak device memory of a run: torch's requested-bytes statistic (the
    sizes of the buffers the caller allocates: input, output, cut tensors,
    parameters, workspace; the library allocates nothing), its peak during
    the runs minus its value before the network was built.  (The
    allocator's own figure adds its block rounding.)  Returns (bytes, ms)."""
    import torch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_stats().get("requested_bytes.all.current", 0)
    plan = M.Plan(layers, hwc, tiling, stage_partition=part, packed_weights=packed, tile_batch=tile_batch,
                  bounds=bounds, row_reuse=reuse)
    net = M.Network(plan, params, batch, dtype)
    x = net.input_tensor(x_np)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()   # after the weights are packed
    for _ in range(runs):
        net.run(x)
    torch.cuda.synchronize()
    peak = torch.cuda.memory_stats()["requested_bytes.all.peak"] - base
    t0 = time.perf_counter()
    n = 20
    for _ in range(n):
        net.run(x)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / n * 1e3
    del net, x
    return peak, ms


def host_cpu():
    """CPU model, logical CPU count and the CPUs this process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def cpu_baseline(wl, params, exec_macs_per_frame, min_wall_s=1.5, cone_s=(5.0, 10.0)):
    """The oracle timed on the host cores (baseline only).

    value: frames/s of the oracle's own fused-tile forward (forward_tiled,
    the workload's tiling, float64) on frame 0, with the layer loops split
    over all usable host cores (at most 16 threads),
    repeated until at least min_wall_s of wall time.  single_thread: the
    oracle on one thread on 2x2-pixel output rectangles of frame 0 (each
    through its whole receptive field, untiled), its MAC rate scaled to the
    configuration's executed MACs per frame."""
    import numpy as np
    from oracle import oracle as O
    info = host_cpu()
    threads = max(1, min(16, info["usable_cpus"] or 1))
    layers = wl.layers
    gs, rows, cols = wl.groups()
    O.set_threads(threads)
    frames, t0 = 0, time.perf_counter()
    while True:
        O.forward_tiled(layers, wl.h, wl.w, wl.c, params["x"][:1], params, gs, rows, cols)
        frames += 1
        if time.perf_counter() - t0 >= min_wall_s:
            break
    tiled_s = (time.perf_counter() - t0) / frames

    O.set_threads(1)
    dims = O.shapes(layers, wl.h, wl.w, wl.c)
    oh, ow = int(dims[-1, 3]), int(dims[-1, 4])
    gr, gc = oh // 2, ow // 2
    R = O.regions(layers, wl.h, wl.w, wl.c, [0], [gr], [gc])[0]
    # centre, corners and edges first, then a deterministic spread over the rest
    first = [(gr // 2) * gc + gc // 2, 0, gr * gc - 1, (gr // 2) * gc, gc - 1, (gr // 4) * gc + gc // 4]
    order = first + [t for t in range(0, gr * gc, 7) if t not in first]
    x0 = params["x"][0]
    macs = 0
    t1 = time.perf_counter()
    used = []
    for t in order:
        y0, y1, x0_, x1 = (int(v) for v in R[t, -1, 4:])
        O.forward_rect(layers, wl.h, wl.w, wl.c, x0, params, y0, y1, x0_, x1)
        for l, L in enumerate(layers):
            if L["op"] == "conv":
                a = int(R[t, l, 5] - R[t, l, 4]) * int(R[t, l, 7] - R[t, l, 6])
                macs += a * int(dims[l, 5]) * L["f"] ** 2 * int(dims[l, 2])
        used.append(t)
        el = time.perf_counter() - t1
        if el >= cone_s[0] or el + el / len(used) > cone_s[1]:
            break
    el = time.perf_counter() - t1
    rate = macs / el
    return {"value": round(1.0 / tiled_s, 4), "unit": "frames/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"{frames} frame(s) (frame 0) of the oracle's fused-tile forward with tiling {wl.tiling}, "
                       f"float64, layer loops on {threads} threads: {tiled_s:.2f} s per frame, "
                       f"{exec_macs_per_frame / tiled_s / 1e9:.2f} GMAC/s"),
            **info,
            "single_thread": {"value": round(rate / exec_macs_per_frame, 5), "unit": "frames/s", "cores": 1,
                              "sample": (f"{len(used)} output rects of 2x2 px of frame 0, each through its full "
                                         f"receptive field of layers 0-15 ({macs / 1e9:.2f} GMAC in {el:.1f} s, "
                                         f"float64, untiled); frames/s = MAC rate / executed MAC per frame"),
                              "gmac_per_s": round(rate / 1e9, 4)}}


def csrc_digest():
    """SHA-256 over the library's kernel and runtime sources: a counter
    measurement taken on other sources no longer describes the kernels."""
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2107_06960_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(workload, stage_layers):
    """HBM bytes per launch of a stage from a committed counter summary
    (profiles/traffic_*.txt): 'key: value' header lines (workload,
    csrc_sha256, copy_bytes, copy_fetch_kib, copy_write_kib) and one line per
    stage, 'stage A-B: fetch_kib=F write_kib=W' (FETCH_SIZE / WRITE_SIZE per
    dispatch).  Each counter is scaled by the bytes of a plain copy of known
    size over what the same counter reads for it.  None if no summary
    matches this workload, stage and sources."""
    import glob
    digest = csrc_digest()
    want = f"stage {stage_layers[0]}-{stage_layers[1]}"
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.txt"))):
        kv, stages = {}, {}
        with open(path) as fh:
            for line in fh:
                line = line.strip()
                if not line or line.startswith("#") or ":" not in line:
                    continue
                k, v = line.split(":", 1)
                if k.startswith("stage "):  # "stage A-B: fetch_kib=F write_kib=W  # kernel name"
                    stages[k.strip()] = dict(f.split("=", 1) for f in v.split("#")[0].split())
                else:
                    kv[k.strip()] = v.strip()
        if kv.get("workload") != workload or kv.get("csrc_sha256") != digest or want not in stages:
            continue
        try:
            cb = float(kv["copy_bytes"])
            fetch = float(stages[want]["fetch_kib"]) * cb / float(kv["copy_fetch_kib"])
            write = float(stages[want]["write_kib"]) * cb / float(kv["copy_write_kib"])
        except (KeyError, ValueError, ZeroDivisionError):
            continue
        return {"bytes": round(fetch + write), "fetch_bytes": round(fetch), "write_bytes": round(write),
                "source": os.path.relpath(path, ROOT)}
    return None


def profiled_launch(workload, layers):
    """Average duration (ms) of the launch running layers [a, b] under
    rocprofv3's kernel trace, from the committed summary
    profiles/stage_kernels_<workload>.md ('launch A-B: avg_us=...' lines
    below a 'csrc_sha256:' line); None when it was taken on other kernel
    sources or has no such line."""
    path = os.path.join(ROOT, "profiles", f"stage_kernels_{workload}.md")
    if not os.path.exists(path):
        return None
    sha, want = None, f"launch {layers[0]}-{layers[1]}:"
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if line.startswith("csrc_sha256:"):
                sha = line.split(":", 1)[1].strip()
            elif line.startswith(want) and sha == csrc_digest():
                for f in line[len(want):].split("#")[0].split():
                    if f.startswith("avg_us="):
                        return {"avg_ms": float(f[7:]) / 1e3, "source": os.path.relpath(path, ROOT)}
    return None


def config_search(args):
    """Configuration search (Algorithm 2) against an exhaustive measurement
    of its search space on this GPU, YOLOv2 layers 0-15 at 608x608, bf16,
    batch 1.  Candidates: the paper's cuts (16 = no cut, 12, 8) x first-group
    grids 1x1..5x5, second group 2x2, each run with every tile of a stage at
    once (tile batch 'all'), with one tile at a time (tile batch 1, the
    paper's execution order) and, for grids of 3x3 and more, one grid row of
    the first group at a time (tile batch t: a memory/time point between the
    two); every candidate is timed like the headline
    (packed weights, warm-up, then host time over the steps) and its peak
    device memory measured (torch's requested bytes).  For each
    device-memory limit the search takes Algorithm 2 under the device model
    of every tile at once, and if no candidate fits, under the model of one
    tile at a time; it is compared with the fastest candidate whose measured
    peak fits, as is the fastest measured candidate whose predicted memory
    fits (the predictor with measured latencies).
    Prints one JSON line per candidate and one summary line."""
    import torch
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W
    torch.cuda.set_device(0)
    layers, hwc = W.YOLOV2_16, (608, 608, 3)
    params = W.make_inputs(layers, *hwc, 1, 0, "bf16")
    cands = []
    for cut in (16, 12, 8):
        for t in (1, 2, 3, 4, 5):
            spec = f"{t}x{t}/NoCut" if cut == 16 else f"{t}x{t}/{cut}/2x2"
            for tb in (0, 1) + ((t,) if t >= 3 else ()):
                cands.append((spec, tb))
    meas = {}
    for spec, tb in cands:
        peak, _ = measure_peak_memory(M, layers, hwc, spec, params, 1, "bf16", params["x"], packed=True,
                                      tile_batch=tb)
        plan = M.Plan(layers, hwc, spec, packed_weights=True, tile_batch=tb)
        net = M.Network(plan, params, 1, "bf16")
        x = net.input_tensor(params["x"])
        for _ in range(args.warmup):
            net.run(x)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            net.run(x)
        torch.cuda.synchronize()
        # the device model follows the plan's tile batch; device_seq is one tile at a time
        model = "device_seq" if tb == 1 else "device"
        meas[(spec, tb)] = {"ms": (time.perf_counter() - t0) / args.steps * 1e3,
                            "peak_mib": peak / 2 ** 20,
                            "predicted_mib": plan.predict_mem(model, 1, "bf16") / 2 ** 20}
        del net, x
        print(json.dumps({"candidate": spec, "tile_batch": tb or "all",
                          **{k: round(v, 4) for k, v in meas[(spec, tb)].items()}}), flush=True)
    rows = []
    for lim in (12, 13, 14, 16, 18, 20, 22, 24, 26, 28, 30, 34, 40):
        spec, pred, fits = M.mafat_get_config(layers, hwc, lim * 2 ** 20, model="device", batch=1, dtype="bf16")
        tb = 0
        if not fits:
            spec, pred, fits = M.mafat_get_config(layers, hwc, lim * 2 ** 20, model="device_seq", batch=1,
                                                  dtype="bf16")
            tb = 1
        ok = [c for c in cands if meas[c]["peak_mib"] <= lim]
        best = min(ok, key=lambda c: meas[c]["ms"]) if ok else None
        okp = [c for c in cands if meas[c]["predicted_mib"] < lim]
        pm = min(okp, key=lambda c: meas[c]["ms"]) if okp else None
        pick = meas[(spec, tb)]
        rows.append({"limit_mib": lim, "search": spec, "search_tile_batch": tb or "all", "search_fits": fits,
                     "search_ms": round(pick["ms"], 4), "search_peak_mib": round(pick["peak_mib"], 2),
                     "best": best[0] if best else None, "best_tile_batch": (best[1] or "all") if best else None,
                     "best_ms": round(meas[best]["ms"], 4) if best else None,
                     "slowdown_vs_best": round(pick["ms"] / meas[best]["ms"] - 1, 4) if best else None,
                     "predicted_measured": pm[0] if pm else None,
                     "predicted_measured_tile_batch": (pm[1] or "all") if pm else None,
                     "predicted_measured_ms": round(meas[pm]["ms"], 4) if pm else None})
    print(json.dumps({"config_search": rows}), flush=True)


def variable_tiling(args):
    """Variable tiling (each group's balanced tile boundaries,
    mafat_balanced_bounds) against the even split, YOLOv2 layers 0-15,
    608x608x3, bf16, batch 1, on the paper's candidates (cuts 16 = no cut,
    12, 8; first-group grids 2x2..5x5; second group 2x2), each with every
    tile of a stage at once and with one tile at a time (the paper's order):
    the largest tile input region of each group, predicted memory (the
    paper's model and the device model of the tile batch), measured peak
    device memory and host time per frame (packed weights, warm-up, then
    the steps).  One JSON line per candidate, then, per device-memory limit,
    the first candidate in Algorithm 2's order whose one-tile-at-a-time
    prediction fits, with even and with balanced boundaries."""
    import torch
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W
    torch.cuda.set_device(0)
    layers, hwc = W.YOLOV2_16, (608, 608, 3)
    params = W.make_inputs(layers, *hwc, 1, 0, "bf16")
    order, meas = [], {}
    for cut in (16, 12, 8):
        for t in (2, 3, 4, 5):
            spec = f"{t}x{t}/NoCut" if cut == 16 else f"{t}x{t}/{cut}/2x2"
            order.append(spec)
            for bounds in (None, "balanced"):
                for tb in (0, 1):
                    peak, _ = measure_peak_memory(M, layers, hwc, spec, params, 1, "bf16", params["x"],
                                                  packed=True, tile_batch=tb, bounds=bounds)
                    plan = M.Plan(layers, hwc, spec, packed_weights=True, tile_batch=tb, bounds=bounds)
                    net = M.Network(plan, params, 1, "bf16")
                    x = net.input_tensor(params["x"])
                    for _ in range(args.warmup):
                        net.run(x)
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    for _ in range(args.steps):
                        net.run(x)
                    torch.cuda.synchronize()
                    ms = (time.perf_counter() - t0) / args.steps * 1e3
                    del net, x
                    largest = []
                    for g in range(plan.n_groups):
                        R = plan.regions(g)
                        largest.append(int(((R[:, 0, 1] - R[:, 0, 0]) * (R[:, 0, 3] - R[:, 0, 2])).max()))
                    rec = {"candidate": spec, "bounds": bounds or "even", "tile_batch": tb or "all",
                           "row_bounds": plan.bounds[0] if plan.bounds else None,
                           "largest_input_region_px": largest,
                           "predicted_paper_mib": round(plan.predict_mem("paper", 1, "bf16") / 2 ** 20, 3),
                           "predicted_mib": round(plan.predict_mem("device" if tb == 0 else "device_seq", 1,
                                                                   "bf16") / 2 ** 20, 3),
                           "peak_mib": round(peak / 2 ** 20, 3), "ms": round(ms, 4)}
                    meas[(spec, bounds, tb)] = rec
                    print(json.dumps(rec), flush=True)
    rows = []
    for lim in (11, 11.5, 12, 12.5, 13, 14):
        row = {"limit_mib": lim}
        for bounds in (None, "balanced"):
            pick = next((c for c in order if meas[(c, bounds, 1)]["predicted_mib"] < lim), None)
            key = bounds or "even"
            row[key] = pick
            row[key + "_ms"] = meas[(pick, bounds, 1)]["ms"] if pick else None
            row[key + "_peak_mib"] = meas[(pick, bounds, 1)]["peak_mib"] if pick else None
        rows.append(row)
    print(json.dumps({"variable_tiling_search": rows}), flush=True)


def row_reuse(args):
    """Row reuse (tile rows in order, every stage output computed once into
    row bands) against the plain partition (every tile of a stage at once,
    halos recomputed) and against one tile at a time (the paper's order),
    YOLOv2 layers 0-15, 608x608x3, bf16, batch 1, packed weights, on the
    paper's candidates (cuts 16 = no cut, 12, 8; first-group grids 2x2..5x5
    and 8x8; second group 2x2): predicted and measured peak device memory,
    host time per frame (warm-up, then the steps) and executed GFLOP.  One
    JSON line per candidate and execution, then, per device-memory limit,
    the first candidate in Algorithm 2's order whose prediction fits, for
    one tile at a time and for row reuse."""
    import torch
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W
    torch.cuda.set_device(0)
    layers, hwc = W.YOLOV2_16, (608, 608, 3)
    params = W.make_inputs(layers, *hwc, 1, 0, "bf16")
    kinds = {"all_tiles": {}, "one_tile": {"tile_batch": 1}, "row_reuse": {"reuse": True}}
    order, meas = [], {}
    for cut in (16, 12, 8):
        for t in (2, 3, 4, 5, 8):
            spec = f"{t}x{t}/NoCut" if cut == 16 else f"{t}x{t}/{cut}/2x2"
            order.append(spec)
            for kind, kw in kinds.items():
                peak, _ = measure_peak_memory(M, layers, hwc, spec, params, 1, "bf16", params["x"], packed=True, **kw)
                plan = M.Plan(layers, hwc, spec, packed_weights=True, tile_batch=kw.get("tile_batch", 0),
                              row_reuse=kw.get("reuse", False))
                net = M.Network(plan, params, 1, "bf16")
                x = net.input_tensor(params["x"])
                for _ in range(args.warmup):
                    net.run(x)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for _ in range(args.steps):
                    net.run(x)
                torch.cuda.synchronize()
                ms = (time.perf_counter() - t0) / args.steps * 1e3
                del net, x
                gflop = 2 * sum(plan.macs(g)[0] for g in range(plan.n_groups)) / 1e9
                rec = {"candidate": spec, "execution": kind,
                       "predicted_mib": round(plan.predict_mem("device", 1, "bf16") / 2 ** 20, 3),
                       "peak_mib": round(peak / 2 ** 20, 3),
                       "workspace_mib": round(plan.workspace_size(1, "bf16") / 2 ** 20, 3),
                       "gflop_executed": round(gflop, 3), "ms": round(ms, 4)}
                meas[(spec, kind)] = rec
                print(json.dumps(rec), flush=True)
    rows = []
    for lim in (11, 11.5, 12, 13, 14, 16, 20):
        row = {"limit_mib": lim}
        for kind in ("one_tile", "row_reuse"):
            pick = next((c for c in order if meas[(c, kind)]["predicted_mib"] < lim), None)
            row[kind] = pick
            row[kind + "_ms"] = meas[(pick, kind)]["ms"] if pick else None
            row[kind + "_peak_mib"] = meas[(pick, kind)]["peak_mib"] if pick else None
        rows.append(row)
    print(json.dumps({"row_reuse_search": rows}), flush=True)


def phase_trace(args):
    """Per-launch phase timing of the benchmark workload from the trace
    build of the library (libmafat_trace.so: `python -m
    paper_2107_06960_amd.build --trace`), which stamps the wall clock (100
    MHz) at the start and end of every workgroup and at the phase
    boundaries of the first, middle and last workgroup of each launch.
    After warm-up steps, each group runs once with the stamps dumped.  One
    JSON line per launch: the spread of workgroup starts, the span from the
    first start to the last end, workgroup durations (p10/p50/p90/max), and
    for the three stamped workgroups the decode, the phase marks (kernel
    specific, in ns from the workgroup's start) and the end."""
    import re
    import tempfile
    import torch
    from paper_2107_06960_amd import build as B
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W
    if not os.path.exists(B.TRACE_LIB):
        print(json.dumps({"error": f"{B.TRACE_LIB} is missing: python -m paper_2107_06960_amd.build --trace"}))
        sys.exit(1)
    M.LIB_PATH = B.TRACE_LIB
    torch.cuda.set_device(0)
    wl = W.WORKLOADS[args.workload]
    params = W.workload_inputs(wl)
    plan, net = bench_network(M, wl, params)
    x = net.input_tensor(params["x"])
    for _ in range(max(args.warmup, 5)):
        net.run(x)
    torch.cuda.synchronize()
    # the runtime prints the stamps on the C stderr: send file descriptor 2
    # to a file while the groups run
    sys.stderr.flush()
    saved = os.dup(2)
    with tempfile.TemporaryFile(mode="w+") as tf:
        os.dup2(tf.fileno(), 2)
        try:
            os.environ["MAFAT_WG_DUMP"] = "1"
            os.environ["MAFAT_TRACE_DUMP"] = "1"
            for g in range(plan.n_groups):
                gin, gout = net.group_io(g, x)
                net.run_group(g, gin, gout)
                torch.cuda.synchronize()
        finally:
            os.environ.pop("MAFAT_WG_DUMP", None)
            os.environ.pop("MAFAT_TRACE_DUMP", None)
            os.dup2(saved, 2)
            os.close(saved)
        tf.seek(0)
        text = tf.read()
    launches, cur = [], None
    for line in text.splitlines():
        m = re.match(r"WGSPAN stage (\d+)-(\d+) kind (\d+) grid (\d+): span (\d+) ns, starts (\d+), first end (\d+), "
                     r"dur p10 (\d+) p50 (\d+) p90 (\d+) max (\d+) ns", line)
        if m:
            v = [int(t) for t in m.groups()]
            cur = {"first_stage_layers": [v[0], v[1]], "workgroups": v[3], "span_ns": v[4], "start_spread_ns": v[5],
                   "first_end_ns": v[6], "wg_ns": {"p10": v[7], "p50": v[8], "p90": v[9], "max": v[10]},
                   "stamped": []}
            launches.append(cur)
            continue
        m = re.match(r"\s+wg(\d) decode \+(-?\d+) staged \+(-?\d+) loopend \+(-?\d+) end \+(-?\d+) iters:(.*)", line)
        if m and cur is not None:
            end = int(m.group(5))
            marks = [int(t) for t in m.group(6).split()]
            rec = {"decode_ns": int(m.group(2)), "loop_end_ns": int(m.group(4)), "end_ns": end,
                   "chunk_marks_ns": [t for t in marks if 0 < t <= end]}
            if 0 < int(m.group(3)) <= end:
                rec["staged_ns"] = int(m.group(3))
            cur["stamped"].append(rec)
            continue
        m = re.match(r"\s+wg(\d) slots 6-9: (-?\d+) (-?\d+) (-?\d+) (-?\d+)", line)
        if m and cur is not None:
            cur.setdefault("slots_6_9_ns", []).append([int(t) for t in m.groups()[1:]])
    kernels = []  # (group, first stage) of every launch, in order
    for g in range(plan.n_groups):
        s, ns = 0, len(plan.stages(g))
        while s < ns:
            kernels.append((g, s))
            s += 2 if plan.stage_fused(g, s, wl.batch, wl.dtype) else 1
    for k, rec in enumerate(launches):
        rec["workload"] = wl.name
        if k < len(kernels):
            g, s = kernels[k]
            rec["kernel"] = plan.stage_kernel(g, s, wl.batch, wl.dtype)
        print(json.dumps(rec), flush=True)


def all_configs(args):
    """Every workload of the build (the paper's configurations and the six
    cut x grid runs), each with every tile at once, with the stage partition, and one
    tile at a time (the paper's order): per-step latency (median, p10, p90 of HIP events on the
    launch stream around each mafat_run_network call, 10 warm-up steps
    first), frames/s at the median, executed TFLOP/s and its fraction of the
    dtype's matrix-core peak, and peak device memory and median latency
    (timed the same way) of the untiled execution of the same layers.  One
    JSON line per workload and variant."""
    import numpy as np
    import torch
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W
    torch.cuda.set_device(0)
    ev = HipEvents()
    stream = torch.cuda.current_stream()

    def event_ms(net, x):
        # 10 warm-up steps, then one start/stop event pair per step
        for _ in range(10):
            net.run(x)
        torch.cuda.synchronize()
        n = args.steps
        hs = ev.create(2 * n)
        for r in range(n):
            ev.record(hs[2 * r], stream)
            net.run(x, stream=stream)
            ev.record(hs[2 * r + 1], stream)
        torch.cuda.synchronize()
        ms = np.array([ev.ms(hs[2 * r], hs[2 * r + 1]) for r in range(n)])
        ev.destroy(hs)
        return tuple(float(np.percentile(ms, q)) for q in (10, 50, 90))

    variants = ((False, 0), (True, 0), (False, 1))  # (stage partition, tile batch: 0 all tiles at once)
    untiled = {}
    for name, wl, part, tb in [(n, w, r, k) for n, w in W.WORKLOADS.items() for r, k in variants]:
        params = W.workload_inputs(wl)
        plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling, stage_partition=part, packed_weights=True, tile_batch=tb)
        net = M.Network(plan, params, wl.batch, wl.dtype)
        x = net.input_tensor(params["x"])
        p10, p50, p90 = event_ms(net, x)
        ex = sum(2 * plan.macs(g)[0] for g in range(plan.n_groups)) * wl.batch
        us = sum(2 * plan.macs(g)[1] for g in range(plan.n_groups)) * wl.batch
        del net, x
        tp, _ = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), wl.tiling, params, wl.batch, wl.dtype,
                                    params["x"], part=part, packed=True, tile_batch=tb)
        if name not in untiled:
            up, _ = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), untiled_groups(wl.layers), params,
                                        wl.batch, wl.dtype, params["x"], packed=True)
            # the untiled execution timed the same way (events, median)
            uplan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), untiled_groups(wl.layers), packed_weights=True)
            unet = M.Network(uplan, params, wl.batch, wl.dtype)
            ux = unet.input_tensor(params["x"])
            untiled[name] = (up, event_ms(unet, ux)[1])
            del unet, ux
        up, ums = untiled[name]
        print(json.dumps({
            "workload": name, "input": f"{wl.h}x{wl.w}x{wl.c}", "batch": wl.batch, "dtype": wl.dtype,
            "tiling": wl.tiling, "stage_partition": part, "tile_batch": tb or "all",
            "weights": "packed" if wl.dtype == "bf16" else "KRSC",
            "steps": args.steps, "ms_p50": round(p50, 5), "ms_p10": round(p10, 5),
            "ms_p90": round(p90, 5), "frames_per_s": round(wl.batch / (p50 * 1e-3), 1),
            "gflop_executed": round(ex / 1e9, 3), "gflop_useful": round(us / 1e9, 3),
            "tflops_executed": round(ex / (p50 * 1e-3) / 1e12, 2),
            "frac_peak": round(ex / (p50 * 1e-3) / 1e12 / PEAK_TFLOPS[wl.dtype], 4),
            "peak_mem_mib": round(tp / 2 ** 20, 2), "untiled_peak_mem_mib": round(up / 2 ** 20, 2),
            "untiled_ms": round(ums, 5)}), flush=True)


def copy_calibration(mib, reps=5):
    """A plain device copy of a known size, for scaling the HBM byte counters."""
    import torch
    n = mib << 20
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "reps": reps, "kernel": "torch uint8 device-to-device copy_"}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="yolo608_5x5_8_2x2")
    ap.add_argument("--batch", type=int, default=0,
                    help="frames per step (default: the workload's own batch); the committed "
                         "profiles cover the workload's own batch only")
    ap.add_argument("--graph", action="store_true", help="replay one step from a captured HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-untiled", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the stage-partition and HIP-graph timings (for profiler runs: only the plain steps)")
    ap.add_argument("--all-configs", action="store_true",
                    help="latency quantiles, throughput and peak memory of every workload (one JSON line each)")
    ap.add_argument("--config-search", action="store_true",
                    help="only evaluate the configuration search against a measured sweep and exit")
    ap.add_argument("--phase-trace", action="store_true",
                    help="only print per-launch phase timing from the trace build of the library and exit")
    ap.add_argument("--variable-tiling", action="store_true",
                    help="only compare balanced (variable) tile boundaries with the even split and exit")
    ap.add_argument("--row-reuse", action="store_true",
                    help="only compare row reuse with all tiles at once and one tile at a time and exit")
    ap.add_argument("--copy-calibration", type=int, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.config_search:
        config_search(args)
        return
    if args.variable_tiling:
        variable_tiling(args)
        return
    if args.row_reuse:
        row_reuse(args)
        return
    if args.phase_trace:
        phase_trace(args)
        return
    if args.all_configs:
        all_configs(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "only the one-GPU path is built: --gpus must be 1 (frames, and the "
                                   "tiles of a group, would shard across GPUs without exchange)"}))
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2107_06960_amd import mafat as M
    from paper_2107_06960_amd import workloads as W

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    torch.cuda.set_device(0)
    wl = W.WORKLOADS[args.workload]
    own_batch = args.batch in (0, wl.batch)
    if not own_batch:
        wl = dataclasses.replace(wl, batch=args.batch)
    params = W.workload_inputs(wl)
    # The library's fast path: weights packed once for the patch kernels
    # (MAFAT_PLAN_PACKED_WEIGHTS, mafat_pack_weights at load, outside the
    # timed steps); the same steps with KRSC weights are reported beside.
    plan, net = bench_network(M, wl, params)
    x = net.input_tensor(params["x"])
    stream = torch.cuda.current_stream()

    step = lambda: net.run(x)  # noqa: E731
    graph = None
    if args.graph:
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(3):
                net.run(x, stream=s)
        torch.cuda.current_stream().wait_stream(s)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            net.run(x, stream=torch.cuda.current_stream())
        step = graph.replay

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    ms_step = el / args.steps * 1e3
    fps = wl.batch * args.steps / el

    def time_variant(tiling=None, **kw):
        # the headline's loop (warm-up steps, then host time over the timed
        # steps between two synchronisations) on another plan
        vplan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling if tiling is None else tiling, **kw)
        vnet = M.Network(vplan, params, wl.batch, wl.dtype)
        vx = vnet.input_tensor(params["x"])
        for _ in range(args.warmup):
            vnet.run(vx)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            vnet.run(vx)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / args.steps * 1e3

    partition_ms = krsc_ms = untiled_ms = balanced_ms = reuse_ms = None
    if not args.no_untiled:
        # The untiled layer-by-layer execution (every stage its own group on
        # a 1x1 grid, same kernels, packed weights), timed exactly like the
        # headline.
        untiled_ms = time_variant(tiling=untiled_groups(wl.layers), packed_weights=True)
    if not args.no_extras:
        # The same workload with the stage partition (each tile computes only its part
        # of every stage output; no halo recompute), and with KRSC weights.
        partition_ms = time_variant(stage_partition=True, packed_weights=True)
        krsc_ms = time_variant()
        # Variable tiling: each group's balanced tile boundaries.
        balanced_ms = time_variant(packed_weights=True, bounds="balanced")
        # Row reuse: tile rows in order, every stage output computed once.
        reuse_ms = time_variant(packed_weights=True, row_reuse=True)

    # The same step replayed from a captured HIP graph (reported beside the
    # plain loop, which is the headline value).
    graph_ms = None
    if graph is None and not args.no_extras:
        gs_ = torch.cuda.Stream()
        gs_.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(gs_):
            for _ in range(3):
                net.run(x, stream=gs_)
        torch.cuda.current_stream().wait_stream(gs_)
        g_ = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_):
            net.run(x, stream=torch.cuda.current_stream())
        for _ in range(args.warmup):
            g_.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g_.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) / args.steps * 1e3
        del g_

    # Per-stage and per-group durations: the same steps again, one run_group
    # call per group, with start/stop events recorded on the launch stream by
    # the kernel dispatches themselves (hipExtLaunchKernel: nothing is
    # inserted between the kernels).  Groups: events only on the start of the
    # first and the end of the last kernel.  Stages: a start and a stop event
    # on every stage's kernel.  All events are created before the timed loops.
    ev = HipEvents()
    ng = plan.n_groups
    stages = [plan.stages(g) for g in range(ng)]
    nsteps_ev = min(args.steps, 100)
    stage_ms = [[0.0] * len(stages[g]) for g in range(ng)]
    group_ms = [0.0] * ng
    gev = [[ev.create(2) for _ in range(ng)] for _ in range(nsteps_ev)]
    sev = [[ev.create(2 * len(stages[g])) for g in range(ng)] for _ in range(nsteps_ev)]
    io = [net.group_io(g, x) for g in range(ng)]
    torch.cuda.synchronize()
    for r in range(nsteps_ev):
        for g in range(ng):
            lst = [None] * (2 * len(stages[g]))
            lst[0], lst[-1] = gev[r][g]
            net.run_group(g, io[g][0], io[g][1], stream=stream, events=lst)
    torch.cuda.synchronize()
    for r in range(nsteps_ev):
        for g in range(ng):
            net.run_group(g, io[g][0], io[g][1], stream=stream, events=sev[r][g])
    torch.cuda.synchronize()
    step_ev_ms = [0.0] * nsteps_ev
    for r in range(nsteps_ev):
        for g in range(ng):
            gm = ev.ms(gev[r][g][0], gev[r][g][1])
            group_ms[g] += gm / nsteps_ev
            step_ev_ms[r] += gm
            hs = sev[r][g]
            for s_ in range(len(stages[g])):
                stage_ms[g][s_] += ev.ms(hs[2 * s_], hs[2 * s_ + 1]) / nsteps_ev
            ev.destroy(gev[r][g])
            ev.destroy(hs)

    flops = [stage_flops(plan, g) for g in range(ng)]
    esz = 2 if wl.dtype == "bf16" else 4
    sio = [stage_io_bytes(plan, g, esz) for g in range(ng)]
    exec_flops = sum(2 * plan.macs(g)[0] for g in range(ng)) * wl.batch
    useful_flops = sum(2 * plan.macs(g)[1] for g in range(ng)) * wl.batch
    peak = PEAK_TFLOPS[wl.dtype]
    per_stage = []  # one entry per kernel launch (a fused pair of stages is one)
    for g in range(ng):
        for ln in plan.launches(g, wl.batch, wl.dtype):
            a, b = stages[g][ln[0]][0], stages[g][ln[-1]][1]
            f = sum(flops[g][s] for s in ln) * wl.batch
            t = stage_ms[g][ln[0]]  # a fused pair's kernel: the first stage's events
            # Which roofline binds a launch: HBM when its algorithmic
            # intensity (flops per algorithmic byte) is below the ridge
            # point of the matrix-core peak over 8 TB/s (312 flop/byte in
            # bf16, 19.7 in fp32: the stand-alone first layer, K = 27, and
            # the 1x1 layers), else the matrix cores; the fp32 3-channel
            # first layer runs on the vector ALUs.
            first_alone = plan.layers[a]["op"] == "conv" and plan.shape(a)[2] == 3 and b <= a + 1
            nb = launch_bytes(sio[g], ln) * wl.batch
            ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)
            if first_alone and wl.dtype == "f32":
                pk, bound = PEAK_VALU_TFLOPS, "alu"
            elif nb > 0 and f / nb < ridge:
                pk, bound = PEAK_HBM_GBS, "hbm"
            else:
                pk, bound = peak, "mfma"
            row = {"group": g, "layers": [a, b], "ms": round(t, 5), "gflop": round(f / 1e9, 4), "bound": bound,
                   "tflops": round(f / (t * 1e-3) / 1e12, 2) if t > 0 else None,
                   "frac_mfma": round(f / (t * 1e-3) / 1e12 / peak, 4) if t > 0 else None,
                   "hbm_mb": round(nb / 1e6, 3),
                   "gbs": round(nb / (t * 1e-3) / 1e9, 1) if t > 0 else None,
                   "hbm_frac": round(nb / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) if t > 0 else None}
            row["frac"] = row["hbm_frac"] if bound == "hbm" else (
                round(f / (t * 1e-3) / 1e12 / pk, 4) if t > 0 else None)
            per_stage.append(row)
    dom = max(per_stage, key=lambda r: r["ms"])
    dom_f = dom["gflop"] * 1e9
    if dom["bound"] == "hbm":
        roof = {"bound": "hbm", "achieved": dom["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": dom["hbm_frac"], "traffic": None}
    else:
        pk = PEAK_VALU_TFLOPS if dom["bound"] == "alu" else peak
        roof = {"bound": dom["bound"], "achieved": round(dom_f / (dom["ms"] * 1e-3) / 1e12, 2), "peak": pk,
                "unit": "TFLOP/s", "frac": round(dom_f / (dom["ms"] * 1e-3) / 1e12 / pk, 4), "traffic": None}
    roof.update({
        "kernel": f"stage layers {dom['layers'][0]}-{dom['layers'][1]} (group {dom['group']})",
        "per_launch_gflop": dom["gflop"], "per_launch_hbm_mb": dom["hbm_mb"], "avg_ms": dom["ms"],
        "timing": "kernel start/stop HIP events of the dispatch (hipExtLaunchKernel) on the launch stream, "
                  "averaged over the event-timed steps of the whole network"})
    # rocprofv3 figures of the committed profiles (taken at the workload's
    # own batch)
    prof = profiled_launch(wl.name, dom["layers"]) if own_batch else None
    if prof is not None:
        # the same launch under rocprofv3's kernel trace (profiler overhead
        # included), and the fraction it gives
        roof["rocprof_avg_ms"] = round(prof["avg_ms"], 5)
        roof["rocprof_frac"] = round(dom_f / (prof["avg_ms"] * 1e-3) / 1e12 / roof["peak"], 4) \
            if roof["unit"] == "TFLOP/s" else None
        roof["rocprof_source"] = prof["source"]
    tr = measured_traffic(wl.name, dom["layers"]) if own_batch else None
    if tr is not None:
        roof["traffic"] = tr["bytes"]
        roof["traffic_detail"] = tr

    res = {
        "metric": METRIC, "value": round(fps, 2), "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic (seeded U[0,1) input, He-normal weights, folded-BN scale/bias)",
        "config": {"workload": wl.name, "network": "YOLOv2 layers 0-15" if len(wl.layers) == 16 else wl.note,
                   "input": f"{wl.h}x{wl.w}x{wl.c}", "batch": wl.batch, "tiling": wl.tiling,
                   "accumulate": "f32", "graph": bool(args.graph), "weights": "packed for the patch kernels"},
        "tflops_executed": round(exec_flops / (ms_step * 1e-3) / 1e12, 2),
        "tflops_useful": round(useful_flops / (ms_step * 1e-3) / 1e12, 2),
        "frac_mfma_peak_executed": round(exec_flops / (ms_step * 1e-3) / 1e12 / peak, 4),
        "gflop_executed_per_step": round(exec_flops / 1e9, 3),
        "gflop_useful_per_step": round(useful_flops / 1e9, 3),
        "graph_ms_per_step": round(graph_ms, 5) if graph_ms is not None else None,
        "stage_partition_ms_per_step": round(partition_ms, 5) if partition_ms is not None else None,
        "krsc_weights_ms_per_step": round(krsc_ms, 5) if krsc_ms is not None else None,
        "balanced_bounds_ms_per_step": round(balanced_ms, 5) if balanced_ms is not None else None,
        "row_reuse_ms_per_step": round(reuse_ms, 5) if reuse_ms is not None else None,
        "step_ms_events": {q: round(float(np.percentile(step_ev_ms, v)), 5)
                           for q, v in (("p10", 10), ("p50", 50), ("p90", 90))},
        "group_ms": [round(v, 5) for v in group_ms],
        "group_frac_mfma_peak": [round(sum(flops[g]) * wl.batch / (group_ms[g] * 1e-3) / 1e12 / peak, 4)
                                 for g in range(ng)],
        "per_stage": per_stage,
        "roofline": roof,
    }
    # The launch that runs layer 0 (the 3-channel first layer, alone or with
    # the stage after it): its achieved HBM rate of algorithmic bytes against
    # 8 TB/s, and the shallow group's (group 0: tile input regions with halo,
    # weights once, group output once, over the group's time).
    r0 = per_stage[0]
    res["first_layer_launch"] = {"layers": r0["layers"], "bound": r0["bound"], "ms": r0["ms"],
                                 "achieved_gbs": r0["gbs"], "hbm_frac": r0["hbm_frac"],
                                 "frac_mfma": r0["frac_mfma"], "algorithmic_mb": r0["hbm_mb"]}
    g0_bytes = launch_bytes(sio[0], list(range(len(stages[0])))) * wl.batch
    res["shallow_group_hbm"] = {"algorithmic_mb": round(g0_bytes / 1e6, 3), "ms": round(group_ms[0], 5),
                                "achieved_gbs": round(g0_bytes / (group_ms[0] * 1e-3) / 1e9, 1),
                                "frac": round(g0_bytes / (group_ms[0] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}

    if not args.no_untiled:
        del net, x
        tp, _ = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), wl.tiling, params, wl.batch,
                                    wl.dtype, params["x"], packed=True)
        ug = untiled_groups(wl.layers)
        up, _ = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), ug, params, wl.batch,
                                    wl.dtype, params["x"], packed=True)
        res["peak_mem_mib"] = round(tp / 2 ** 20, 2)
        res["untiled_peak_mem_mib"] = round(up / 2 ** 20, 2)
        res["untiled_ms_per_step"] = round(untiled_ms, 5)
        res["tiled_over_untiled_time"] = round(ms_step / untiled_ms, 4)
        if not args.no_extras:
            # The paper's execution order: one tile at a time through its
            # group (mafat_plan_set_tile_batch(plan, 1)): less workspace,
            # many more launches.
            sp, sms = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), wl.tiling, params, wl.batch,
                                          wl.dtype, params["x"], packed=True, tile_batch=1)
            res["tiles_in_sequence"] = {"peak_mem_mib": round(sp / 2 ** 20, 2), "ms_per_step": round(sms, 5)}
            # Row reuse: tile rows in order, every stage output computed once
            # into row bands (its time from the headline's loop above).
            rp, _ = measure_peak_memory(M, wl.layers, (wl.h, wl.w, wl.c), wl.tiling, params, wl.batch,
                                        wl.dtype, params["x"], packed=True, reuse=True)
            res["row_reuse"] = {"peak_mem_mib": round(rp / 2 ** 20, 2),
                                "ms_per_step": round(reuse_ms, 5) if reuse_ms is not None else None}

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, params, sum(plan.macs(g)[0] for g in range(ng)))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
