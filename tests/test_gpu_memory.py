"""GPU: the device memory model of mafat_predict_mem against the device
memory a run actually holds (torch's allocator statistics), on every
full-size workload, the six configurations of the 608x608 sweep among them.

The library allocates nothing; the caller's buffers (input, output, cut
tensors, parameters, workspace) are all there is.  Measured: torch's
requested-bytes statistic (the sizes asked of its allocator, before its
rounding and block part), its peak over a run of the network minus its
value before the network was built; the prediction must equal it exactly.
(The allocator's own allocated-bytes figure, which rounds and may hand out a
larger cached block, is printed alongside.)"""
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import require_gpu

FULL = ["tiny", "yolo416_ftp3", "yolo608_5x5_8_2x2", "yolo608_4x4_12_1x1_b8"] + \
    ["yolo608_sweep_" + t.replace("/", "_") for t in W.SWEEP6]


@pytest.mark.gpu
@pytest.mark.parametrize("part,packed,tile_batch,reuse", [(False, False, 0, False), (True, False, 0, False),
                                                            (False, True, 0, False), (False, True, 1, False),
                                                            (False, False, 0, True), (False, True, 0, True)])
@pytest.mark.parametrize("name", FULL)
def test_device_model_matches_measured_peak(name, part, packed, tile_batch, reuse):
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    wl = W.WORKLOADS[name]
    print(f"[memory] {name}: {wl.h}x{wl.w}x{wl.c} {wl.tiling} batch={wl.batch} {wl.dtype} stage_partition={part} packed={packed} "
          f"tile_batch={tile_batch} row_reuse={reuse}", flush=True)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_stats().get("requested_bytes.all.current", 0)
    base_alloc = torch.cuda.memory_allocated()
    p = W.workload_inputs(wl)
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling, stage_partition=part, packed_weights=packed,
                  tile_batch=tile_batch, row_reuse=reuse)
    net = M.Network(plan, p, wl.batch, wl.dtype)
    x = net.input_tensor(p["x"])
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    net.run(x)
    torch.cuda.synchronize()
    used = torch.cuda.memory_stats()["requested_bytes.all.peak"] - base
    alloc = torch.cuda.max_memory_allocated() - base_alloc
    pred = plan.predict_mem("device", wl.batch, wl.dtype)
    print(f"[memory] {name}: predicted {pred} B, requested {used} B (allocator blocks {alloc} B)", flush=True)
    assert used == pred
    del net, x


@pytest.mark.gpu
@pytest.mark.parametrize("mib", [12, 16, 24])
def test_search_under_device_limit_runs_within_it(mib):
    # Algorithm 2 with the sequential device model picks a configuration;
    # run one tile at a time, it holds exactly the predicted bytes, which
    # are below the limit
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    spec, pred, fits = M.mafat_get_config(W.YOLOV2_16, (608, 608, 3), mib << 20, model="device_seq",
                                          dtype="bf16")
    print(f"[memory] search under {mib} MiB: {spec}, predicted {pred} B", flush=True)
    assert fits
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_stats().get("requested_bytes.all.current", 0)
    p = W.workload_inputs(wl)
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, tile_batch=1)
    net = M.Network(plan, p, 1, "bf16")
    x = net.input_tensor(p["x"])
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    net.run(x)
    torch.cuda.synchronize()
    used = torch.cuda.memory_stats()["requested_bytes.all.peak"] - base
    assert used == pred < (mib << 20)
    del net, x


@pytest.mark.gpu
@pytest.mark.parametrize("mib", [11, 12])
def test_balanced_search_under_device_limit_runs_within_it(mib):
    # variable tiling: the search with balanced boundaries
    # (mafat_get_config_balanced, the sequential device model) fits at
    # 11 MiB, where no evenly tiled candidate does, and the plan it names,
    # run one tile at a time with its balanced boundaries, holds exactly the
    # predicted bytes
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    spec, pred, fits = M.mafat_get_config(W.YOLOV2_16, (608, 608, 3), mib << 20, model="device_seq",
                                          dtype="bf16", balanced=True)
    _, _, even_fits = M.mafat_get_config(W.YOLOV2_16, (608, 608, 3), mib << 20, model="device_seq", dtype="bf16")
    print(f"[memory] balanced search under {mib} MiB: {spec}, predicted {pred} B (even tiles fit: {even_fits})",
          flush=True)
    assert fits
    if mib == 11:
        assert not even_fits
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_stats().get("requested_bytes.all.current", 0)
    p = W.workload_inputs(wl)
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, tile_batch=1, bounds="balanced")
    net = M.Network(plan, p, 1, "bf16")
    x = net.input_tensor(p["x"])
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    net.run(x)
    torch.cuda.synchronize()
    used = torch.cuda.memory_stats()["requested_bytes.all.peak"] - base
    assert used == pred < (mib << 20)
    del net, x


@pytest.mark.gpu
@pytest.mark.parametrize("spec", ["3x3/NoCut", "5x5/12/2x2", "5x5/8/2x2"])
@pytest.mark.parametrize("tile_batch", [0, 1])
def test_device_model_matches_measured_peak_balanced(spec, tile_batch):
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    print(f"[memory] balanced {spec} tile_batch={tile_batch}", flush=True)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    base = torch.cuda.memory_stats().get("requested_bytes.all.current", 0)
    p = W.workload_inputs(wl)
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, packed_weights=True, tile_batch=tile_batch, bounds="balanced")
    net = M.Network(plan, p, 1, "bf16")
    x = net.input_tensor(p["x"])
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    net.run(x)
    torch.cuda.synchronize()
    used = torch.cuda.memory_stats()["requested_bytes.all.peak"] - base
    assert used == plan.predict_mem("device", 1, "bf16")
    del net, x
