"""Host-side pieces of bench.py (no GPU): the per-launch accounting of
algorithmic bytes and the traffic summary lookup."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2107_06960_amd import mafat as M  # noqa: E402
from paper_2107_06960_amd import workloads as W  # noqa: E402


def _lib():
    if not os.path.exists(M.LIB_PATH):
        from paper_2107_06960_amd import build
        build.build(verbose=False)
    return M.lib()


def test_launch_bytes_of_fused_pair():
    # the fused layers 4-5 launch reads layer 4's input regions, writes layer
    # 5's output rectangles and reads both layers' weights; layer 4's
    # 128-channel output never goes to memory
    _lib()
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling, packed_weights=True)
    io = bench.stage_io_bytes(plan, 0, 2)
    launches = plan.launches(0, 1, "bf16")
    assert launches == [[0, 1], [2, 3], [4]]
    fused = bench.launch_bytes(io, [2, 3])
    assert fused == io[2][0] + io[3][1] + io[2][2] + io[3][2]
    assert fused < bench.launch_bytes(io, [2]) + bench.launch_bytes(io, [3])
    # layer 4 (3x3, 64 -> 128) and layer 5 (1x1, 128 -> 64) weights, bf16,
    # plus float32 scale and bias
    assert io[2][2] == 128 * 9 * 64 * 2 + 8 * 128 and io[3][2] == 64 * 128 * 2 + 8 * 64
    # a single-stage launch is that stage's own sum
    assert bench.launch_bytes(io, [0]) == sum(io[0])


def test_traffic_summary_matches_sources_or_is_ignored():
    # the committed summary is used only for the kernel sources it was taken
    # on; for those it gives positive fetch and write bytes per launch
    tr = bench.measured_traffic("yolo608_5x5_8_2x2", [8, 8])
    if tr is not None:
        assert tr["fetch_bytes"] > 0 and tr["write_bytes"] > 0
        assert tr["bytes"] == tr["fetch_bytes"] + tr["write_bytes"]
    assert bench.measured_traffic("no_such_workload", [8, 8]) is None


def test_profiled_launch_matches_sources_or_is_ignored():
    # the committed per-launch rocprofv3 averages are used only for the
    # kernel sources they were taken on
    p = bench.profiled_launch("yolo608_5x5_8_2x2", [0, 3])
    if p is not None:
        assert 0 < p["avg_ms"] < 1.0 and p["source"].startswith("profiles/")
    assert bench.profiled_launch("no_such_workload", [0, 3]) is None
    assert bench.profiled_launch("yolo608_5x5_8_2x2", [99, 99]) is None
