"""CPU tests of the C ABI: the library loads without a GPU, exports every
symbol the header declares, its plan (host code) matches the oracle's regions
bit for bit, and invalid requests return the documented status codes
(all checked before any HIP call)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2107_06960_amd import mafat as M
from paper_2107_06960_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(M.LIB_PATH):
        from paper_2107_06960_amd import build
        build.build(verbose=False)
    return M.lib()


def test_exports_every_declared_symbol(lib):
    hdr = open(os.path.join(ROOT, "include", "mafat.h")).read()
    declared = set(re.findall(r"\b(mafat_[a-z_]+)\s*\(", hdr))
    assert declared == set(M.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def _oracle_macs(orc, layers, h, w, c, gs, rows, cols):
    dims = orc.shapes(layers, h, w, c)
    out = []
    for g, R in enumerate(orc.regions(layers, h, w, c, gs, rows, cols)):
        ex = un = 0
        for k in range(R.shape[1]):
            l = gs[g] + k
            L = layers[l]
            if L["op"] != W.CONV:
                continue
            per = int(dims[l, 5]) * L["f"] ** 2 * int(dims[l, 2])
            un += int(dims[l, 3]) * int(dims[l, 4]) * per
            for t in range(R.shape[0]):
                oy0, oy1, ox0, ox1 = R[t, k, 4:]
                ex += int(oy1 - oy0) * int(ox1 - ox0) * per
        out.append((ex, un))
    return out


@pytest.mark.parametrize("name", sorted(W.WORKLOADS))
def test_plan_regions_and_macs_match_oracle(lib, orc, name):
    wl = W.WORKLOADS[name]
    gs, r, c = wl.groups()
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling)
    R = orc.regions(wl.layers, wl.h, wl.w, wl.c, gs, r, c)
    macs = _oracle_macs(orc, wl.layers, wl.h, wl.w, wl.c, gs, r, c)
    for g in range(len(gs)):
        assert np.array_equal(plan.regions(g), R[g])
        assert plan.macs(g) == macs[g]
        assert plan.num_tiles(g) == R[g].shape[0] == r[g] * c[g]
    dims = orc.shapes(wl.layers, wl.h, wl.w, wl.c)
    for l in range(len(wl.layers)):
        assert plan.shape(l) == tuple(dims[l])


def _random_supported(rng):
    # "same" 1x1 / 3x3 convolutions and 2x2/2 pools, and now and then any
    # filter, stride <= filter (so that receptive fields stay rectangles) and
    # padding < filter, for convolutions and max-pools
    layers, c = [], int(rng.integers(1, 40))
    for _ in range(int(rng.integers(1, 7))):
        u = rng.random()
        if u < 0.25:
            layers.append(W.maxpool())
        elif u < 0.6:
            layers.append(W.conv(int(rng.integers(1, 70)), int(rng.choice([1, 3]))))
        else:
            f = int(rng.integers(1, 8))
            s = int(rng.integers(1, min(f, 3) + 1))
            p = int(rng.integers(0, f))
            if rng.random() < 0.5:
                layers.append(W.maxpool(f, s, p))
            else:
                layers.append(W.conv(int(rng.integers(1, 40)), f, s=s, p=p))
    return layers, c


def test_plan_regions_random_match_bruteforce(lib, orc):
    rng = np.random.default_rng(99)
    done = 0
    while done < 150:
        layers, c = _random_supported(rng)
        h, w = int(rng.integers(2, 70)), int(rng.integers(2, 70))
        try:
            dims = orc.shapes(layers, h, w, c)
        except orc.OracleError:
            continue
        n = len(layers)
        ng = int(rng.integers(1, min(3, n) + 1))
        gs = [0] + sorted(int(v) for v in rng.choice(np.arange(1, n), ng - 1, replace=False)) if ng > 1 else [0]
        rows, cols = [], []
        for g in range(ng):
            last = (gs[g + 1] if g + 1 < ng else n) - 1
            rows.append(int(rng.integers(1, min(6, dims[last, 3]) + 1)))
            cols.append(int(rng.integers(1, min(6, dims[last, 4]) + 1)))
        plan = M.Plan(layers, (h, w, c), (gs, rows, cols))
        B = orc.regions_bruteforce(layers, h, w, c, gs, rows, cols)
        for g in range(ng):
            assert np.array_equal(plan.regions(g), B[g]), (layers, h, w, c, gs, rows, cols)
        done += 1


def test_other_cnn_regions_and_stages(lib, orc):
    # strided and padded convolutions and pools (a ResNet-style stem, a 3x3
    # stride-1 pool, a 5x5 convolution): regions equal the oracle's brute
    # force; only 2x2/2 pools join the convolution before them in a stage
    layers = W.OTHER_CNN
    for tiling in ("3x3/NoCut", "2x3/4/2x2", "4x4/2/3x2/6/1x2"):
        gs, r, c = W.parse_tiling(tiling, len(layers))
        plan = M.Plan(layers, (224, 200, 3), tiling)
        B = orc.regions_bruteforce(layers, 224, 200, 3, gs, r, c)
        for g in range(len(gs)):
            assert np.array_equal(plan.regions(g), B[g]), tiling
    plan = M.Plan(layers, (224, 200, 3), "1x1/NoCut")
    assert plan.stages(0) == [(0, 0), (1, 1), (2, 2), (3, 3), (4, 4), (5, 5), (6, 7), (8, 8)]
    dims = orc.shapes(layers, 224, 200, 3)
    assert [plan.shape(l) for l in range(len(layers))] == [tuple(d) for d in dims]


def test_stages_fuse_conv_and_following_pool(lib):
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2")
    assert plan.stages(0) == [(0, 1), (2, 3), (4, 4), (5, 5), (6, 7)]
    assert plan.stages(1) == [(8, 8), (9, 9), (10, 11), (12, 12), (13, 13), (14, 14), (15, 15)]
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), "3x3/3/2x2")   # group 2 starts with a pool
    assert plan.stages(0) == [(0, 1), (2, 2)]
    assert plan.stages(1)[0] == (3, 3)


def _kernels(plan, batch, dtype):
    return [[plan.stage_kernel(g, s, batch, dtype) for s in range(len(plan.stages(g)))]
            for g in range(plan.n_groups)]


def test_stage_kernels(lib):
    # which kernel family runs each stage (host-side routing, no GPU)
    import bench
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    for part in (False, True):
        plan = M.Plan(wl.layers, (608, 608, 3), wl.tiling, stage_partition=part, packed_weights=True)
        assert _kernels(plan, 1, "bf16") == [
            ["patch_first", "patch_first", "patch_1x1", "patch_1x1", "patch"],
            ["patch", "ring", "patch", "patch", "ring", "patch", "ring"]]
    # float32: the first layer alone, every other stage on the fp32 matrix cores
    plan = M.Plan(W.YOLOV2_16, (416, 416, 3), "3x3/NoCut")
    assert _kernels(plan, 1, "f32") == [["first_layer"] + ["mfma_f32"] * 11]
    # every stage its own group: no fused pairs
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), bench.untiled_groups(W.YOLOV2_16), packed_weights=True)
    assert [k[0] for k in _kernels(plan, 1, "bf16")] == \
        ["first_layer", "patch", "patch", "ring", "patch", "patch", "ring", "patch", "patch", "ring", "patch", "ring"]
    # an input frame of 2^31 bytes leaves the matrix-core kernels' 32-bit
    # byte offsets: the generic kernel; one column less stays on them
    for dtype, big, small in (("bf16", (4096, 4096, 64), (4096, 4095, 64)),
                              ("f32", (2048, 2048, 128), (2048, 2047, 128))):
        assert _kernels(M.Plan([W.conv(16)], big, "2x2"), 1, dtype) == [["generic"]]
        assert _kernels(M.Plan([W.conv(16)], small, "2x2"), 1, dtype) == [["patch" if dtype == "bf16" else "mfma_f32"]]
    # strided, large-filter and padded-pool layers: generic kernels and lone
    # pools; "same" 3x3 / 1x1 layers among them stay on the matrix cores
    plan = M.Plan(W.OTHER_CNN, (224, 200, 3), "3x3/NoCut")
    assert _kernels(plan, 1, "bf16") == [["generic", "pool", "patch", "generic", "pool", "generic", "ring", "patch"]]
    # errors
    h = plan.handle
    out = ctypes.c_int32()
    assert lib.mafat_plan_stage_kernel(h, 1, 0, 1, M.MAFAT_BF16, ctypes.byref(out)) == M.MAFAT_EINVAL
    assert lib.mafat_plan_stage_kernel(h, 0, 8, 1, M.MAFAT_BF16, ctypes.byref(out)) == M.MAFAT_EINVAL
    assert lib.mafat_plan_stage_kernel(h, 0, 0, 0, M.MAFAT_BF16, ctypes.byref(out)) == M.MAFAT_EINVAL
    assert lib.mafat_plan_stage_kernel(h, 0, 0, 1, 7, ctypes.byref(out)) == M.MAFAT_EUNSUPPORTED
    assert lib.mafat_plan_stage_kernel(h, 0, 0, 1, M.MAFAT_BF16, None) == M.MAFAT_EINVAL


def test_fused_pair_detection(lib):
    # bf16: layers 0-1 (3 -> 32, pool) run inside layers 2-3 (3x3 32 -> 64,
    # pool), and layer 4 (3x3, 64 -> 128) with layer 5 (1x1, 128 -> 64), in
    # one kernel each, whatever the batch or plan flags; f32 and other shapes
    # not
    for flags in ({}, {"stage_partition": True}, {"packed_weights": True}):
        plan = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2", **flags)
        for batch in (1, 8):
            got = [plan.stage_fused(0, s, batch, "bf16") for s in range(len(plan.stages(0)))]
            assert got == [True, False, True, False, False], (flags, batch, got)
            assert plan.launches(0, batch, "bf16") == [[0, 1], [2, 3], [4]]
            assert not any(plan.stage_fused(1, s, batch, "bf16") for s in range(len(plan.stages(1))))
        assert not any(plan.stage_fused(0, s, 1, "f32") for s in range(len(plan.stages(0))))
    # a cut between layers 4 and 5 separates them
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), "3x3/5/2x2")
    assert plan.stages(0)[-1] == (4, 4) and not plan.stage_fused(0, len(plan.stages(0)) - 1, 1, "bf16")
    # other channel counts, a pool after the 3x3, or a 3x3 second layer: no
    for layers in ([W.conv(96), W.conv(64, 1)], [W.conv(128), W.conv(48, 1)], [W.conv(128), W.conv(128, 1)],
                   [W.conv(128), W.maxpool(), W.conv(64, 1)], [W.conv(128), W.conv(64)]):
        plan = M.Plan(layers, (32, 32, 64), "2x2/NoCut")
        assert not plan.stage_fused(0, 0, 1, "bf16"), layers
    # the 1x1 may have 32 outputs as well
    plan = M.Plan([W.conv(128), W.conv(32, 1)], (32, 32, 64), "2x2/NoCut")
    assert plan.stage_fused(0, 0, 1, "bf16") and plan.stage_kernel(0, 0, 1, "bf16") == "patch_1x1"
    plan = M.Plan([W.conv(128), W.conv(64, 1, W.LINEAR)], (32, 32, 64), "2x2/NoCut")
    assert plan.stage_fused(0, 0, 1, "bf16") and not plan.stage_fused(0, 1, 1, "bf16")
    # the first-layer pair needs the group's first stage to be the 3-channel
    # layer with a pool and the next a 3x3 32 -> 64 with a pool, in one group
    assert not M.Plan(W.YOLOV2_16, (96, 96, 3), "3x3/2/2x2").stage_fused(0, 0, 1, "bf16")   # cut between
    assert M.Plan(W.YOLOV2_16, (96, 96, 3), "3x3/4/2x2").stage_fused(0, 0, 1, "bf16")
    for layers in ([W.conv(16), W.maxpool(), W.conv(64), W.maxpool()],      # 16 first-layer outputs
                   [W.conv(32), W.conv(64), W.maxpool()],                   # no pool after the first
                   [W.conv(32), W.maxpool(), W.conv(64)],                   # no pool after the second
                   [W.conv(32), W.maxpool(), W.conv(128), W.maxpool()],     # 128 outputs
                   [W.conv(32), W.maxpool(), W.conv(64, 1), W.maxpool()]):  # 1x1 second
        assert not M.Plan(layers, (64, 64, 3), "2x2/NoCut").stage_fused(0, 0, 1, "bf16"), layers
    with pytest.raises(M.MafatError):
        plan.stage_fused(0, 2, 1, "bf16")


def test_tile_batch(lib):
    # tiles in batches of K: the workspace holds K tiles' intermediates per
    # scratch buffer; with one tile at a time finer grids need less memory
    # (the paper's trend), with all tiles at once more
    layers, hwc = W.YOLOV2_16, (608, 608, 3)
    full = M.Plan(layers, hwc, "5x5/NoCut")
    one = M.Plan(layers, hwc, "5x5/NoCut", tile_batch=1)
    seven = M.Plan(layers, hwc, "5x5/NoCut", tile_batch=7)
    big = M.Plan(layers, hwc, "5x5/NoCut", tile_batch=99)   # >= the tile count: all at once
    ws = {k: p.workspace_size(1, "bf16") for k, p in (("full", full), ("one", one), ("seven", seven), ("big", big))}
    assert ws["big"] == ws["full"]
    assert ws["one"] < ws["seven"] < ws["full"]
    per_tile = ws["one"] // 256 * 256
    assert abs(ws["seven"] - 7 * ws["one"]) <= 7 * 256 and abs(ws["full"] - 25 * ws["one"]) <= 25 * 256, (ws, per_tile)
    dev = lambda t, k: M.Plan(layers, hwc, t, tile_batch=k).predict_mem("device", 1, "bf16")
    seq = [dev(t, 1) for t in ("1x1/NoCut", "2x2/NoCut", "3x3/NoCut", "5x5/NoCut")]
    assert seq == sorted(seq, reverse=True) and seq[-1] < seq[0], seq
    par = [dev(t, 0) for t in ("1x1/NoCut", "3x3/NoCut", "5x5/NoCut")]
    assert par == sorted(par), par
    # the stage layout is unchanged; errors
    assert one.stages(0) == full.stages(0)
    with pytest.raises(M.MafatError) as e:
        M.Plan(layers, hwc, "5x5/NoCut", stage_partition=True, tile_batch=3)
    assert e.value.rc == M.MAFAT_EUNSUPPORTED
    M.Plan(layers, hwc, "5x5/NoCut", stage_partition=True, tile_batch=25)   # every tile at once: allowed
    assert M.lib().mafat_plan_set_tile_batch(full.handle, -1) == M.MAFAT_EINVAL
    assert M.lib().mafat_plan_set_tile_batch(None, 1) == M.MAFAT_EINVAL
    # back to all tiles at once
    assert M.lib().mafat_plan_set_tile_batch(one.handle, 0) == 0
    assert one.workspace_size(1, "bf16") == ws["full"]


def test_workspace_size(lib):
    plan = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2")
    b1 = plan.workspace_size(1, "bf16")
    assert b1 > 0 and b1 % 256 == 0
    assert plan.workspace_size(4, "bf16") >= 4 * b1 - 256
    assert plan.workspace_size(1, "f32") >= 2 * b1 - 256
    one = M.Plan([W.conv(8)], (16, 16, 3), "2x2")          # single stage: no scratch
    assert one.workspace_size(3, "f32") == 0


def test_stage_partition_plan(lib):
    # stage partition: executed MACs equal the untiled ones (even extents) and
    # never exceed them (odd extents: the rows/columns a pool drops are not
    # computed); the workspace is two full stage outputs per frame
    for tiling in ("5x5/8/2x2", "3x3/NoCut", "4x4/12/1x1"):
        plan = M.Plan(W.YOLOV2_16, (608, 608, 3), tiling, stage_partition=True)
        plain = M.Plan(W.YOLOV2_16, (608, 608, 3), tiling)
        for g in range(plan.n_groups):
            ex, un = plan.macs(g)
            assert ex == un == plain.macs(g)[1]
        assert plan.stages(0) == plain.stages(0)
        # largest stage output that is not a group output, over all groups
        big = 0
        for g in range(plan.n_groups):
            for (a, b) in plan.stages(g)[:-1]:
                d = plan.shape(b)
                big = max(big, d[3] * d[4] * d[5])
        big = (big + 127) // 128 * 128
        nst = max(len(plan.stages(g)) for g in range(plan.n_groups))
        assert plan.workspace_size(3, "bf16") == (3 * 2 * big * 2 + 255) // 256 * 256 or nst < 3
    odd = M.Plan(W.YOLOV2_16, (71, 93, 3), "3x2/8/2x2", stage_partition=True)
    for g in range(odd.n_groups):
        ex, un = odd.macs(g)
        assert 0 < ex <= un
    # unknown flags
    arr = (M.mafat_layer * 1)(M.mafat_layer(0, 8, 3, 1, 1, 1))
    h = ctypes.c_void_p()
    one = (ctypes.c_int32 * 1)(1)
    rc = M.lib().mafat_plan_create_flags(arr, 1, 16, 16, 3, (ctypes.c_int32 * 1)(0), 1, one, one, 8, ctypes.byref(h))
    assert rc == M.MAFAT_EINVAL and not h.value


def test_packed_weights_plan(lib):
    # packed weights: only bf16 3x3 layers run by the patch kernel are
    # packed (same bytes as KRSC when c_out is a multiple of the block);
    # plans without the flag pack nothing; packing a KRSC layer is EINVAL
    plain = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2")
    packed = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2", packed_weights=True)
    for l, L in enumerate(W.YOLOV2_16):
        assert M.mafat_packed_weights_size(plain.handle, l, "bf16") == 0
        assert M.mafat_packed_weights_size(packed.handle, l, "f32") == 0
        n = M.mafat_packed_weights_size(packed.handle, l, "bf16")
        if L["op"] == W.CONV and L["f"] == 3 and l > 0:
            d = packed.shape(l)
            assert n == d[5] * 9 * d[2] * 2, l
        else:
            assert n == 0, l
    assert packed.predict_mem("device", 1, "bf16") == plain.predict_mem("device", 1, "bf16")
    # first layer: KRSC, rejected before anything is enqueued
    assert M.lib().mafat_pack_weights(packed.handle, 0, M.MAFAT_BF16, 16, 16, None) == M.MAFAT_EINVAL
    assert M.lib().mafat_pack_weights(packed.handle, 8, M.MAFAT_BF16, None, 16, None) == M.MAFAT_EINVAL
    with pytest.raises(M.MafatError):
        M.mafat_packed_weights_size(packed.handle, 99, "bf16")
    arr = (M.mafat_layer * 1)(M.mafat_layer(0, 8, 3, 1, 1, 1))
    h = ctypes.c_void_p()
    one = (ctypes.c_int32 * 1)(1)
    assert M.lib().mafat_plan_create_flags(arr, 1, 16, 16, 3, (ctypes.c_int32 * 1)(0), 1, one, one, 8,
                                           ctypes.byref(h)) == M.MAFAT_EINVAL


def _create_rc(layers, h, w, c, gs, rows, cols):
    n = len(layers)
    arr = (M.mafat_layer * max(1, n))()
    for k, L in enumerate(layers):
        arr[k] = M.mafat_layer(*L)
    h_ = ctypes.c_void_p()
    rc = M.lib().mafat_plan_create(arr, n, h, w, c, (ctypes.c_int32 * len(gs))(*gs), len(gs),
                                   (ctypes.c_int32 * len(rows))(*rows), (ctypes.c_int32 * len(cols))(*cols),
                                   ctypes.byref(h_))
    if h_.value:
        M.lib().mafat_plan_destroy(h_.value)
    return rc


def test_plan_create_error_codes(lib):
    conv3 = (0, 8, 3, 1, 1, 1)
    pool = (1, 0, 2, 2, 0, 0)
    ok = _create_rc([conv3, pool], 16, 16, 3, [0], [2], [2])
    assert ok == M.MAFAT_OK
    assert _create_rc([(0, 8, 5, 1, 2, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_OK            # 5x5
    assert _create_rc([(0, 8, 3, 2, 1, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_OK            # stride 2
    assert _create_rc([(1, 0, 3, 2, 1, 0)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_OK            # 3x3 pool
    assert _create_rc([(0, 8, 13, 1, 6, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EUNSUPPORTED  # 13x13
    assert _create_rc([(0, 8, 3, 5, 1, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EUNSUPPORTED   # stride 5
    assert _create_rc([(1, 0, 3, 2, 3, 0)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EUNSUPPORTED   # padding 3 >= f
    assert _create_rc([(0, 8, 3, 1, -1, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EUNSUPPORTED  # padding < 0
    assert _create_rc([(0, 8, 3, 1, 1, 7)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EUNSUPPORTED  # activation
    assert _create_rc([(9, 8, 3, 1, 1, 1)], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EINVAL        # op
    assert _create_rc([conv3, pool], 16, 16, 3, [0], [9], [1]) == M.MAFAT_ESHAPE               # grid > out
    assert b"grid 9x1" in M.lib().mafat_last_error()
    assert _create_rc([conv3, pool], 16, 16, 3, [1], [1], [1]) == M.MAFAT_ESHAPE               # start != 0
    assert _create_rc([conv3, pool], 16, 16, 3, [0, 0], [1, 1], [1, 1]) == M.MAFAT_ESHAPE      # not increasing
    assert _create_rc([conv3, pool], 16, 16, 3, [0, 2], [1, 1], [1, 1]) == M.MAFAT_ESHAPE      # start >= n
    assert _create_rc([conv3, pool], 0, 16, 3, [0], [1], [1]) == M.MAFAT_ESHAPE                # empty input
    assert _create_rc([pool, pool], 3, 3, 3, [0], [1], [1]) == M.MAFAT_ESHAPE                  # 1x1 -> pool
    assert _create_rc([conv3], 40000, 4, 3, [0], [1], [1]) == M.MAFAT_ESHAPE                   # > 32767
    assert _create_rc([], 16, 16, 3, [0], [1], [1]) == M.MAFAT_EINVAL
    assert M.lib().mafat_plan_create(None, 1, 1, 1, 1, None, 1, None, None, None) == M.MAFAT_EINVAL
    assert b"NULL" in M.lib().mafat_last_error()


def test_num_tiles_errors(lib):
    plan = M.Plan(W.TINY, (64, 64, 3), "2x2/2/1x2")
    n = ctypes.c_int32(-1)
    assert M.lib().mafat_plan_num_tiles(plan.handle, 1, ctypes.byref(n)) == M.MAFAT_OK and n.value == 2
    assert M.lib().mafat_plan_num_tiles(plan.handle, 2, ctypes.byref(n)) == M.MAFAT_EINVAL
    assert M.lib().mafat_plan_num_tiles(plan.handle, -1, ctypes.byref(n)) == M.MAFAT_EINVAL
    assert M.lib().mafat_plan_num_tiles(None, 0, ctypes.byref(n)) == M.MAFAT_EINVAL
    assert M.lib().mafat_plan_num_tiles(plan.handle, 0, None) == M.MAFAT_EINVAL


def test_run_argument_errors_before_any_launch(lib):
    plan = M.Plan(W.TINY, (64, 64, 3), "2x2")
    need = plan.workspace_size(1, "f32")
    L = M.lib()
    vp = ctypes.c_void_p
    fake = 1 << 20          # aligned, never dereferenced: validation fails first
    w = M._ptrs([fake, None, fake])
    # workspace too small
    rc = L.mafat_run_group(plan.handle, 0, 1, M.MAFAT_F32, fake, fake * 4, w, w, w, fake, need - 1, None)
    assert rc == M.MAFAT_EWORKSPACE
    # unsupported dtype, bad batch, bad group, null plan
    assert L.mafat_run_group(plan.handle, 0, 1, 7, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EUNSUPPORTED
    assert L.mafat_run_group(plan.handle, 0, 0, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_group(plan.handle, 3, 1, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_group(None, 0, 1, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    # misaligned / null tensors, overlapping x and y, missing weights
    assert L.mafat_run_group(plan.handle, 0, 1, 0, fake + 4, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_group(plan.handle, 0, 1, 0, None, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_group(plan.handle, 0, 1, 0, fake, fake + 256, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    nw = M._ptrs([None, None, fake])
    assert L.mafat_run_group(plan.handle, 0, 1, 0, fake, fake * 4, nw, w, w, fake, need, None) == M.MAFAT_EINVAL
    # workspace misaligned
    assert L.mafat_run_group(plan.handle, 0, 1, 0, fake, fake * 4, w, w, w, fake + 16, need, None) == M.MAFAT_EINVAL
    # the timed variant: same checks, and its events array is required
    ev = M._ptrs([None] * 4)
    rc = L.mafat_run_group_timed(plan.handle, 0, 1, M.MAFAT_F32, fake, fake * 4, w, w, w, fake, need - 1, None, ev)
    assert rc == M.MAFAT_EWORKSPACE
    rc = L.mafat_run_group_timed(plan.handle, 0, 1, M.MAFAT_F32, fake, fake * 4, w, w, w, fake, need, None, None)
    assert rc == M.MAFAT_EINVAL and b"events" in L.mafat_last_error()
    # network with several groups but no cut buffers
    plan2 = M.Plan(W.TINY, (64, 64, 3), "2x2/2/2x2")
    assert L.mafat_run_network(plan2.handle, 1, 0, fake, fake * 4, None, w, w, w, fake, 1 << 30, None) == M.MAFAT_EINVAL
    # single stage: stage index out of range, bad group, then the group checks
    ns = plan.stages(0)
    assert L.mafat_run_stage(plan.handle, 0, len(ns), 1, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_stage(plan.handle, 0, -1, 1, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    assert L.mafat_run_stage(plan.handle, 1, 0, 1, 0, fake, fake * 4, w, w, w, fake, need, None) == M.MAFAT_EINVAL
    rc = L.mafat_run_stage(plan.handle, 0, 0, 1, M.MAFAT_F32, fake, fake * 4, w, w, w, fake, need - 1, None)
    assert rc == M.MAFAT_EWORKSPACE
    assert M.lib().mafat_status_string(M.MAFAT_EWORKSPACE) == b"workspace too small"
    # a group split into tile batches cannot run one stage at a time
    plan3 = M.Plan(W.TINY, (64, 64, 3), "2x2", tile_batch=1)
    need3 = plan3.workspace_size(1, "f32")
    rc = L.mafat_run_stage(plan3.handle, 0, 0, 1, M.MAFAT_F32, fake, fake * 4, w, w, w, fake, need3, None)
    assert rc == M.MAFAT_EUNSUPPORTED
