"""GPU parity: the HIP library through its C ABI against the CPU oracle on
the same seeded inputs.

Tolerance (normwise, max|gpu - ref| / max|ref| per compared tensor):
1e-4 for float32, 2e-2 for bfloat16 activations/weights with float32
accumulation; the oracle is float64 on the same (bf16-rounded) values.
Group outputs (the cut tensors) are compared as well as the final output.
"""
import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()


def _check_full(orc, layers, h, w, c, tiling, batch, dtype, seed=0, part=False):
    print(f"[parity] {h}x{w}x{c} {tiling} batch={batch} {dtype} seed={seed} stage_partition={part}", flush=True)
    p = W.make_inputs(layers, h, w, c, batch, seed, dtype)
    out, cuts, net, _ = run_gpu(layers, h, w, c, p, tiling, batch, dtype, part=part)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    err = normwise_err(out, ref)
    assert err <= TOL[dtype], (tiling, dtype, err)
    gs, _, _ = W.parse_tiling(tiling, len(layers))
    for g in range(len(gs) - 1):
        cref = orc.forward_layers(layers, h, w, c, p["x"], p, 0, gs[g + 1] - 1)
        e = normwise_err(cuts[g], cref)
        assert e <= TOL[dtype], (tiling, dtype, "cut", g, e)
    return err


def test_tiny_f32(orc):
    wl = W.WORKLOADS["tiny"]
    err = _check_full(orc, wl.layers, wl.h, wl.w, wl.c, wl.tiling, 1, "f32")
    print("tiny f32 err", err)


def test_tiny_bf16(orc):
    wl = W.WORKLOADS["tiny"]
    _check_full(orc, wl.layers, wl.h, wl.w, wl.c, wl.tiling, 2, "bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tiling", ["1x1/NoCut", "3x3/NoCut", "5x5/8/2x2", "2x3/4/3x2", "4x4/12/1x1"])
def test_yolo_small_image(orc, dtype, tiling):
    # the 16-layer YOLOv2 stack on an 80x80 image: every layer kind, all
    # channel widths (32..512), ragged tiles
    _check_full(orc, W.YOLOV2_16, 80, 80, 3, tiling, 1, dtype, seed=3)


def test_yolo_odd_image_batch(orc):
    # odd extents: every max-pool drops a row/column
    _check_full(orc, W.YOLOV2_16, 71, 93, 3, "3x2/8/2x2", 2, "bf16", seed=5)


@pytest.mark.parametrize("h,w,pool", [(96, 96, False), (96, 100, False), (96, 96, True), (96, 100, True)])
def test_patch_block_shapes(orc, h, w, pool):
    # one 3x3 conv, 64 -> 256 channels (bf16), on one tile: the runtime
    # takes 192-row patch blocks here, 12x16 for 96x96 and 16x12 for
    # 96x100 (fewer blocks), with and without the fused pool
    layers = [dict(op=W.CONV, c_out=256, f=3, s=1, p=1, act=W.LEAKY)]
    if pool:
        layers.append(dict(op=W.MAXPOOL, f=2, s=2, p=0))
    _check_full(orc, layers, h, w, 64, "1x1/NoCut", 1, "bf16", seed=21)


def test_many_tiles_chunked_launch(orc):
    # 9x8 = 72 tiles > one launch's 64-tile argument block
    _check_full(orc, W.TINY, 64, 64, 3, "9x8", 1, "f32", seed=9)


@pytest.mark.parametrize("seed", [11, 12, 13, 14])
def test_random_stacks(orc, seed):
    rng = np.random.default_rng(seed)
    layers = []
    c = int(rng.choice([3, 16, 32, 48]))
    c0 = c
    for _ in range(int(rng.integers(2, 6))):
        if rng.random() < 0.3 and layers and layers[-1]["op"] == W.CONV:
            layers.append(W.maxpool())
        else:
            layers.append(W.conv(int(rng.choice([16, 32, 48, 64, 20])), int(rng.choice([1, 3])),
                                 act=str(rng.choice([W.LEAKY, W.LINEAR]))))
    h, w = int(rng.integers(20, 60)), int(rng.integers(20, 60))
    n = len(layers)
    cut = int(rng.integers(1, n)) if n > 2 else None
    tiling = f"{rng.integers(1, 4)}x{rng.integers(1, 4)}" + (f"/{cut}/{rng.integers(1, 3)}x{rng.integers(1, 3)}" if cut else "")
    for dtype in ("f32", "bf16"):
        _check_full(orc, layers, h, w, c0, tiling, 1, dtype, seed=seed)


def test_every_output_written_once_and_guards_untouched():
    import torch
    from paper_2107_06960_amd import mafat as M
    wl = W.WORKLOADS["tiny"]
    p = W.workload_inputs(wl)
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), "3x3")
    net = M.Network(plan, p, 1, "f32")
    x = net.input_tensor(p["x"])
    guard = 4096
    big = torch.full((guard * 2 + net.y.numel(),), float("nan"), device="cuda")
    big[:guard] = 12345.0
    big[-guard:] = 12345.0
    y = big[guard:guard + net.y.numel()].view_as(net.y)
    net.run_group(0, x, y)
    torch.cuda.synchronize()
    assert not torch.isnan(y).any()
    assert torch.all(big[:guard] == 12345.0) and torch.all(big[-guard:] == 12345.0)


def test_deterministic_bitwise():
    import torch
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    p = W.make_inputs(W.YOLOV2_16, 128, 128, 3, 1, 0, "bf16")
    from paper_2107_06960_amd import mafat as M
    plan = M.Plan(W.YOLOV2_16, (128, 128, 3), wl.tiling)
    net = M.Network(plan, p, 1, "bf16")
    x = net.input_tensor(p["x"])
    a = net.run(x).clone()
    b = net.run(x).clone()
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_run_stage_sequence_equals_run_group(dtype):
    # mafat_run_stage for every stage in order == mafat_run_group, bit for bit
    import torch
    from paper_2107_06960_amd import mafat as M
    print(f"[parity] run_stage sequence vs run_group, YOLOv2 96x96 {dtype}", flush=True)
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, 4, dtype)
    plan = M.Plan(W.YOLOV2_16, (96, 96, 3), "3x3/8/2x2")
    net = M.Network(plan, p, 1, dtype)
    x = net.input_tensor(p["x"])
    ref = net.run(x).clone()
    refc = [c.clone() for c in net.cuts]
    net.y.zero_()
    for c in net.cuts:
        c.zero_()
    for g in range(plan.n_groups):
        gin, gout = net.group_io(g, x)
        for s in range(len(plan.stages(g))):
            net.run_stage(g, s, gin, gout)
    torch.cuda.synchronize()
    assert torch.equal(net.y.view(torch.int16 if dtype == "bf16" else torch.int32),
                       ref.view(torch.int16 if dtype == "bf16" else torch.int32))
    for a, b in zip(net.cuts, refc):
        assert torch.equal(a, b)



@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_graph_replay_equals_eager(dtype):
    # The network captured in a HIP graph (torch.cuda.CUDAGraph) and replayed
    # three times, with eager runs of another input and synchronisations in
    # between: every replay equals the eager result bit for bit.
    import torch
    from paper_2107_06960_amd import mafat as M
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, 4, dtype)
    q = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, 5, dtype)
    plan = M.Plan(W.YOLOV2_16, (96, 96, 3), "3x3/8/2x2")
    net = M.Network(plan, p, 1, dtype)
    x = net.input_tensor(p["x"])
    x_other = net.input_tensor(q["x"])
    eager = net.run(x).clone()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        net.run(x, stream=s)
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        net.run(x, stream=torch.cuda.current_stream())
    for k in range(3):
        other = net.run(x_other).clone()        # eager work between replays
        torch.cuda.synchronize()
        assert not torch.equal(other, eager)
        net.y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(net.y, eager), k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("tiling", ["3x3/NoCut", "5x5/8/2x2", "2x3/4/3x2"])
def test_stage_partition(orc, dtype, tiling):
    # stage partition: each tile computes only its part of every stage output,
    # reading the halo from its neighbours' parts
    _check_full(orc, W.YOLOV2_16, 80, 80, 3, tiling, 1, dtype, seed=3, part=True)


def test_stage_partition_odd_batch(orc):
    # odd extents (pools drop a row/column), batch 2, ragged partitions
    _check_full(orc, W.YOLOV2_16, 71, 93, 3, "3x2/8/2x2", 2, "bf16", seed=5, part=True)
    _check_full(orc, W.TINY, 64, 64, 3, "9x8", 1, "f32", seed=9, part=True)


def test_stage_partition_equals_plain_partition_f32():
    # f32: the same sums in the same order per output element, so tile
    # the stage partition and the plain tile partition agree to rounding of the accumulation
    # order only (the kernels' block shapes may differ)
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, 7, "f32")
    a = run_gpu(W.YOLOV2_16, 96, 96, 3, p, "4x4/8/2x2", 1, "f32", want_cuts=False)
    b = run_gpu(W.YOLOV2_16, 96, 96, 3, p, "4x4/8/2x2", 1, "f32", want_cuts=False, part=True)
    assert normwise_err(b, a) <= TOL["f32"]


# A VGG-style stack (3x3 convolutions in pairs and triples between pools,
# linear last layer): another CNN than YOLOv2 for the generalisations the
# method names as future work (more groups, non-square grids, other nets).
VGG_LIKE = [W.conv(64), W.conv(64), W.maxpool(), W.conv(128), W.conv(128), W.maxpool(),
            W.conv(256), W.conv(256), W.conv(256, act=W.LINEAR)]


@pytest.mark.parametrize("part", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_more_groups_and_other_networks(orc, dtype, part):
    # four groups on YOLOv2 (cuts after every pool but the first)
    _check_full(orc, W.YOLOV2_16, 80, 80, 3, "4x4/4/3x3/8/2x2/12/1x1", 1, dtype, seed=31, part=part)
    # three groups with non-square grids on the VGG-style stack
    _check_full(orc, VGG_LIKE, 64, 64, 3, "3x2/3/2x3/6/1x2", 1, dtype, seed=32, part=part)


@pytest.mark.parametrize("tiling,batch", [("3x3/NoCut", 1), ("2x3/4/2x2", 2), ("4x4/2/3x2/6/1x2", 1)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_and_padded_layers(orc, dtype, tiling, batch):
    # a ResNet-style stem (7x7 stride-2 convolution, 3x3 stride-2 padded
    # max-pool), a stride-2 3x3 convolution, a 3x3 stride-1 max-pool, a 5x5
    # convolution: the generic kernels, tiled, against the oracle
    _check_full(orc, W.OTHER_CNN, 224, 200, 3, tiling, batch, dtype, seed=41)
    _check_full(orc, W.OTHER_CNN, 97, 131, 3, tiling, 1, dtype, seed=42, part=True)


# The largest filter and stride the plan takes (11, 4), a 9x9 stride-3
# convolution, padded 3x3 / 5x5 pools and a 1x1 stride-4 convolution.
WIDE_STRIDES = [W.conv(32, 11, s=4, p=2), W.maxpool(3, 2, 0), W.conv(48, 5), W.maxpool(5, 1, 2),
                W.conv(16, 9, s=3, p=4), W.conv(16, 1, s=4, p=0)]


@pytest.mark.parametrize("tiling", ["3x3/NoCut", "2x3/2/2x1", "5x4/4/3x3"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_largest_filters_and_strides(orc, dtype, tiling):
    # 227x227 -> 56x56 -> 27x27 -> 27x27 -> 27x27 -> 9x9 -> 3x3
    _check_full(orc, WIDE_STRIDES, 227, 227, 3, tiling, 1, dtype, seed=51)
    # 203x251 -> 50x62 -> 24x30 -> ... -> 8x10 -> 2x3, stage partition
    _check_full(orc, WIDE_STRIDES, 203, 251, 3, "2x2/2/2x3", 1, dtype, seed=52, part=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_pixel_tiles(orc, dtype):
    # every tile one output pixel: 20x20 = 400 tiles in group 1 (7 launches
    # per stage) and 10x10 in group 2; ragged 1xN and Nx1 grids
    layers = [W.conv(32), W.maxpool(), W.conv(32), W.maxpool(), W.conv(32, 1)]
    _check_full(orc, layers, 40, 40, 32, "20x20/2/10x10", 1, dtype, seed=61)
    _check_full(orc, layers, 40, 42, 32, "1x21/2/10x1", 2, dtype, seed=62)


@pytest.mark.parametrize("dtype,hwc", [("bf16", (4096, 4096, 64)), ("f32", (2048, 2048, 128))])
def test_two_gib_input_frame(orc, dtype, hwc):
    # An input frame of 2^31 bytes: past the matrix-core kernels' 32-bit
    # byte offsets, so the runtime routes the stage to the generic kernel;
    # every output element is checked for being written, sampled
    # rectangles (corners, edges, tile seams, interior) against the oracle.
    from paper_2107_06960_amd import mafat as M
    h, w, c = hwc
    layers = [W.conv(16)]
    print(f"[parity] {h}x{w}x{c} {dtype}: 2^31-byte frame, generic kernel", flush=True)
    assert M.Plan(layers, hwc, "2x2").stage_kernel(0, 0, 1, dtype) == "generic"
    # parameters by the usual recipe; the input (10^9 elements) seeded
    # U[0, 1) in steps of 1/256, exact in bf16 (no rounding pass needed)
    p = W.make_inputs(layers, 8, 8, c, 1, 71, dtype)
    rng = np.random.default_rng(71)
    p["x"] = rng.integers(0, 256, size=(1, h, w, c), dtype=np.uint8).astype(np.float32) / np.float32(256)
    out, _, net, _ = run_gpu(layers, h, w, c, p, "2x2", 1, dtype)
    del net
    assert not np.isnan(out).any()
    x = p["x"][0]
    rects = [(0, 2, 0, 2), (h - 2, h, w - 2, w), (0, 2, w // 2 - 1, w // 2 + 1), (h // 2 - 1, h // 2 + 1, 0, 2),
             (h // 2 - 1, h // 2 + 1, w // 2 - 1, w // 2 + 1), (1234, 1240, 777, 781), (h - 5, h, 3, 9)]
    for (y0, y1, x0, x1) in rects:
        # the oracle on the input rows/columns these outputs read (a 3x3
        # "same" convolution: one more on each side, clipped to the image)
        a0, a1, b0, b1 = max(0, y0 - 1), min(h, y1 + 1), max(0, x0 - 1), min(w, x1 + 1)
        sub = orc.forward_layers(layers, a1 - a0, b1 - b0, c, x[None, a0:a1, b0:b1], p)[0]
        ref = sub[y0 - a0:y1 - a0, x0 - b0:x1 - b0]
        err = normwise_err(out[0, y0:y1, x0:x1], ref)
        assert err <= TOL[dtype], ((y0, y1, x0, x1), err)


def test_pack_weights_kernel_layout():
    # the repack kernel against the layout written out with torch ops:
    # [cout/BN][cin/32][9][BN][32], rows past c_out zero
    import torch
    from paper_2107_06960_amd import mafat as M
    layers = [W.conv(96), W.conv(48)]   # c_out not a multiple of the block: zero rows
    plan = M.Plan(layers, (40, 40, 64), "1x1", packed_weights=True)
    g = torch.Generator().manual_seed(3)
    for l in range(2):
        d = plan.shape(l)
        cout, cin = d[5], d[2]
        n = M.mafat_packed_weights_size(plan.handle, l, "bf16")
        assert n > 0
        w = torch.randn(cout, 3, 3, cin, generator=g).to(torch.bfloat16).cuda()
        out = torch.full((n // 2,), float("nan"), dtype=torch.bfloat16, device="cuda")
        M.mafat_pack_weights(plan.handle, l, "bf16", w.data_ptr(), out.data_ptr())
        torch.cuda.synchronize()
        nst = cin // 32
        blocks = n // 2 // (nst * 9 * 32)       # nblk * BN (the block size is the runtime's choice)
        matched = False
        for bn in (16, 32, 64, 128, 256):
            if blocks % bn or (cout + bn - 1) // bn * bn != blocks:
                continue
            ref = torch.zeros(blocks, 3, 3, cin, dtype=torch.bfloat16, device="cuda")
            ref[:cout] = w
            ref = ref.view(blocks // bn, bn, 9, nst, 32).permute(0, 3, 2, 1, 4).contiguous().view(-1)
            matched = matched or torch.equal(out, ref)
        assert matched, l


@pytest.mark.parametrize("part", [False, True])
def test_packed_weights_bit_identical(part):
    # the same stage configurations read the same weights from the packed
    # layout: the output is bit for bit that of KRSC weights (batch 1)
    import torch
    p = W.make_inputs(W.YOLOV2_16, 128, 128, 3, 1, 8, "bf16")
    from paper_2107_06960_amd import mafat as M
    outs = []
    for packed in (False, True):
        plan = M.Plan(W.YOLOV2_16, (128, 128, 3), "5x5/8/2x2", stage_partition=part, packed_weights=packed)
        net = M.Network(plan, p, 1, "bf16")
        outs.append(net.run(net.input_tensor(p["x"])).clone())
        torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


def test_packed_weights_parity(orc):
    # batch 2 (stage configurations of one frame), odd extents, with the stage partition
    from paper_2107_06960_amd import mafat as M
    layers, h, w, c = W.YOLOV2_16, 71, 93, 3
    p = W.make_inputs(layers, h, w, c, 2, 5, "bf16")
    plan = M.Plan(layers, (h, w, c), "3x2/8/2x2", stage_partition=True, packed_weights=True)
    net = M.Network(plan, p, 2, "bf16")
    y = net.run(net.input_tensor(p["x"]))
    import torch
    torch.cuda.synchronize()
    out = y.float().cpu().numpy().astype(np.float64)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    assert normwise_err(out, ref) <= TOL["bf16"]


# A 3x3 conv with 128 outputs followed by a 1x1 conv 128 -> 64 (YOLOv2's
# layers 4-5): the runtime runs the pair as one kernel in bf16.
FUSED_PAIR = [W.conv(128), W.conv(64, 1)]


@pytest.mark.parametrize("part,packed,act2,n2", [(False, False, W.LEAKY, 64), (True, False, W.LEAKY, 64),
                                                   (False, True, W.LINEAR, 64), (True, True, W.LEAKY, 64),
                                                   (False, True, W.LEAKY, 32), (True, False, W.LINEAR, 32)])
def test_fused_pair_parity(orc, part, packed, act2, n2):
    # ragged extents (blocks of 16x16 past the tile edges), 2x3 tiles, batch 2
    from paper_2107_06960_amd import mafat as M
    import torch
    layers = [W.conv(128), W.conv(n2, 1, act2)]
    h, w, c = 45, 61, 64
    print(f"[parity] fused pair {h}x{w}x{c} 1x1 outputs {n2} stage_partition={part} packed={packed} act2={act2}",
          flush=True)
    p = W.make_inputs(layers, h, w, c, 2, 21, "bf16")
    plan = M.Plan(layers, (h, w, c), "2x3/NoCut", stage_partition=part, packed_weights=packed)
    net = M.Network(plan, p, 2, "bf16")
    net.y.fill_(float("nan"))
    y = net.run(net.input_tensor(p["x"]))
    torch.cuda.synchronize()
    out = y.float().cpu().numpy().astype(np.float64)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    err = normwise_err(out, ref)
    assert err <= TOL["bf16"], err


# The pair inside a group (scratch buffers on both sides), several rounds
# of workgroups: the fused kernel must not write the buffer it reads.
FUSED_MID = [W.conv(64), W.conv(128), W.conv(64, 1), W.conv(32)]


@pytest.mark.parametrize("layers,h,w,c,batch,tiling,part", [
    (FUSED_PAIR, 50, 39, 64, 1, "3x2/NoCut", False),
    ([W.conv(128), W.conv(32, 1)], 50, 39, 32, 2, "2x2/NoCut", False),
    (FUSED_MID, 120, 136, 32, 6, "2x2/NoCut", False),
    (FUSED_MID, 120, 136, 32, 6, "2x2/NoCut", True),
])
def test_fused_pair_equals_separate_stages(orc, layers, h, w, c, batch, tiling, part):
    # the fused kernel == its two stages run one by one (the 3x3 stage's
    # bf16 outputs through memory, then the 1x1 kernel), bit for bit: the
    # same roundings and the same accumulation order over the 128 channels
    import torch
    from paper_2107_06960_amd import mafat as M
    print(f"[parity] fused pair vs separate stages {h}x{w}x{c} batch={batch} {tiling} stage_partition={part}", flush=True)
    p = W.make_inputs(layers, h, w, c, batch, 22, "bf16")
    plan = M.Plan(layers, (h, w, c), tiling, stage_partition=part)
    net = M.Network(plan, p, batch, "bf16")
    x = net.input_tensor(p["x"])
    ref = net.run(x).clone()
    net.y.zero_()
    gin, gout = net.group_io(0, x)
    for s in range(len(plan.stages(0))):
        net.run_stage(0, s, gin, gout)
    torch.cuda.synchronize()
    d = (net.y.float() - ref.float()).abs().max().item()
    assert torch.equal(net.y.view(torch.int16), ref.view(torch.int16)), d
    out = ref.float().cpu().numpy().astype(np.float64)
    for f in (0, batch - 1):
        e = normwise_err(out[f], orc.forward_layers(layers, h, w, c, p["x"][f:f + 1], p)[0])
        assert e <= TOL["bf16"], (f, e)


FIRST_PAIR = [W.conv(32), W.maxpool(), W.conv(64), W.maxpool(), W.conv(32, 1)]


@pytest.mark.parametrize("h,w,batch,tiling,part,packed", [
    (96, 96, 1, "3x3/NoCut", False, True),
    (71, 93, 3, "2x3/NoCut", False, False),
    (130, 66, 2, "4x2/4/1x1", False, True),
    (71, 93, 2, "3x2/NoCut", True, True),
    (40, 48, 1, "1x1/NoCut", False, True),
    (608, 608, 1, "5x5/4/2x2", False, True),    # the 14x18 blocks (one round of workgroups)
    (600, 584, 2, "5x5/NoCut", False, False),
])
def test_first_layer_pair_equals_separate_stages(orc, h, w, batch, tiling, part, packed):
    # the 3-channel first layer + pool computed inside the 3x3 stage's
    # workgroups (its output never leaves LDS) == the two stages run one by
    # one through memory, bit for bit (same MFMA sequences and roundings);
    # and the oracle
    import torch
    from paper_2107_06960_amd import mafat as M
    print(f"[parity] first-layer pair vs separate stages {h}x{w}x3 batch={batch} {tiling} "
          f"stage_partition={part} packed={packed}", flush=True)
    p = W.make_inputs(FIRST_PAIR, h, w, 3, batch, 23, "bf16")
    plan = M.Plan(FIRST_PAIR, (h, w, 3), tiling, stage_partition=part, packed_weights=packed)
    assert plan.stage_fused(0, 0, batch, "bf16")
    net = M.Network(plan, p, batch, "bf16")
    x = net.input_tensor(p["x"])
    net.y.fill_(float("nan"))
    ref = net.run(x).clone()
    refc = [c.clone() for c in net.cuts]
    assert not torch.isnan(ref).any()
    net.y.zero_()
    for g in range(plan.n_groups):
        gin, gout = net.group_io(g, x)
        for s in range(len(plan.stages(g))):
            net.run_stage(g, s, gin, gout)
    torch.cuda.synchronize()
    assert torch.equal(net.y.view(torch.int16), ref.view(torch.int16))
    for a, b in zip(net.cuts, refc):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    out = ref.float().cpu().numpy().astype(np.float64)
    e = normwise_err(out, orc.forward_layers(FIRST_PAIR, h, w, 3, p["x"], p))
    assert e <= TOL["bf16"], e


@pytest.mark.parametrize("which", ["all", "ends"])
def test_run_group_events(which):
    # per-stage events (all entries) and group events (first and last only,
    # the rest NULL) around a group with two fused pairs: the run succeeds, the
    # output is unchanged, the intervals are ordered
    import sys
    import os
    import torch
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from bench import HipEvents
    from paper_2107_06960_amd import mafat as M
    print(f"[parity] run_group events={which}", flush=True)
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, 9, "bf16")
    plan = M.Plan(W.YOLOV2_16, (96, 96, 3), "3x3/8/2x2", packed_weights=True)
    assert plan.launches(0) == [[0, 1], [2, 3], [4]]
    net = M.Network(plan, p, 1, "bf16")
    x = net.input_tensor(p["x"])
    ref = net.run(x).clone()
    ev = HipEvents()
    n = len(plan.stages(0))
    evs = ev.create(2 * n)
    lst = list(evs) if which == "all" else [evs[0]] + [None] * (2 * n - 2) + [evs[-1]]
    gin, gout = net.group_io(0, x)
    net.run_group(0, gin, gout, events=lst)
    for g in range(1, plan.n_groups):
        a, b = net.group_io(g, x)
        net.run_group(g, a, b)
    torch.cuda.synchronize()
    assert torch.equal(net.y, ref)
    assert ev.ms(evs[0], evs[-1]) > 0
    if which == "all":
        for s in range(n):
            assert ev.ms(evs[2 * s], evs[2 * s + 1]) >= 0
            if s + 1 < n:
                assert ev.ms(evs[2 * s + 1], evs[2 * s + 2]) >= 0
        assert ev.ms(evs[0], evs[1]) > 0  # the first-layer pair's kernel (layers 0-3)
        assert ev.ms(evs[4], evs[5]) > 0  # the fused pair's kernel (layers 4-5)
    ev.destroy(evs)


@pytest.mark.parametrize("dtype,tiling,k", [("bf16", "5x5/8/2x2", 1), ("bf16", "5x5/8/2x2", 3),
                                             ("bf16", "5x5/8/2x2", 7), ("f32", "3x3/NoCut", 2),
                                             ("f32", "5x5/8/2x2", 4)])
def test_tile_batch_bit_identical(dtype, tiling, k):
    # tiles in batches of k (each batch through all stages, the workspace
    # holding k tiles) == every tile at once, bit for bit, cut tensors too;
    # bf16 runs the fused layers 4-5 inside every batch
    import torch
    from paper_2107_06960_amd import mafat as M
    print(f"[parity] tile batch {k}: YOLOv2 96x96 {tiling} {dtype} batch=2", flush=True)
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 2, 12, dtype)
    res = []
    for tb in (0, k):
        plan = M.Plan(W.YOLOV2_16, (96, 96, 3), tiling, packed_weights=(dtype == "bf16"), tile_batch=tb)
        net = M.Network(plan, p, 2, dtype)
        net.y.fill_(float("nan"))
        y = net.run(net.input_tensor(p["x"])).clone()
        torch.cuda.synchronize()
        res.append((y, [c.clone() for c in net.cuts], plan.workspace_size(2, dtype)))
    assert res[1][2] < res[0][2]
    assert torch.equal(res[0][0], res[1][0])
    for a, b in zip(res[0][1], res[1][1]):
        assert torch.equal(a, b)


def test_tile_batch_parity(orc):
    # one tile at a time, odd extents, batch 2, against the oracle
    from paper_2107_06960_amd import mafat as M
    import torch
    layers, h, w, c = W.YOLOV2_16, 71, 93, 3
    print(f"[parity] tile batch 1: YOLOv2 {h}x{w} 3x2/8/2x2 bf16 batch=2", flush=True)
    p = W.make_inputs(layers, h, w, c, 2, 13, "bf16")
    plan = M.Plan(layers, (h, w, c), "3x2/8/2x2", packed_weights=True, tile_batch=1)
    net = M.Network(plan, p, 2, "bf16")
    y = net.run(net.input_tensor(p["x"]))
    torch.cuda.synchronize()
    out = y.float().cpu().numpy().astype(np.float64)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    assert normwise_err(out, ref) <= TOL["bf16"]


def test_run_network_one_call(orc):
    # the one-call form (uploads the parameters, runs, returns the output)
    # == a Network's run, bit for bit, with and without `out`
    import torch
    from paper_2107_06960_amd import mafat as M
    layers, (h, w, c) = W.YOLOV2_16, (96, 96, 3)
    print(f"[parity] run_network one call {h}x{w}x{c} 3x3/8/2x2 bf16 batch 2", flush=True)
    p = W.make_inputs(layers, h, w, c, 2, 41, "bf16")
    plan = M.Plan(layers, (h, w, c), "3x3/8/2x2")
    net = M.Network(plan, p, 2, "bf16")
    x = net.input_tensor(p["x"])
    ref = net.run(x).clone()
    y = M.run_network(plan, x, p)
    out = torch.empty_like(ref)
    y2 = M.run_network(plan, x, p, out=out)
    torch.cuda.synchronize()
    assert y2 is out
    assert torch.equal(y.view(torch.int16), ref.view(torch.int16))
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    e = normwise_err(ref.float().cpu().numpy().astype(np.float64), orc.forward_layers(layers, h, w, c, p["x"], p))
    assert e <= TOL["bf16"], e
