"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (same plan, batch, dtype and stage kernels).

The whole network runs on the GPU; the oracle then computes sampled output
rectangles one by one from the input (its forward_rect back-projects the
rectangle through the layers and convolves only that region, untiled, in
float64), for the final output and for every cut tensor between groups.
Rectangles are placed at the image corners, on the tile seams of the
group that produced the tensor, and in the interior, so the halo and
border handling of the tiles around them are all exercised.  For batched
workloads, the first, a middle and the last frame are sampled.

Tolerance: normwise over each rectangle (see gpu_util.TOL).
"""
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu, run_gpu

FULL = ["yolo416_ftp3", "yolo608_5x5_8_2x2", "yolo608_4x4_12_1x1_b8"] + \
    ["yolo608_sweep_" + t.replace("/", "_") for t in W.SWEEP6]


def _seams(extent, parts):
    # first row/column of each tile after the first: floor(i * E / N)
    return [i * extent // parts for i in range(1, parts)]


def sample_rects(h, w, rows, cols, size=2):
    """Rectangles (y0, y1, x0, x1) of side `size` on an h x w tensor tiled
    rows x cols: the 4 corners, one across the first and one across the
    last tile seam (rows and columns together), and one at the centre."""
    def span(a, e):
        a = max(0, min(a, e - size))
        return a, a + size
    sy, sx = _seams(h, rows), _seams(w, cols)
    picks = [(0, 0), (0, w), (h, 0), (h, w), (h // 2, w // 2)]
    if sy or sx:
        fy, ly = (sy[0], sy[-1]) if sy else (h // 2, h // 2)
        fx, lx = (sx[0], sx[-1]) if sx else (w // 2, w // 2)
        picks += [(fy, fx), (ly, lx)]
    out = []
    for cy, cx in picks:
        r = span(cy - size // 2, h) + span(cx - size // 2, w)
        if r not in out:
            out.append(r)
    return out


def test_sample_rects_cover_seams():
    # host-side check of the sampler: corners and both seams of a 5x5 grid
    r = sample_rects(76, 76, 5, 5)
    assert (0, 2, 0, 2) in r and (74, 76, 74, 76) in r and (0, 2, 74, 76) in r
    seams = _seams(76, 5)
    assert any(y0 < seams[0] < y1 and x0 < seams[0] < x1 for (y0, y1, x0, x1) in r)
    assert any(y0 < seams[-1] < y1 and x0 < seams[-1] < x1 for (y0, y1, x0, x1) in r)
    assert all(0 <= y0 < y1 <= 76 and 0 <= x0 < x1 <= 76 for (y0, y1, x0, x1) in r)


@pytest.mark.gpu
@pytest.mark.parametrize("name", FULL)
def test_fullsize_sampled(orc, name):
    require_gpu()
    wl = W.WORKLOADS[name]
    print(f"[fullsize] {name}: {wl.h}x{wl.w}x{wl.c} {wl.tiling} batch={wl.batch} {wl.dtype}", flush=True)
    p = W.workload_inputs(wl)
    out, cuts, _, _ = run_gpu(wl.layers, wl.h, wl.w, wl.c, p, wl.tiling, wl.batch, wl.dtype)
    gs, grows, gcols = W.parse_tiling(wl.tiling, len(wl.layers))
    frames = [0] if wl.batch == 1 else [0, wl.batch // 2, wl.batch - 1]
    tensors = [(cuts[g], gs[g + 1], (grows[g], gcols[g])) for g in range(len(gs) - 1)]
    tensors.append((out, len(wl.layers), (grows[-1], gcols[-1])))
    worst = 0.0
    for got, nl, (rows, cols) in tensors:
        layers = wl.layers[:nl]
        th, tw = got.shape[1], got.shape[2]
        for f in frames:
            for (y0, y1, x0, x1) in sample_rects(th, tw, rows, cols):
                ref = orc.forward_rect(layers, wl.h, wl.w, wl.c, p["x"][f], p, y0, y1, x0, x1)
                err = normwise_err(got[f, y0:y1, x0:x1, :], ref)
                worst = max(worst, err)
                assert err <= TOL[wl.dtype], (name, nl, f, (y0, y1, x0, x1), err)
    print(f"[fullsize] {name}: worst normwise error {worst:.3g}", flush=True)



@pytest.mark.gpu
@pytest.mark.parametrize("k", [1, 5])
def test_fullsize_tile_batch_bit_identical(k):
    # the benchmark workload at full size, tiles in batches of k (one tile,
    # one grid row of the first group) == every tile at once, bit for bit
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    wl = W.WORKLOADS["yolo608_5x5_8_2x2"]
    print(f"[fullsize] {wl.name} tile batch {k} vs all tiles", flush=True)
    p = W.workload_inputs(wl)
    outs = []
    for tb in (0, k):
        plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling, packed_weights=True, tile_batch=tb)
        net = M.Network(plan, p, wl.batch, wl.dtype)
        outs.append(net.run(net.input_tensor(p["x"])).clone())
        torch.cuda.synchronize()
        del net
    assert torch.equal(outs[0], outs[1])
