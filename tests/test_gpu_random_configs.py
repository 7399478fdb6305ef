"""GPU parity on seeded random configurations: random conv / max-pool
stacks (filters 1-5, strides 1-2, any padding below the filter, linear or
leaky activations, 16-96 channels), random input extents, 1-3 groups with
random grids, f32 or bf16, packed or KRSC weights, the stage partition,
tile batches and batch 1-2 -- each run of the HIP library compared with the
oracle's untiled forward (normwise, the tolerance of each dtype), with the
output filled with NaN first so an element no kernel writes fails.  A second
set draws the same kind of configurations with variable tiling: random or
balanced tile boundaries per group (without the stage partition); a third
with row reuse (tile rows in order, every stage output computed once into
row bands), with even or random row boundaries."""
import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu

pytestmark = pytest.mark.gpu


def _bounds(brng, dims, ends, rows, cols):
    """Random or balanced boundaries for every group (None: balanced)."""
    if brng.random() < 0.3:
        return None
    rb, cb = [], []
    for e, r, c in zip(ends, rows, cols):
        for E, N, out in ((int(dims[e - 1, 3]), r, rb), (int(dims[e - 1, 4]), c, cb)):
            inner = sorted(int(v) for v in brng.choice(np.arange(1, E), N - 1, replace=False)) if N > 1 else []
            out.append([0] + inner + [E])
    return rb, cb


def _case(seed, orc, variable=False, reuse=False):
    from paper_2107_06960_amd import mafat as M
    rng = np.random.default_rng(1000 + seed)
    brng = np.random.default_rng(5000 + seed)
    for _ in range(100):  # draw until the plan is valid
        c0 = int(rng.choice([3, 16, 32, 64]))
        layers = []
        for _ in range(int(rng.integers(2, 7))):
            if layers and layers[-1]["op"] == W.CONV and rng.random() < 0.3:
                f = int(rng.choice([2, 3]))
                layers.append(W.maxpool(f, int(rng.choice([1, 2])), int(rng.integers(0, f))))
            else:
                f = int(rng.choice([1, 3, 3, 3, 5]))
                s = int(rng.choice([1, 1, 1, 2]))
                p = (f - 1) // 2 if rng.random() < 0.7 else int(rng.integers(0, f))
                layers.append(W.conv(int(rng.choice([16, 32, 48, 64, 96])), f,
                                     act=str(rng.choice([W.LEAKY, W.LINEAR])), s=s, p=p))
        h, w = (int(v) for v in rng.integers(24, 90, size=2))
        dims = orc.shapes(layers, h, w, c0)
        if (dims[:, 3] < 1).any() or (dims[:, 4] < 1).any():
            continue
        n = len(layers)
        starts = [0] + sorted(int(v) for v in rng.choice(np.arange(1, n), size=int(rng.integers(0, min(2, n - 1) + 1)),
                                                       replace=False))
        ends = starts[1:] + [n]
        rows = [int(rng.integers(1, min(4, dims[e - 1, 3]) + 1)) for e in ends]
        cols = [int(rng.integers(1, min(4, dims[e - 1, 4]) + 1)) for e in ends]
        dtype = str(rng.choice(["f32", "bf16"]))
        part = bool(rng.random() < 0.3)
        packed = bool(rng.random() < 0.5)
        tb = 0 if part else int(rng.choice([0, 0, 1, 3]))
        batch = int(rng.choice([1, 2]))
        bounds = None
        if variable or reuse:
            if part:
                continue
            bounds = _bounds(brng, dims, ends, rows, cols) or ("balanced" if variable else None)
        if reuse:
            tb = 0
        try:
            plan = M.Plan(layers, (h, w, c0), (starts, rows, cols), stage_partition=part, packed_weights=packed,
                          tile_batch=tb, bounds=bounds, row_reuse=reuse)
        except M.MafatError:
            continue
        return plan, layers, (h, w, c0), dtype, batch, (starts, rows, cols, part, packed, tb, plan.bounds, reuse)
    raise AssertionError("no valid configuration drawn")


def _run(orc, seed, variable, reuse=False):
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    plan, layers, (h, w, c0), dtype, batch, desc = _case(seed, orc, variable, reuse)
    kind = " variable tiling" if variable else (" row reuse" if reuse else "")
    print(f"[random {seed}{kind}] {h}x{w}x{c0} {dtype} batch={batch} layers="
          f"{[(L['op'], L.get('c_out'), L['f'], L['s'], L['p']) for L in layers]} "
          f"groups/rows/cols/partition/packed/tile_batch/bounds/reuse={desc}", flush=True)
    p = W.make_inputs(layers, h, w, c0, batch, 2000 + seed, dtype)
    net = M.Network(plan, p, batch, dtype)
    x = net.input_tensor(p["x"])
    net.y.fill_(float("nan"))
    out = net.run(x).float().cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    ref = orc.forward_layers(layers, h, w, c0, p["x"], p)
    assert not np.isnan(out).any()
    err = normwise_err(out, ref)
    assert err <= TOL[dtype], (seed, err)


@pytest.mark.parametrize("seed", range(32))
def test_random_configuration(orc, seed):
    _run(orc, seed, False)


@pytest.mark.parametrize("seed", range(16))
def test_random_configuration_variable_tiling(orc, seed):
    _run(orc, 100 + seed, True)


@pytest.mark.parametrize("seed", range(16))
def test_random_configuration_row_reuse(orc, seed):
    _run(orc, 200 + seed, False, reuse=True)
