"""Row reuse: the data reuse between tiles of section 3 (a tile takes the
overlap that tiles run before it already computed) with a group's tiles run
one grid row after another, every layer output computed once into row bands.

Oracle pins (CPU): the row-reuse forward equals the untiled forward bit for
bit on random stacks, groupings and tile rows (its bands are readable
windows, so a read outside a band is an error, not a wrong value); its band
geometry equals a brute force over the filter windows (which rows a part
reads, where each layer's parts end).

Library (CPU, through the C ABI): the workspace of a row-reuse plan holds
exactly the bands the brute force gives (float32, where every stage output
has its bands); executed MACs equal the untiled ones; error codes.

GPU: the library with row reuse against the oracle's untiled forward (small
sizes in full, several tilings, f32 and bf16, packed weights, batch 2, odd
extents), and against the plain fused tile partition.
"""
import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu, run_gpu


def _random_bounds(rng, E, N):
    inner = sorted(int(v) for v in rng.choice(np.arange(1, E), N - 1, replace=False)) if N > 1 else []
    return [0] + inner + [E]


def _random_case(orc, rng, max_rows=6, min_extent=4, max_extent=30):
    """A random stack (convolutions of any filter, stride and padding,
    max-pools), 1-3 groups, random tile rows and row boundaries."""
    while True:
        n = int(rng.integers(1, 6))
        layers = []
        for _ in range(n):
            if rng.random() < 0.6:
                f = int(rng.choice([1, 2, 3, 5]))
                s = 1 if f == 1 else int(rng.choice([1, 1, 2]))
                layers.append(W.conv(int(rng.integers(1, 4)), f, s=s, p=int(rng.integers(0, f))))
            else:
                f = int(rng.choice([2, 3]))
                layers.append(W.maxpool(f, int(rng.choice([1, 2])), int(rng.integers(0, (f + 1) // 2))))
        h, w = int(rng.integers(min_extent, max_extent)), int(rng.integers(min_extent, max_extent))
        try:
            dims = orc.shapes(layers, h, w, 2)
        except orc.OracleError:
            continue
        ng = int(rng.integers(1, min(3, n) + 1))
        gs = [0] + sorted(int(v) for v in rng.choice(np.arange(1, n), ng - 1, replace=False)) if ng > 1 else [0]
        rows, rb = [], []
        for g in range(ng):
            last = (gs[g + 1] if g + 1 < ng else n) - 1
            H = int(dims[last, 3])
            rows.append(int(rng.integers(1, min(max_rows, H) + 1)))
            rb.append(_random_bounds(rng, H, rows[-1]))
        return layers, h, w, gs, rows, rb


# ------------------------------------------------------------------ brute force geometry

def _reads(L, r, E_in):
    """Input rows (inside the tensor) that output row r of layer L reads."""
    return [r * L["s"] + k - L["p"] for k in range(L["f"]) if 0 <= r * L["s"] + k - L["p"] < E_in]


def _geometry(layers, dims, g0, g1, bounds):
    """Row reuse in a group by brute force over the filter windows.  R[l]:
    where layer l's parts end (the group output's are the tile rows; an
    earlier layer's part i ends after the last row that the next layer's
    parts 0..i read); bands[l][i] = (lo, hi): tile row i's band of layer l's
    output -- from the first row its next layer's part reads (or its own
    first row) to the end of its own part.  None when a part is empty."""
    R = {g1: list(bounds)}
    for l in range(g1 - 1, g0 - 1, -1):
        nxt, E_in = R[l + 1], int(dims[l + 1, 0])
        cur = [0]
        for i in range(1, len(nxt)):
            rd = [y for r in range(nxt[i]) for y in _reads(layers[l + 1], r, E_in)]
            cur.append(max(rd) + 1 if rd else 0)
        R[l] = cur
    bands = {}
    for l in range(g0, g1):
        nxt, cur, E_in = R[l + 1], R[l], int(dims[l + 1, 0])
        bl = []
        for i in range(len(cur) - 1):
            rd = [y for r in range(nxt[i], nxt[i + 1]) for y in _reads(layers[l + 1], r, E_in)]
            if not rd or cur[i + 1] <= cur[i]:
                return None, None
            bl.append((min(min(rd), cur[i]), cur[i + 1]))
        bands[l] = bl
    return R, bands


# ------------------------------------------------------------------ oracle pins

def test_oracle_row_reuse_equals_untiled(orc):
    rng = np.random.default_rng(2301)
    for _ in range(150):
        layers, h, w, gs, rows, rb = _random_case(orc, rng)
        p = W.make_inputs(layers, h, w, 2, 2, seed=int(rng.integers(1 << 30)))
        ref = orc.forward_layers(layers, h, w, 2, p["x"], p)
        bounds = rb if rng.random() < 0.7 else None
        got, cuts = orc.forward_row_reuse(layers, h, w, 2, p["x"], p, gs, rows, want_cuts=True, row_bounds=bounds)
        assert np.array_equal(ref, got), (layers, h, w, gs, rows, bounds)
        for k, cut in enumerate(gs[1:]):
            assert np.array_equal(orc.forward_layers(layers, h, w, 2, p["x"], p, 0, cut - 1), cuts[k])


def test_oracle_row_reuse_yolo_equals_untiled(orc):
    # YOLOv2's layers 0-15 at 96x96 (the paper's stack on a small input),
    # one to four groups, bf16 rounding at every layer
    p = W.make_inputs(W.YOLOV2_16, 96, 96, 3, 1, seed=5)
    for rb in (False, True):
        ref = orc.forward_layers(W.YOLOV2_16, 96, 96, 3, p["x"], p, round_bf16=rb)
        for spec in ("3x3/NoCut", "5x5/8/2x2", "4x4/4/3x3/8/2x2/12/1x1", "6x6/NoCut"):
            gs, r, _ = W.parse_tiling(spec, 16)
            got = orc.forward_row_reuse(W.YOLOV2_16, 96, 96, 3, p["x"], p, gs, r, round_bf16=rb)
            assert np.array_equal(ref, got), (spec, rb)


def test_oracle_row_reuse_geometry_bruteforce(orc):
    rng = np.random.default_rng(2302)
    checked = 0
    for _ in range(400):
        layers, h, w, gs, rows, rb = _random_case(orc, rng)
        dims = orc.shapes(layers, h, w, 2)
        got = orc.row_reuse_band_rows(layers, h, w, 2, gs, rows, rb)
        want = np.zeros(len(layers), dtype=np.int64)
        ok = True
        for g, g0 in enumerate(gs):
            g1 = (gs[g + 1] if g + 1 < len(gs) else len(layers)) - 1
            _, bands = _geometry(layers, dims, g0, g1, rb[g])
            if bands is None:
                ok = False
                break
            for l, bl in bands.items():
                want[l] = max(hi - lo for lo, hi in bl)
        if not ok:
            continue
        assert np.array_equal(got, want), (layers, h, w, gs, rows, rb)
        checked += 1
    assert checked > 100


def test_oracle_row_reuse_yolo_bands_by_hand(orc):
    # YOLOv2 at 608x608, 5x5/8/2x2: the group-2 output (38 rows) in two tile
    # rows [0, 19, 38].  Layer 15 is 1x1 (its parts read their own rows),
    # layer 14 3x3 (one row either side): layer 14's parts end at 19 and 38,
    # layer 13's at 20 and 38; row 1's band of layer 13's output starts at
    # 18 (the first row layer 14's part [19, 38) reads), so it holds 20 rows;
    # row 0's holds [0, 20): 20 rows.
    gs, r, _ = W.parse_tiling("5x5/8/2x2", 16)
    band = orc.row_reuse_band_rows(W.YOLOV2_16, 608, 608, 3, gs, r)
    assert band[15] == 0 and band[7] == 0           # group outputs
    assert band[14] == 19                           # [0, 19) and [19, 38): the 1x1 reads its own rows
    assert band[13] == 20                           # [0, 20) and [18, 38)
    # layer 9 (1x1, 76 rows) feeds layer 10 (3x3) and the pool 11: layer 11's
    # parts end at 21 and 38 (layer 12 reads row 20), layer 10's at 42 and
    # 76, layer 9's at 43 and 76; row 1's band of layer 9 starts at 41
    assert band[9] == 43


def test_oracle_row_reuse_bad_arguments(orc):
    L = [W.conv(2, 3), W.maxpool(2, 2, 0)]
    x = np.zeros((1, 8, 8, 1))
    p = W.make_inputs(L, 8, 8, 1, 1, seed=1)
    with pytest.raises(orc.OracleError):
        orc.forward_row_reuse(L, 8, 8, 1, x, p, [0], [5])            # more tile rows than output rows
    with pytest.raises(orc.OracleError):
        orc.forward_row_reuse(L, 8, 8, 1, x, p, [0], [2], row_bounds=[[0, 3, 3]])
    with pytest.raises(orc.OracleError):
        orc.forward_row_reuse(L, 8, 8, 1, x, p, [1], [1])            # groups must start at layer 0


# ------------------------------------------------------------------ library (host)

@pytest.fixture(scope="module")
def M():
    import os
    from paper_2107_06960_amd import mafat
    if not os.path.exists(mafat.LIB_PATH):
        from paper_2107_06960_amd import build
        build.build(verbose=False)
    mafat.lib()
    return mafat


def _stage_ends(layers, g0, g1):
    """Last layer of every stage of the library's group [g0, g1]: a
    convolution followed (inside the group) by a 2x2/2 max-pool is one
    stage with it."""
    ends, l = [], g0
    while l <= g1:
        pool2 = (l + 1 <= g1 and layers[l]["op"] == W.CONV and layers[l + 1]["op"] == W.MAXPOOL and
                 layers[l + 1]["f"] == 2 and layers[l + 1]["s"] == 2 and layers[l + 1]["p"] == 0)
        ends.append(l + 1 if pool2 else l)
        l = ends[-1] + 1
    return ends


def _expected_workspace(layers, dims, gs, rb, batch, esz):
    """Row reuse in float32 (no stage output kept on chip): every stage
    output but the group's has its bands, each band_rows x width x channels,
    rounded up to 128 elements; one buffer where every row's taken-over rows
    move to rows that do not overlap them, else two.  The largest group."""
    best = 0
    for g, g0 in enumerate(gs):
        g1 = (gs[g + 1] if g + 1 < len(gs) else len(layers)) - 1
        R, bands = _geometry(layers, dims, g0, g1, rb[g])
        if bands is None:
            return None
        frame = 0
        for e in _stage_ends(layers, g0, g1)[:-1]:
            bl = bands[e]
            rows = max(hi - lo for lo, hi in bl)
            one = all(R[e][i] - bl[i][0] <= bl[i][0] - bl[i - 1][0] for i in range(1, len(bl)))
            frame += (1 if one else 2) * ((rows * int(dims[e, 4]) * int(dims[e, 5]) + 127) // 128 * 128)
        best = max(best, (batch * frame * esz + 255) // 256 * 256)
    return best


def test_library_row_reuse_workspace_matches_bruteforce(M, orc):
    cases = [(W.YOLOV2_16, 608, 608, 3, spec) for spec in ("5x5/8/2x2", "4x4/12/1x1", "3x3/NoCut", "8x8/8/4x4",
                                                           "2x2/4/3x3/8/2x2/12/2x2")]
    for layers, h, w, c, spec in cases:
        gs, r, cc = W.parse_tiling(spec, len(layers))
        dims = orc.shapes(layers, h, w, c)
        rb = [[int(v) for v in np.floor(np.arange(r[g] + 1) * dims[(gs[g + 1] if g + 1 < len(gs) else 16) - 1, 3]
                                            / r[g])] for g in range(len(gs))]
        plan = M.Plan(layers, (h, w, c), spec, row_reuse=True)
        for batch in (1, 3):
            assert plan.workspace_size(batch, "f32") == _expected_workspace(layers, dims, gs, rb, batch, 4), spec
    rng = np.random.default_rng(2303)
    checked = 0
    for _ in range(300):
        layers, h, w, gs, rows, rb = _random_case(orc, rng, max_extent=40)
        dims = orc.shapes(layers, h, w, 2)
        want = _expected_workspace(layers, dims, gs, rb, 2, 4)
        if want is None:
            continue
        cols = [1] * len(gs)
        plan = M.Plan(layers, (h, w, 2), (gs, rows, cols), bounds=(rb, None), row_reuse=True)
        assert plan.workspace_size(2, "f32") == want, (layers, h, w, gs, rows, rb)
        checked += 1
    assert checked > 100


def test_library_row_reuse_macs_and_memory_models(M):
    for spec in ("5x5/8/2x2", "4x4/12/1x1", "3x3/NoCut"):
        plan = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, row_reuse=True, packed_weights=True)
        for g in range(plan.n_groups):
            executed, untiled = plan.macs(g)
            assert executed == untiled, spec
        # the tile rows already run one after another: both device models agree
        dev = M.mafat_predict_mem(plan.handle, M.MAFAT_MEM_DEVICE, 1, M.MAFAT_BF16)
        seq = M.mafat_predict_mem(plan.handle, M.MAFAT_MEM_DEVICE_SEQ, 1, M.MAFAT_BF16)
        assert dev == seq
        plain = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, packed_weights=True)
        assert plan.workspace_size(1, "bf16") < plain.workspace_size(1, "bf16"), spec
    # bf16 keeps the fused pairs' first outputs on chip: no bands for them
    p32 = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/NoCut", row_reuse=True)
    assert p32.workspace_size(1, "bf16") < p32.workspace_size(1, "f32") // 2


def test_library_row_reuse_errors(M):
    L = W.YOLOV2_16
    gs, r, c = W.parse_tiling("3x3/8/2x2", 16)
    with pytest.raises(M.MafatError) as e:
        M.mafat_plan_create(L, 608, 608, 3, gs, r, c, M.MAFAT_PLAN_STAGE_PARTITION | M.MAFAT_PLAN_ROW_REUSE)
    assert e.value.rc == M.MAFAT_EUNSUPPORTED
    plan = M.Plan(L, (608, 608, 3), "3x3/8/2x2", row_reuse=True)
    with pytest.raises(M.MafatError) as e:
        M.mafat_plan_set_tile_batch(plan.handle, 2)
    assert e.value.rc == M.MAFAT_EUNSUPPORTED
    rc = M.lib().mafat_run_stage(plan.handle, 0, 0, 1, M.MAFAT_F32, None, None, None, None, None, None, 0, None)
    assert rc == M.MAFAT_EUNSUPPORTED
    # with given boundaries: the plan follows them
    rb = [[0, 30, 50, 76], [0, 19, 38]]
    M.Plan(L, (608, 608, 3), "3x3/8/2x2", bounds=(rb, None), row_reuse=True)


# ------------------------------------------------------------------ GPU parity

@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("spec,hw,batch,packed", [
    ("5x5/8/2x2", (160, 160), 1, True),
    ("3x3/NoCut", (96, 128), 2, False),
    ("4x4/4/3x3/8/2x2/12/1x1", (200, 168), 2, True),
    ("6x5/8/3x2", (142, 190), 1, False),
    ("2x2/12/2x2", (64, 64), 2, True),
])
def test_gpu_row_reuse_parity(orc, dtype, spec, hw, batch, packed):
    require_gpu()
    h, w = hw
    layers = W.YOLOV2_16
    if dtype == "f32":
        packed = False
    print(f"[row reuse] {h}x{w}x3 {spec} batch={batch} {dtype} packed={packed}", flush=True)
    p = W.make_inputs(layers, h, w, 3, batch, seed=41, dtype=dtype)
    out, cuts, net, _ = run_gpu(layers, h, w, 3, p, spec, batch, dtype, reuse=True, packed=packed)
    gs, _, _ = W.parse_tiling(spec, 16)
    ref = orc.forward_layers(layers, h, w, 3, p["x"], p)
    assert not np.isnan(out).any()
    err = normwise_err(out, ref)
    print(f"[row reuse] normwise output {err:.3e}", flush=True)
    assert err <= TOL[dtype]
    for k, cut in enumerate(gs[1:]):
        rc = orc.forward_layers(layers, h, w, 3, p["x"], p, 0, cut - 1)
        assert not np.isnan(cuts[k]).any()
        assert normwise_err(cuts[k], rc) <= TOL[dtype], (k, cut)
    # the plain fused tile partition on the same inputs agrees as closely
    plain = run_gpu(layers, h, w, 3, p, spec, batch, dtype, want_cuts=False, packed=packed)
    assert normwise_err(out, plain) <= TOL[dtype]


@pytest.mark.gpu
def test_gpu_row_reuse_random_stacks(orc):
    """Random stacks of every supported layer kind, random tile rows, row
    boundaries and columns, f32 and bf16."""
    require_gpu()
    rng = np.random.default_rng(2304)
    for k in range(12):
        while True:
            layers, h, w, gs, rows, rb = _random_case(orc, rng, max_extent=48)
            if any(L["op"] == W.CONV for L in layers):
                break
        layers = [dict(L, c_out=int(rng.choice([16, 32, 48]))) if L["op"] == W.CONV else L for L in layers]
        dims = orc.shapes(layers, h, w, 32)
        cols = [int(rng.integers(1, min(4, int(dims[(gs[g + 1] if g + 1 < len(gs) else len(layers)) - 1, 4])) + 1))
                for g in range(len(gs))]
        dtype = "bf16" if k % 2 else "f32"
        print(f"[row reuse random {k}] {h}x{w}x32 {dtype} layers={[(L['op'], L.get('c_out'), L['f'], L['s'], L['p']) for L in layers]} "
              f"groups={gs} rows={rows} cols={cols} bounds={rb}", flush=True)
        p = W.make_inputs(layers, h, w, 32, 2, seed=100 + k, dtype=dtype)
        out = run_gpu(layers, h, w, 32, p, (gs, rows, cols), 2, dtype, want_cuts=False, bounds=(rb, None),
                      reuse=True)
        ref = orc.forward_layers(layers, h, w, 32, p["x"], p)
        assert not np.isnan(out).any()
        assert normwise_err(out, ref) <= TOL[dtype], k


def test_library_search_with_row_reuse(M):
    # Algorithm 2 over candidates planned with row reuse (mafat_get_config_flags)
    # = the first candidate, in the paper's order, whose row-reuse plan's
    # device-model prediction plus the bias is below the limit
    layers, hwc = W.YOLOV2_16, (608, 608, 3)
    order = [(16, t) for t in (1, 2, 3, 4, 5)] + [(c, t) for c in (12, 8) for t in (1, 2, 3, 4, 5)]
    spec = lambda cut, t: f"{t}x{t}/NoCut" if cut == 16 else f"{t}x{t}/{cut}/2x2"
    pred = {k: M.Plan(layers, hwc, spec(*k), row_reuse=True).predict_mem("device", 1, "bf16") for k in order}
    for mib in (8, 12, 13, 14, 16, 20, 40):
        got, p, fits = M.mafat_get_config(layers, hwc, mib << 20, model="device", dtype="bf16",
                                          flags=M.MAFAT_PLAN_ROW_REUSE)
        first = next((k for k in order if pred[k] < (mib << 20)), None)
        if first is None:
            assert not fits and got == spec(*order[-1]), mib
        else:
            assert fits and got == spec(*first) and p == pred[first], (mib, got, first)
    # with balanced boundaries too
    got, p, fits = M.mafat_get_config(layers, hwc, 14 << 20, model="device", dtype="bf16",
                                      flags=M.MAFAT_PLAN_ROW_REUSE, balanced=True)
    assert fits and p < 14 << 20
    with pytest.raises(M.MafatError):
        M.mafat_get_config(layers, hwc, 14 << 20, model="device", flags=M.MAFAT_PLAN_ROW_REUSE |
                           M.MAFAT_PLAN_STAGE_PARTITION)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gpu_row_reuse_wide_rows(orc, dtype):
    """Tile rows of more tiles than one launch describes (70 per row: two
    launches per stage and row), three rows, batch 2."""
    require_gpu()
    layers, (h, w, c) = W.TINY, (40, 600, 3)
    gs, rows, cols = [0], [3], [70]
    print(f"[row reuse] {h}x{w}x{c} 3x70 batch=2 {dtype}", flush=True)
    p = W.make_inputs(layers, h, w, c, 2, seed=43, dtype=dtype)
    out = run_gpu(layers, h, w, c, p, (gs, rows, cols), 2, dtype, want_cuts=False, reuse=True)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    assert not np.isnan(out).any()
    assert normwise_err(out, ref) <= TOL[dtype]


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gpu_row_reuse_odd_channels(orc, dtype):
    """Channel counts whose band rows are not whole 16-byte pieces (3, 5, 7
    channels): the take-over copies then run as copy launches of their own
    (2-byte pieces) instead of riding in a stage launch."""
    require_gpu()
    layers = [W.conv(5, 3), W.conv(7, 3), W.maxpool(2, 2, 0), W.conv(3, 3), W.conv(5, 1)]
    h, w, c = 45, 37, 3
    gs, rows, cols = [0, 3], [4, 3], [2, 1]
    print(f"[row reuse] odd channels {h}x{w}x{c} batch=2 {dtype}", flush=True)
    p = W.make_inputs(layers, h, w, c, 2, seed=47, dtype=dtype)
    out = run_gpu(layers, h, w, c, p, (gs, rows, cols), 2, dtype, want_cuts=False, reuse=True)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    assert not np.isnan(out).any()
    assert normwise_err(out, ref) <= TOL[dtype]
