"""Variable tiling (section 6 proposes it as future work: end tiles sized
unlike the inner ones, so that the tasks vary less and the largest footprint
falls).

Oracle pins (CPU): tile regions with given boundaries against receptive-field
brute force; the tiled forward with given boundaries equals the untiled
forward bit for bit (fused tile partitioning is exact for any partition);
the brute-force balanced boundaries against closed forms (stacks without a
halo; YOLOv2's first group, whose task extents are derived by hand below)
and against properties any optimum has.

Library (CPU, through the C ABI): mafat_balanced_bounds equals the oracle's
brute force; plans made with mafat_plan_create_bounds have the oracle's
regions; the error codes.

GPU: the library with balanced and with random boundaries against the
oracle's tiled forward with the same boundaries, f32 and bf16.
"""
import itertools

import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu, run_gpu


def _random_bounds(rng, E, N):
    inner = sorted(int(v) for v in rng.choice(np.arange(1, E), N - 1, replace=False)) if N > 1 else []
    return [0] + inner + [E]


def _random_case(orc, rng, max_parts=5, min_extent=4, max_extent=24):
    while True:
        n = int(rng.integers(1, 5))
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
        rows, cols, rb, cb = [], [], [], []
        for g in range(ng):
            last = (gs[g + 1] if g + 1 < ng else n) - 1
            H, Wd = int(dims[last, 3]), int(dims[last, 4])
            rows.append(int(rng.integers(1, min(max_parts, H) + 1)))
            cols.append(int(rng.integers(1, min(max_parts, Wd) + 1)))
            rb.append(_random_bounds(rng, H, rows[-1]))
            cb.append(_random_bounds(rng, Wd, cols[-1]))
        return layers, h, w, gs, rows, cols, rb, cb


# ------------------------------------------------------------------ oracle pins

def test_oracle_bounds_regions_equal_bruteforce(orc):
    rng = np.random.default_rng(606)
    for _ in range(250):
        layers, h, w, gs, rows, cols, rb, cb = _random_case(orc, rng)
        A = orc.regions(layers, h, w, 2, gs, rows, cols, rb, cb)
        B = orc.regions_bruteforce(layers, h, w, 2, gs, rows, cols, rb, cb)
        for g, (a, b) in enumerate(zip(A, B)):
            assert np.array_equal(a, b), (layers, h, w, gs, rows, cols, rb, cb)
            # the tiles' outputs at the group's last layer are the given boundaries
            for i in range(rows[g]):
                for j in range(cols[g]):
                    assert list(a[i * cols[g] + j, -1, 4:]) == [rb[g][i], rb[g][i + 1], cb[g][j], cb[g][j + 1]]


def test_oracle_floor_bounds_equal_even_split(orc):
    gs, r, c = W.parse_tiling("5x5/8/2x2", 16)
    dims = orc.shapes(W.YOLOV2_16, 608, 608, 3)
    rb, cb = [], []
    for g in range(len(gs)):
        last = (gs[g + 1] if g + 1 < len(gs) else 16) - 1
        rb.append([i * int(dims[last, 3]) // r[g] for i in range(r[g] + 1)])
        cb.append([j * int(dims[last, 4]) // c[g] for j in range(c[g] + 1)])
    A = orc.regions(W.YOLOV2_16, 608, 608, 3, gs, r, c)
    B = orc.regions(W.YOLOV2_16, 608, 608, 3, gs, r, c, rb, cb)
    for a, b in zip(A, B):
        assert np.array_equal(a, b)


def test_oracle_tiled_bounds_equal_untiled(orc):
    rng = np.random.default_rng(707)
    for _ in range(100):
        layers, h, w, gs, rows, cols, rb, cb = _random_case(orc, rng)
        p = W.make_inputs(layers, h, w, 2, 2, seed=int(rng.integers(1 << 30)))
        ref = orc.forward_layers(layers, h, w, 2, p["x"], p)
        got, cuts = orc.forward_tiled(layers, h, w, 2, p["x"], p, gs, rows, cols, want_cuts=True,
                                      row_bounds=rb, col_bounds=cb)
        assert np.array_equal(ref, got), (layers, h, w, gs, rows, cols, rb, cb)
        for k, cut in enumerate(gs[1:]):
            assert np.array_equal(orc.forward_layers(layers, h, w, 2, p["x"], p, 0, cut - 1), cuts[k])


def test_oracle_bad_bounds_are_errors(orc):
    L = [W.conv(2, 3)]
    for rb in ([[0, 3, 3, 8]], [[1, 4, 8]], [[0, 4, 7]], [[0, 5, 4, 8]]):
        with pytest.raises(orc.OracleError):
            orc.regions(L, 8, 8, 1, [0], [len(rb[0]) - 1], [1], rb, None)
    with pytest.raises(orc.OracleError):
        orc.balanced_bounds(L, 8, 8, 1, 0, 0, 0, 9)   # more parts than rows


def _task_extents(orc, layers, h, w, c, g0, g1, axis, bounds):
    """Task extents of the parts along one axis, from the oracle's regions of
    a one-group plan over layers [g0, g1] (the group input is layer g0's)."""
    dims = orc.shapes(layers, h, w, c)
    sub = layers[g0:g1 + 1]
    hh, ww, cc = (int(v) for v in dims[g0, :3])
    N = len(bounds) - 1
    rb = [bounds] if axis == 0 else None
    cb = [bounds] if axis == 1 else None
    R = orc.regions(sub, hh, ww, cc, [0], [N if axis == 0 else 1], [N if axis == 1 else 1], rb, cb)[0]
    lo, hi = (0, 1) if axis == 0 else (2, 3)
    return [int(R[t, 0, hi] - R[t, 0, lo]) for t in range(N)]


def test_balanced_without_halo_is_the_most_even_split(orc):
    # 1x1 convolutions and 2x2/2 pools read no halo: a part of k output rows
    # has a task of k * (product of strides) rows, so the optimum is the most
    # even split, the shorter parts first (first in lexicographic order)
    stacks = [[W.conv(3, 1)], [W.maxpool(), W.conv(2, 1)], [W.conv(2, 1), W.maxpool(), W.maxpool()]]
    for layers in stacks:
        for E in (5, 7, 12, 13):
            h = E * (4 if len(layers) == 3 else 2 if len(layers) == 2 else 1)
            dims = orc.shapes(layers, h, h, 2)
            assert dims[-1, 3] == E
            for N in range(1, min(E, 6) + 1):
                q, r = divmod(E, N)
                sizes = [q] * (N - r) + [q + 1] * r
                want = [0] + list(itertools.accumulate(sizes))
                got = orc.balanced_bounds(layers, h, h, 2, 0, len(layers) - 1, 0, N)
                assert list(got) == want, (layers, E, N, got)


def _yolo_group1_task(a, b):
    # YOLOv2 layers 0-7 at 608x608 (conv3, pool, conv3, pool, conv3, conv1,
    # conv3, pool; 76 output rows).  Back-projecting output rows [a, b):
    # pool -> [2a, 2b); conv3 p1 -> [2a-1, 2b+1); conv1 -> same;
    # conv3 -> [2a-2, 2b+2); pool -> [4a-4, 4b+4); conv3 -> [4a-5, 4b+5);
    # pool -> [8a-10, 8b+10); conv3 -> [8a-11, 8b+11); clipped to [0, 608).
    return min(608, 8 * b + 11) - max(0, 8 * a - 11)


def _best_by_enumeration(task, E, N):
    best = None
    for inner in itertools.combinations(range(1, E), N - 1):
        b = (0,) + inner + (E,)
        t = [task(b[i], b[i + 1]) for i in range(N)]
        key = (max(t), sum(v * v for v in t))
        if best is None or key < best[0]:
            best = (key, list(b))
    return best


def test_balanced_yolo_group1_closed_form(orc):
    # by hand from the task formula above: an end part of k rows reads 8k+11
    # input rows, an inner part 8k+22; three parts 26/24/26 -> 219/214/219,
    # four 20/18/18/20 -> 171/166/166/171, five 16/14/15/15/16 ->
    # 139/134/142/142/139 (the even split 15/15/15/15/16 also peaks at 142
    # but has the larger sum of squares)
    hand = {3: [0, 26, 50, 76], 4: [0, 20, 38, 56, 76], 5: [0, 16, 30, 45, 60, 76]}
    peaks = {3: 219, 4: 171, 5: 142}
    for N in (1, 2, 3, 4, 5):
        key, bounds = _best_by_enumeration(_yolo_group1_task, 76, N)
        got = list(orc.balanced_bounds(W.YOLOV2_16, 608, 608, 3, 0, 7, 0, N))
        assert got == bounds, (N, got, bounds)
        assert [_yolo_group1_task(got[i], got[i + 1]) for i in range(N)] == \
            _task_extents(orc, W.YOLOV2_16, 608, 608, 3, 0, 7, 0, got)
        if N in hand:
            assert got == hand[N] and key[0] == peaks[N]
        # columns: the stack is square and symmetric
        assert list(orc.balanced_bounds(W.YOLOV2_16, 608, 608, 3, 0, 7, 1, N)) == got


def test_balanced_properties_random(orc):
    # any optimum: its largest task is at most the even split's, and its
    # mirror image (for a stack whose back-projection is mirror-symmetric:
    # stride 1, padding (f-1)/2, odd filters, extents that map exactly) has
    # the same largest task and sum of squares
    rng = np.random.default_rng(808)
    for _ in range(60):
        layers, h, w, gs, rows, cols, _, _ = _random_case(orc, rng, max_extent=30)
        n = len(layers)
        g0 = int(rng.integers(0, n))
        dims = orc.shapes(layers, h, w, 2)
        E = int(dims[-1, 3])
        N = int(rng.integers(1, min(E, 5) + 1))
        bal = list(orc.balanced_bounds(layers, h, w, 2, g0, n - 1, 0, N))
        even = [i * E // N for i in range(N + 1)]
        tb = _task_extents(orc, layers, h, w, 2, g0, n - 1, 0, bal)
        te = _task_extents(orc, layers, h, w, 2, g0, n - 1, 0, even)
        assert max(tb) <= max(te)
        assert (max(tb), sum(v * v for v in tb)) <= (max(te), sum(v * v for v in te))
    sym = [W.conv(2, 3), W.conv(2, 5), W.conv(2, 1), W.conv(2, 3)]
    for E in (9, 16, 23):
        for N in (2, 3, 4):
            bal = list(orc.balanced_bounds(sym, E, E, 2, 0, 3, 0, N))
            mir = [E - v for v in reversed(bal)]
            tb = _task_extents(orc, sym, E, E, 2, 0, 3, 0, bal)
            tm = _task_extents(orc, sym, E, E, 2, 0, 3, 0, mir)
            assert (max(tb), sum(v * v for v in tb)) == (max(tm), sum(v * v for v in tm))
            assert bal <= mir   # the first in lexicographic order


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


def test_library_balanced_bounds_match_oracle(M, orc):
    for g0, g1 in ((0, 7), (0, 11), (0, 15), (8, 15), (12, 15)):
        for N in (1, 2, 3, 4, 5):
            rb, cb = M.mafat_balanced_bounds(W.YOLOV2_16, 608, 608, 3, g0, g1, N, N)
            assert rb == list(orc.balanced_bounds(W.YOLOV2_16, 608, 608, 3, g0, g1, 0, N)), (g0, g1, N)
            assert cb == list(orc.balanced_bounds(W.YOLOV2_16, 608, 608, 3, g0, g1, 1, N)), (g0, g1, N)
    rng = np.random.default_rng(909)
    done = 0
    while done < 300:
        layers, h, w, _, _, _, _, _ = _random_case(orc, rng, max_extent=40)
        n = len(layers)
        g0 = int(rng.integers(0, n))
        dims = orc.shapes(layers, h, w, 2)
        R = int(rng.integers(1, min(int(dims[-1, 3]), 5) + 1))
        C = int(rng.integers(1, min(int(dims[-1, 4]), 5) + 1))
        rb, cb = M.mafat_balanced_bounds(layers, h, w, 2, g0, n - 1, R, C)
        assert rb == list(orc.balanced_bounds(layers, h, w, 2, g0, n - 1, 0, R)), (layers, h, w, g0, R)
        assert cb == list(orc.balanced_bounds(layers, h, w, 2, g0, n - 1, 1, C)), (layers, h, w, g0, C)
        done += 1


def test_library_bounds_plan_regions_match_oracle(M, orc):
    rng = np.random.default_rng(1010)
    for _ in range(150):
        layers, h, w, gs, rows, cols, rb, cb = _random_case(orc, rng, max_extent=40)
        plan = M.Plan(layers, (h, w, 2), (gs, rows, cols), bounds=(rb, cb))
        B = orc.regions_bruteforce(layers, h, w, 2, gs, rows, cols, rb, cb)
        for g in range(len(gs)):
            assert np.array_equal(plan.regions(g), B[g]), (layers, h, w, gs, rows, cols, rb, cb)
    # only rows given: columns split evenly
    gs, r, c = W.parse_tiling("5x5/8/2x2", 16)
    rows_only = M.Plan(W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2", bounds=([[0, 16, 30, 45, 60, 76], [0, 19, 38]], None))
    want = orc.regions(W.YOLOV2_16, 608, 608, 3, gs, r, c, [[0, 16, 30, 45, 60, 76], [0, 19, 38]], None)
    for g in range(2):
        assert np.array_equal(rows_only.regions(g), want[g])


def test_library_balanced_plan(M, orc):
    # Plan(bounds="balanced") takes each group's mafat_balanced_bounds; the
    # largest tile input region is never larger than the even split's
    for spec in ("3x3/NoCut", "5x5/8/2x2", "4x4/12/2x2", "3x3/8/2x2"):
        even = M.Plan(W.YOLOV2_16, (608, 608, 3), spec)
        bal = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, bounds="balanced")
        gs, r, c = W.parse_tiling(spec, 16)
        for g in range(len(gs)):
            g1 = (gs[g + 1] if g + 1 < len(gs) else 16) - 1
            rb, cb = M.mafat_balanced_bounds(W.YOLOV2_16, 608, 608, 3, gs[g], g1, r[g], c[g])
            assert bal.bounds[0][g] == rb and bal.bounds[1][g] == cb
            Rb, Re = bal.regions(g), even.regions(g)
            area = lambda R: (R[:, 0, 1] - R[:, 0, 0]) * (R[:, 0, 3] - R[:, 0, 2])
            assert area(Rb).max() <= area(Re).max(), spec


def test_library_bounds_errors(M):
    L = W.YOLOV2_16
    gs, r, c = W.parse_tiling("3x3/8/2x2", 16)
    bad_rows = (
        [[0, 30, 30, 76], [0, 19, 38]],   # not strictly increasing
        [[0, 30, 50, 75], [0, 19, 38]],   # does not end at the extent
        [[1, 30, 50, 76], [0, 19, 38]],   # does not start at 0
    )
    for rb in bad_rows:
        with pytest.raises(M.MafatError) as e:
            M.mafat_plan_create(L, 608, 608, 3, gs, r, c, 0, row_bounds=rb, col_bounds=None)
        assert e.value.rc == M.MAFAT_ESHAPE
    with pytest.raises(M.MafatError) as e:
        M.mafat_plan_create(L, 608, 608, 3, gs, r, c, M.MAFAT_PLAN_STAGE_PARTITION,
                            row_bounds=[[0, 26, 50, 76], [0, 19, 38]], col_bounds=None)
    assert e.value.rc == M.MAFAT_EUNSUPPORTED
    with pytest.raises(M.MafatError) as e:
        M.mafat_balanced_bounds(L, 608, 608, 3, 0, 7, 77, 1)   # more parts than rows
    assert e.value.rc == M.MAFAT_ESHAPE
    with pytest.raises(M.MafatError) as e:
        M.mafat_balanced_bounds(L, 608, 608, 3, 8, 7, 2, 2)    # empty layer range
    assert e.value.rc == M.MAFAT_EINVAL
    with pytest.raises(ValueError):
        M.Plan(L, (608, 608, 3), "3x3/8/2x2", bounds="uneven")


# ------------------------------------------------------------------ GPU parity

@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["balanced", "random"])
def test_gpu_variable_tiling_parity(orc, dtype, kind):
    require_gpu()
    rng = np.random.default_rng(1111)
    h = w = 160
    layers = W.YOLOV2_16
    spec = "5x5/8/3x3"
    gs, r, c = W.parse_tiling(spec, 16)
    if kind == "balanced":
        bounds = "balanced"
    else:
        dims = orc.shapes(layers, h, w, 3)
        rb, cb = [], []
        for g in range(len(gs)):
            last = (gs[g + 1] if g + 1 < len(gs) else 16) - 1
            rb.append(_random_bounds(rng, int(dims[last, 3]), r[g]))
            cb.append(_random_bounds(rng, int(dims[last, 4]), c[g]))
        bounds = (rb, cb)
    print(f"[variable tiling] {h}x{w}x3 {spec} {kind} {dtype}", flush=True)
    p = W.make_inputs(layers, h, w, 3, 2, seed=31, dtype=dtype)
    out, cuts, net, _ = run_gpu(layers, h, w, 3, p, spec, 2, dtype, bounds=bounds)
    rb, cb = net.plan.bounds
    print(f"[variable tiling] row bounds {rb} col bounds {cb}", flush=True)
    ref, rcuts = orc.forward_tiled(layers, h, w, 3, p["x"], p, gs, r, c, want_cuts=True,
                                   row_bounds=rb, col_bounds=cb)
    assert not np.isnan(out).any()
    err = normwise_err(out, ref)
    cerr = normwise_err(cuts[0], rcuts[0])
    print(f"[variable tiling] normwise output {err:.3e} cut {cerr:.3e}", flush=True)
    assert err <= TOL[dtype] and cerr <= TOL[dtype]


# ------------------------------------------------------------------ predictor and search

def test_paper_model_with_bounds_matches_oracle(M):
    from oracle import predictor as P
    rng = np.random.default_rng(1212)
    for spec in ("3x3/NoCut", "5x5/NoCut", "4x4/12/2x2", "5x5/8/2x2"):
        gs, r, c = W.parse_tiling(spec, 16)
        bal = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, bounds="balanced")
        rb, cb = bal.bounds
        assert bal.predict_mem("paper", 1, "f32") == 4 * P.predict_mem(W.YOLOV2_16, 608, 608, 3, gs, r, c, rb, cb)
        heights = [bal.group_out_shape(g)[0] for g in range(len(gs))]
        rrb = [_random_bounds(rng, e, k) for e, k in zip(heights, r)]
        rnd = M.Plan(W.YOLOV2_16, (608, 608, 3), spec, bounds=(rrb, None))
        assert rnd.predict_mem("paper", 1, "bf16") == \
            2 * P.predict_mem(W.YOLOV2_16, 608, 608, 3, gs, r, c, rrb, None)


@pytest.mark.parametrize("mb", [40, 45, 50, 55, 64])
def test_balanced_search_matches_oracle(M, mb):
    # Algorithm 2 with every candidate balanced (the paper's model, float32,
    # bias 31 MiB, 608x608): the library's search equals the oracle's; at
    # these limits the balanced search stops no later in Algorithm 2's order
    # than the even one (its predictions are lower on the deep groups)
    from oracle import predictor as P
    MiB = 1 << 20
    spec, pred, fits = M.mafat_get_config(W.YOLOV2_16, (608, 608, 3), mb * MiB, model="paper", dtype="f32",
                                          bias_bytes=31 * MiB, balanced=True)
    cut, t, g2, opred, ofits = P.get_config(W.YOLOV2_16, 608, 608, 3, mb * MiB, balanced_tiles=True)
    ospec = f"{t}x{t}/NoCut" if cut == 16 else f"{t}x{t}/{cut}/{g2}x{g2}"
    assert (ospec, opred, ofits) == (spec, pred, fits)
    even, epred, efits = M.mafat_get_config(W.YOLOV2_16, (608, 608, 3), mb * MiB, model="paper", dtype="f32",
                                            bias_bytes=31 * MiB)
    print(f"{mb} MiB: even tiles {even} ({epred / MiB:.2f} MiB), balanced {spec} ({pred / MiB:.2f} MiB)")
    assert fits or not efits
    order = [f"{t}x{t}/NoCut" for t in range(1, 6)] + [f"{t}x{t}/{c}/2x2" for c in (12, 8) for t in range(1, 6)]
    if fits and efits:
        assert order.index(spec) <= order.index(even)


def test_library_balanced_bounds_large_extents(M):
    # the largest extents the plan takes: the windowed search stays exact
    # (a halo-free stack: the most even split, shorter parts first) and quick
    import time
    t0 = time.perf_counter()
    for E, N in ((32767, 64), (32767, 7), (32767, 1), (30000, 30000 // 2)):
        rb, _ = M.mafat_balanced_bounds([W.conv(2, 1)], E, 2, 1, 0, 0, N, 1)
        q, r = divmod(E, N)
        assert [rb[i + 1] - rb[i] for i in range(N)] == [q] * (N - r) + [q + 1] * r
    # a stack with halos at a large extent: never worse than the even split
    layers = [W.conv(2, 3), W.maxpool(), W.conv(2, 5), W.conv(2, 3, s=2, p=1)]
    h = 32000
    plan = M.Plan(layers, (h, 8, 1), "1x1/NoCut")
    E = plan.group_out_shape(0)[0]
    rb, _ = M.mafat_balanced_bounds(layers, h, 8, 1, 0, 3, 17, 1)
    even = [i * E // 17 for i in range(18)]

    def largest_task(bounds):
        R = M.Plan(layers, (h, 8, 1), ([0], [17], [1]), bounds=([bounds], None)).regions(0)
        return int((R[:, 0, 1] - R[:, 0, 0]).max())

    assert largest_task(rb) <= largest_task(even)
    assert time.perf_counter() - t0 < 30
