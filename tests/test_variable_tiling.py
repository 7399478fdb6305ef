"""Variable tiling (section 6 proposes it as future work: end tiles sized
unlike the inner ones, so that the tasks vary less and the largest footprint
falls).

Oracle pins (CPU): tile regions with given boundaries against receptive-field
brute force; the tiled forward with given boundaries equals the untiled
forward bit for bit (fused tile partitioning is exact for any partition);
the brute-force balanced boundaries against closed forms (stacks without a
halo; YOLOv2's first group, whose task extents are derived by hand below)
and against properties any optimum has.
"""
import itertools

import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W


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
