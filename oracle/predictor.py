"""The paper's memory predictor (Algorithm 1, section 4.1) and configuration
search (Algorithm 2, section 4.2), written from their description in plain
Python on top of the oracle's region tables.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``; the product path never
imports it.  It shares no code with the library (``mafat_predict_mem`` /
``mafat_get_config``), which the tests compare against it.

Readings (where the paper is silent or garbled):
  * "Grid" (the traversal function the paper takes from DeepThings) is the
    exact receptive-field back-projection of each tile through the group,
    clipped to the tensor: the oracle's ``regions``, pinned by brute force.
  * The loop over layers in Algorithm 1 visits every layer of the group
    (its printed bounds run from the bottom layer while l <= top, which
    visits none); tiles run over i in [0, N), j in [0, M).
  * scratch = w_out * h_out * c_in * F^2 / S uses integer division by S; it
    applies to every layer as written (a max-pool layer too).
  * Algorithm 2's "LG2 <- 4" is a 2 x 2 second-group grid (four tiles);
    "cut 16" on the 16-layer network means no cut; its unused getMaxLayer
    call is ignored.
  * Variable tiling (proposed in section 6): the same predictor and search
    over tiles with given boundaries; the search's balanced variant takes
    each group's brute-force balanced boundaries (``oracle.balanced_bounds``).
"""
from __future__ import annotations

from . import oracle as O


def predict_layer_group(layers, h, w, c, group_start, rows, cols, g, row_bounds=None, col_bounds=None):
    """Algorithm 1 for group g of a configuration: the largest, over the
    group's tiles and layers, of scratch + output + 2 * input, in elements
    (the caller multiplies by the element size and adds the bias).
    row_bounds / col_bounds: per-group tile boundaries, or None (even)."""
    dims = O.shapes(layers, h, w, c)
    R = O.regions(layers, h, w, c, group_start, rows, cols, row_bounds, col_bounds)[g]
    best = 0
    n_tiles, n_lay = R.shape[0], R.shape[1]
    for t in range(n_tiles):
        for k in range(n_lay):
            l = group_start[g] + k
            iy0, iy1, ix0, ix1, oy0, oy1, ox0, ox1 = (int(v) for v in R[t, k])
            w_in, h_in = ix1 - ix0, iy1 - iy0
            w_out, h_out = ox1 - ox0, oy1 - oy0
            c_in, c_out = int(dims[l, 2]), int(dims[l, 5])
            f, s = layers[l]["f"], layers[l]["s"]
            scratch = w_out * h_out * c_in * f * f // s
            inp = w_in * h_in * c_in
            out = w_out * h_out * c_out
            mem = scratch + out + inp * 2
            if mem > best:
                best = mem
    return best


def predict_mem(layers, h, w, c, group_start, rows, cols, row_bounds=None, col_bounds=None):
    """A configuration's prediction: the maximum over its layer groups."""
    return max(predict_layer_group(layers, h, w, c, group_start, rows, cols, g, row_bounds, col_bounds)
               for g in range(len(group_start)))


def balanced(layers, h, w, c, group_start, rows, cols):
    """Each group's balanced row and column boundaries (brute force)."""
    n = len(layers)
    rb, cb = [], []
    for g, g0 in enumerate(group_start):
        g1 = (group_start[g + 1] if g + 1 < len(group_start) else n) - 1
        rb.append([int(v) for v in O.balanced_bounds(layers, h, w, c, g0, g1, 0, rows[g])])
        cb.append([int(v) for v in O.balanced_bounds(layers, h, w, c, g0, g1, 1, cols[g])])
    return rb, cb


def get_config(layers, h, w, c, limit_bytes, elem_bytes=4, bias_bytes=31 << 20,
               cuts=(16, 12, 8), tiles=(1, 2, 3, 4, 5), lg2=2, balanced_tiles=False):
    """Algorithm 2: cuts in order, first-group grids t x t in order, the
    second group on an lg2 x lg2 grid; the first configuration whose
    prediction (bytes) plus the bias is below the limit, else the last one
    tried.  balanced_tiles: every candidate with its balanced boundaries.
    Returns (cut, t, lg2 or 0, prediction + bias, fits)."""
    n = len(layers)
    last = None
    for cut in cuts:
        for t in tiles:
            if 0 < cut < n:
                gs, rr = [0, cut], [t, lg2]
            else:
                gs, rr = [0], [t]
            rb, cb = balanced(layers, h, w, c, gs, rr, rr) if balanced_tiles else (None, None)
            pred = predict_mem(layers, h, w, c, gs, rr, rr, rb, cb) * elem_bytes + bias_bytes
            last = (cut if 0 < cut < n else n, t, lg2 if 0 < cut < n else 0, pred)
            if pred < limit_bytes:
                return last + (True,)
    return last + (False,)
