"""ctypes wrapper of the CPU oracle (``mafat_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by
the benchmark's CPU-baseline leg.  The product path never imports it.

Layers are the dicts of ``paper_2107_06960_amd.workloads`` (op, c_out, f, s,
p, act).  Arrays are float64 NHWC numpy arrays; the wrapper converts float32
inputs exactly.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mafat_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


class _Layer(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int) for k in ("op", "c_out", "f", "s", "p", "act")]


_OPS = {"conv": 0, "max": 1}
_ACTS = {"linear": 0, "leaky": 1}
ERRORS = {0: "ok", -1: "invalid argument", -2: "tile read outside its region",
          -3: "out of memory", -4: "receptive field is not a rectangle"}


class OracleError(RuntimeError):
    def __init__(self, rc):
        super().__init__(f"oracle error {rc}: {ERRORS.get(rc, '?')}")
        self.rc = rc


def build(force: bool = False) -> str:
    """Compiles the oracle with plain -O2 and no floating-point contraction."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(
            os.path.getmtime(_SRC), os.path.getmtime(os.path.join(_HERE, "mafat_oracle.h"))):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-std=c99", "-O2", "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        ip, dp = ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)
        dpp = ctypes.POINTER(dp)
        lp = ctypes.POINTER(_Layer)
        i = ctypes.c_int
        L.orc_shapes.argtypes = [lp, i, i, i, i, ip]
        L.orc_forward_layers.argtypes = [lp, i, i, i, i, i, i, i, dp, dpp, dpp, dpp, i, dp]
        L.orc_regions_size.argtypes = [i, ip, i, ip, ip]
        L.orc_regions.argtypes = [lp, i, i, i, i, ip, i, ip, ip, ip]
        L.orc_regions_bruteforce.argtypes = [lp, i, i, i, i, ip, i, ip, ip, ip]
        L.orc_forward_tiled.argtypes = [lp, i, i, i, i, i, ip, i, ip, ip, dp, dpp, dpp, dpp, i, dp, dpp]
        L.orc_forward_rect.argtypes = [lp, i, i, i, i, dp, dpp, dpp, dpp, i, i, i, i, i, dp]
        L.orc_regions_bounds.argtypes = [lp, i, i, i, i, ip, i, ip, ip, ip, ip, ip]
        L.orc_regions_bruteforce_bounds.argtypes = [lp, i, i, i, i, ip, i, ip, ip, ip, ip, ip]
        L.orc_forward_tiled_bounds.argtypes = [lp, i, i, i, i, i, ip, i, ip, ip, ip, ip, dp, dpp, dpp,
                                               dpp, i, dp, dpp]
        L.orc_balanced_bounds.argtypes = [lp, i, i, i, i, i, i, i, i, ip]
        L.orc_forward_row_reuse.argtypes = [lp, i, i, i, i, i, ip, i, ip, ip, dp, dpp, dpp, dpp, i, dp, dpp,
                                            ip]
        L.orc_set_threads.argtypes = [i]
        L.orc_round_bf16.argtypes = [ctypes.c_double]
        L.orc_round_bf16.restype = ctypes.c_double
        _lib = L
    return _lib


def _layers(layers):
    arr = (_Layer * len(layers))()
    for k, L in enumerate(layers):
        arr[k] = _Layer(_OPS[L["op"]], int(L.get("c_out", 0)), int(L["f"]), int(L["s"]),
                        int(L["p"]), _ACTS[L.get("act", "linear")])
    return arr


def _ints(v):
    v = np.ascontiguousarray(np.asarray(v, dtype=np.int32))
    return v, v.ctypes.data_as(ctypes.POINTER(ctypes.c_int))


def _dbl(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ptr_list(arrs):
    """float64 copies of per-layer arrays and a double** over them (None -> NULL)."""
    keep = [None if a is None else _dbl(a)[0] for a in arrs]
    pp = (ctypes.POINTER(ctypes.c_double) * len(arrs))()
    for k, a in enumerate(keep):
        pp[k] = a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if a is not None else None
    return keep, pp


def _check(rc):
    if rc != 0:
        raise OracleError(rc)


def shapes(layers, h, w, c):
    """int array (n, 6): in_h, in_w, in_c, out_h, out_w, out_c per layer."""
    out = np.zeros((len(layers), 6), dtype=np.int32)
    _check(lib().orc_shapes(_layers(layers), len(layers), h, w, c,
                            out.ctypes.data_as(ctypes.POINTER(ctypes.c_int))))
    return out


def forward_layers(layers, h, w, c, x, params, l0=0, l1=None, round_bf16=False):
    """Untiled forward of layers [l0, l1]; x is the input of layer l0 (B,H,W,C)."""
    n = len(layers)
    l1 = n - 1 if l1 is None else l1
    dims = shapes(layers, h, w, c)
    x, xp = _dbl(x)
    batch = x.shape[0]
    y = np.zeros((batch, dims[l1, 3], dims[l1, 4], dims[l1, 5]), dtype=np.float64)
    kw, wp = _ptr_list(params["w"])
    ks, sp = _ptr_list(params["scale"])
    kb, bp = _ptr_list(params["bias"])
    _check(lib().orc_forward_layers(_layers(layers), n, h, w, c, l0, l1, batch, xp, wp, sp, bp,
                                    int(round_bf16), y.ctypes.data_as(ctypes.POINTER(ctypes.c_double))))
    return y


def _bounds(bounds):
    """Per-group boundary lists (None: even splits for every group) as one
    concatenated int array and its pointer (NULL for None)."""
    if bounds is None:
        return None, None
    flat = np.ascontiguousarray(np.concatenate([np.asarray(b, dtype=np.int32) for b in bounds]))
    return flat, flat.ctypes.data_as(ctypes.POINTER(ctypes.c_int))


def _region_call(fn, layers, h, w, c, group_start, rows, cols, with_bounds=False, row_bounds=None,
                 col_bounds=None):
    n = len(layers)
    gs, gsp = _ints(group_start)
    r, rp = _ints(rows)
    cc, cp = _ints(cols)
    size = lib().orc_regions_size(n, gsp, len(gs), rp, cp)
    if size < 0:
        raise OracleError(size)
    out = np.zeros(size, dtype=np.int32)
    outp = out.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
    if with_bounds:
        rb, rbp = _bounds(row_bounds)
        cb, cbp = _bounds(col_bounds)
        _check(fn(_layers(layers), n, h, w, c, gsp, len(gs), rp, cp, rbp, cbp, outp))
    else:
        _check(fn(_layers(layers), n, h, w, c, gsp, len(gs), rp, cp, outp))
    res, off = [], 0
    for g in range(len(gs)):
        end = gs[g + 1] if g + 1 < len(gs) else n
        nl, nt = end - gs[g], r[g] * cc[g]
        res.append(out[off:off + nt * nl * 8].reshape(nt, nl, 8))
        off += nt * nl * 8
    return res


def regions(layers, h, w, c, group_start, rows, cols, row_bounds=None, col_bounds=None):
    """List over groups of int arrays (tiles, layers_in_group, 8):
    in y0,y1,x0,x1 then out y0,y1,x0,x1 (half-open).  row_bounds /
    col_bounds: per-group boundary lists (rows+1 / cols+1 values each), or
    None for even splits."""
    if row_bounds is None and col_bounds is None:
        return _region_call(lib().orc_regions, layers, h, w, c, group_start, rows, cols)
    return _region_call(lib().orc_regions_bounds, layers, h, w, c, group_start, rows, cols, True,
                        row_bounds, col_bounds)


def regions_bruteforce(layers, h, w, c, group_start, rows, cols, row_bounds=None, col_bounds=None):
    if row_bounds is None and col_bounds is None:
        return _region_call(lib().orc_regions_bruteforce, layers, h, w, c, group_start, rows, cols)
    return _region_call(lib().orc_regions_bruteforce_bounds, layers, h, w, c, group_start, rows, cols,
                        True, row_bounds, col_bounds)


def balanced_bounds(layers, h, w, c, g0, g1, axis, parts):
    """Balanced tile boundaries along one axis (0 rows, 1 columns) of group
    [g0, g1], by brute force (see orc_balanced_bounds)."""
    out = np.zeros(parts + 1, dtype=np.int32)
    _check(lib().orc_balanced_bounds(_layers(layers), len(layers), h, w, c, g0, g1, axis, parts,
                                     out.ctypes.data_as(ctypes.POINTER(ctypes.c_int))))
    return out


def forward_tiled(layers, h, w, c, x, params, group_start, rows, cols, round_bf16=False,
                  want_cuts=False, row_bounds=None, col_bounds=None):
    n = len(layers)
    dims = shapes(layers, h, w, c)
    x, xp = _dbl(x)
    batch = x.shape[0]
    y = np.zeros((batch, dims[-1, 3], dims[-1, 4], dims[-1, 5]), dtype=np.float64)
    gs, gsp = _ints(group_start)
    r, rp = _ints(rows)
    cc, cp = _ints(cols)
    cuts = []
    cut_pp = None
    if want_cuts and len(gs) > 1:
        cut_pp = (ctypes.POINTER(ctypes.c_double) * (len(gs) - 1))()
        for g in range(len(gs) - 1):
            last = gs[g + 1] - 1
            a = np.zeros((batch, dims[last, 3], dims[last, 4], dims[last, 5]), dtype=np.float64)
            cuts.append(a)
            cut_pp[g] = a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    kw, wp = _ptr_list(params["w"])
    ks, sp = _ptr_list(params["scale"])
    kb, bp = _ptr_list(params["bias"])
    rb, rbp = _bounds(row_bounds)
    cb, cbp = _bounds(col_bounds)
    _check(lib().orc_forward_tiled_bounds(_layers(layers), n, h, w, c, batch, gsp, len(gs), rp, cp,
                                          rbp, cbp, xp, wp, sp, bp, int(round_bf16),
                                          y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), cut_pp))
    return (y, cuts) if want_cuts else y


def forward_row_reuse(layers, h, w, c, x, params, group_start, rows, round_bf16=False, want_cuts=False,
                      row_bounds=None):
    """Row reuse (orc_forward_row_reuse): every group's tile rows in order,
    each layer output computed once into row bands.  Returns y (and the cut
    tensors with want_cuts)."""
    n = len(layers)
    dims = shapes(layers, h, w, c)
    x, xp = _dbl(x)
    batch = x.shape[0]
    y = np.zeros((batch, dims[-1, 3], dims[-1, 4], dims[-1, 5]), dtype=np.float64)
    gs, gsp = _ints(group_start)
    r, rp = _ints(rows)
    cuts = []
    cut_pp = None
    if want_cuts and len(gs) > 1:
        cut_pp = (ctypes.POINTER(ctypes.c_double) * (len(gs) - 1))()
        for g in range(len(gs) - 1):
            last = gs[g + 1] - 1
            a = np.zeros((batch, dims[last, 3], dims[last, 4], dims[last, 5]), dtype=np.float64)
            cuts.append(a)
            cut_pp[g] = a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    kw, wp = _ptr_list(params["w"])
    ks, sp = _ptr_list(params["scale"])
    kb, bp = _ptr_list(params["bias"])
    rb, rbp = _bounds(row_bounds)
    _check(lib().orc_forward_row_reuse(_layers(layers), n, h, w, c, batch, gsp, len(gs), rp, rbp, xp, wp, sp,
                                       bp, int(round_bf16), y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                       cut_pp, None))
    return (y, cuts) if want_cuts else y


def row_reuse_band_rows(layers, h, w, c, group_start, rows, row_bounds=None):
    """Per layer, the most rows any of its row-reuse bands holds (0 for a
    group's last layer): the geometry of orc_forward_row_reuse alone."""
    n = len(layers)
    gs, gsp = _ints(group_start)
    r, rp = _ints(rows)
    rb, rbp = _bounds(row_bounds)
    out = np.zeros(n, dtype=np.int32)
    _check(lib().orc_forward_row_reuse(_layers(layers), n, h, w, c, 1, gsp, len(gs), rp, rbp, None, None, None,
                                       None, 0, None, None, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int))))
    return out


def forward_rect(layers, h, w, c, x1, params, oy0, oy1, ox0, ox1, round_bf16=False):
    """Output of the whole stack on one output rectangle of one frame x1 (H,W,C)."""
    n = len(layers)
    dims = shapes(layers, h, w, c)
    x1, xp = _dbl(x1)
    y = np.zeros((oy1 - oy0, ox1 - ox0, dims[-1, 5]), dtype=np.float64)
    kw, wp = _ptr_list(params["w"])
    ks, sp = _ptr_list(params["scale"])
    kb, bp = _ptr_list(params["bias"])
    _check(lib().orc_forward_rect(_layers(layers), n, h, w, c, xp, wp, sp, bp, int(round_bf16),
                                  oy0, oy1, ox0, ox1, y.ctypes.data_as(ctypes.POINTER(ctypes.c_double))))
    return y


def set_threads(n: int) -> None:
    """Threads of the layer loops (output-row bands; results unchanged)."""
    _check(lib().orc_set_threads(int(n)))


def round_bf16(v: float) -> float:
    return lib().orc_round_bf16(float(v))
