"""Thin ctypes binding of libmafat.so (the C ABI declared in include/mafat.h).

Functions keep the C names (``mafat_plan_create``, ``mafat_run_group``,
``mafat_run_network``, ...) and only marshal arguments: every step of the
computation runs in the library's HIP kernels.  PyTorch is used only to own
device memory and to supply the stream.  There is no fallback: if the
library is missing, loading raises.

``Plan`` wraps a plan handle; ``Network`` holds device copies of the
parameters and runs the whole stack.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import workloads as W

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmafat.so")

MAFAT_OK, MAFAT_EINVAL, MAFAT_ESHAPE, MAFAT_EUNSUPPORTED = 0, -1, -2, -3
MAFAT_EWORKSPACE, MAFAT_EHIP, MAFAT_ENOMEM = -4, -5, -6
MAFAT_CONV, MAFAT_MAXPOOL = 0, 1
MAFAT_ACT_LINEAR, MAFAT_ACT_LEAKY01 = 0, 1
MAFAT_F32, MAFAT_BF16 = 0, 1
MAFAT_MEM_DEVICE, MAFAT_MEM_PAPER, MAFAT_MEM_DEVICE_SEQ = 0, 1, 2
MAFAT_PLAN_STAGE_PARTITION, MAFAT_PLAN_PACKED_WEIGHTS, MAFAT_PLAN_ROW_REUSE = 1, 2, 4
MAFAT_STATIC_WORKSPACE_MIB = 32   # include/mafat.h: size of the static workspace of mafat_run_network_static
MEM_MODELS = {"device": MAFAT_MEM_DEVICE, "paper": MAFAT_MEM_PAPER, "device_seq": MAFAT_MEM_DEVICE_SEQ}
DTYPES = {"f32": MAFAT_F32, "bf16": MAFAT_BF16}

# Every symbol include/mafat.h declares.
EXPORTS = ("mafat_plan_create", "mafat_plan_create_flags", "mafat_plan_create_bounds",
           "mafat_balanced_bounds", "mafat_plan_destroy",
           "mafat_packed_weights_size", "mafat_pack_weights", "mafat_plan_layer_shape", "mafat_plan_group",
           "mafat_plan_num_tiles", "mafat_plan_regions", "mafat_plan_macs", "mafat_plan_stages", "mafat_plan_stage_layers",
           "mafat_plan_stage_fused", "mafat_plan_stage_kernel", "mafat_plan_set_tile_batch",
           "mafat_workspace_size", "mafat_run_group", "mafat_run_group_timed", "mafat_run_stage", "mafat_run_network",
           "mafat_run_network_static",
           "mafat_predict_mem", "mafat_get_config", "mafat_get_config_balanced", "mafat_get_config_flags", "mafat_status_string",
           "mafat_last_error")


class mafat_layer(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in ("op", "c_out", "f", "s", "p", "act")]


class mafat_rect(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in ("y0", "y1", "x0", "x1")]


class MafatError(RuntimeError):
    def __init__(self, fn, rc, detail):
        super().__init__(f"{fn} failed: {rc} ({_status(rc)}): {detail}")
        self.rc = rc


_lib = None


def lib():
    """Loads libmafat.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2107_06960_amd.build`")
        # torch ships its own HIP runtime under the same soname; importing it
        # first makes libmafat bind to that one instead of loading a second
        # runtime from /opt/rocm.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        vp, vpp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)
        i32p = ctypes.POINTER(i32)
        planp = ctypes.c_void_p
        L.mafat_plan_create.argtypes = [ctypes.POINTER(mafat_layer), i32, i32, i32, i32, i32p, i32,
                                        i32p, i32p, ctypes.POINTER(planp)]
        L.mafat_plan_create_flags.argtypes = [ctypes.POINTER(mafat_layer), i32, i32, i32, i32, i32p, i32,
                                              i32p, i32p, i32, ctypes.POINTER(planp)]
        L.mafat_plan_create_bounds.argtypes = [ctypes.POINTER(mafat_layer), i32, i32, i32, i32, i32p, i32,
                                               i32p, i32p, i32p, i32p, i32, ctypes.POINTER(planp)]
        L.mafat_balanced_bounds.argtypes = [ctypes.POINTER(mafat_layer), i32, i32, i32, i32, i32, i32, i32, i32,
                                            i32p, i32p]
        L.mafat_plan_destroy.argtypes = [planp]
        L.mafat_packed_weights_size.argtypes = [planp, i32, i32, ctypes.POINTER(sz)]
        L.mafat_pack_weights.argtypes = [planp, i32, i32, vp, vp, vp]
        L.mafat_plan_destroy.restype = None
        L.mafat_plan_layer_shape.argtypes = [planp, i32, i32p]
        L.mafat_plan_group.argtypes = [planp, i32, i32p, i32p, i32p]
        L.mafat_plan_num_tiles.argtypes = [planp, i32, i32p]
        L.mafat_plan_regions.argtypes = [planp, i32, ctypes.POINTER(mafat_rect),
                                         ctypes.POINTER(mafat_rect), i64]
        L.mafat_plan_macs.argtypes = [planp, i32, ctypes.POINTER(i64), ctypes.POINTER(i64)]
        L.mafat_plan_stages.argtypes = [planp, i32, i32p]
        L.mafat_plan_stage_layers.argtypes = [planp, i32, i32, i32p, i32p]
        L.mafat_plan_stage_fused.argtypes = [planp, i32, i32, i32, i32, i32p]
        L.mafat_plan_stage_kernel.argtypes = [planp, i32, i32, i32, i32, i32p]
        L.mafat_plan_set_tile_batch.argtypes = [planp, i32]
        L.mafat_workspace_size.argtypes = [planp, i32, i32, ctypes.POINTER(sz)]
        L.mafat_run_group.argtypes = [planp, i32, i32, i32, vp, vp, vpp, vpp, vpp, vp, sz, vp]
        L.mafat_run_group_timed.argtypes = [planp, i32, i32, i32, vp, vp, vpp, vpp, vpp, vp, sz, vp, vpp]
        L.mafat_run_stage.argtypes = [planp, i32, i32, i32, i32, vp, vp, vpp, vpp, vpp, vp, sz, vp]
        L.mafat_run_network.argtypes = [planp, i32, i32, vp, vp, vpp, vpp, vpp, vpp, vp, sz, vp]
        L.mafat_run_network_static.argtypes = [planp, i32, i32, vp, vp, vpp, vpp, vpp, vpp, vp]
        i64p = ctypes.POINTER(i64)
        L.mafat_predict_mem.argtypes = [planp, i32, i32, i32, i64p]
        L.mafat_get_config.argtypes = [ctypes.POINTER(mafat_layer), i32, i32, i32, i32, i32, i32, i32, i64, i64,
                                       i32p, i32, i32p, i32, i32, i32p, i32p, i32p, i64p, i32p]
        L.mafat_get_config_balanced.argtypes = L.mafat_get_config.argtypes
        a = list(L.mafat_get_config.argtypes)
        L.mafat_get_config_flags.argtypes = a[:15] + [i32, i32] + a[15:]
        L.mafat_status_string.argtypes = [ctypes.c_int]
        L.mafat_status_string.restype = ctypes.c_char_p
        L.mafat_last_error.argtypes = []
        L.mafat_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _status(rc):
    return lib().mafat_status_string(rc).decode()


def _check(fn, rc):
    if rc != MAFAT_OK:
        raise MafatError(fn, rc, lib().mafat_last_error().decode())


def _ptrs(vals):
    arr = (ctypes.c_void_p * max(1, len(vals)))()
    for k, v in enumerate(vals):
        arr[k] = v
    return arr


# ------------------------------------------------------------------ C names

def _layer_array(layers):
    arr = (mafat_layer * len(layers))()
    for k, L in enumerate(layers):
        op = MAFAT_CONV if L["op"] == W.CONV else MAFAT_MAXPOOL
        act = MAFAT_ACT_LEAKY01 if L.get("act") == W.LEAKY else MAFAT_ACT_LINEAR
        arr[k] = mafat_layer(op, int(L.get("c_out", 0)), int(L["f"]), int(L["s"]), int(L["p"]), act)
    return arr


def _flat_bounds(bounds):
    """Per-group boundary lists -> one concatenated int32 array (None -> NULL)."""
    if bounds is None:
        return None
    flat = [int(v) for b in bounds for v in b]
    return (ctypes.c_int32 * len(flat))(*flat)


def mafat_plan_create(layers, in_h, in_w, in_c, group_start, grid_rows, grid_cols, flags=0,
                      row_bounds=None, col_bounds=None):
    """Returns a plan handle (int); raises MafatError with the library's status.
    flags: 0, or MAFAT_PLAN_STAGE_PARTITION or MAFAT_PLAN_ROW_REUSE, and/or
    MAFAT_PLAN_PACKED_WEIGHTS (mafat_plan_create_flags).  row_bounds / col_bounds: per-group lists of
    rows+1 / cols+1 tile boundaries (mafat_plan_create_bounds), or None."""
    n = len(layers)
    arr = _layer_array(layers)
    gs = (ctypes.c_int32 * len(group_start))(*group_start)
    rr = (ctypes.c_int32 * len(grid_rows))(*grid_rows)
    cc = (ctypes.c_int32 * len(grid_cols))(*grid_cols)
    h = ctypes.c_void_p()
    if row_bounds is not None or col_bounds is not None:
        _check("mafat_plan_create_bounds",
               lib().mafat_plan_create_bounds(arr, n, in_h, in_w, in_c, gs, len(group_start), rr, cc,
                                              _flat_bounds(row_bounds), _flat_bounds(col_bounds), flags,
                                              ctypes.byref(h)))
    elif flags:
        _check("mafat_plan_create_flags",
               lib().mafat_plan_create_flags(arr, n, in_h, in_w, in_c, gs, len(group_start), rr, cc, flags,
                                             ctypes.byref(h)))
    else:
        _check("mafat_plan_create",
               lib().mafat_plan_create(arr, n, in_h, in_w, in_c, gs, len(group_start), rr, cc, ctypes.byref(h)))
    return h.value


def mafat_balanced_bounds(layers, in_h, in_w, in_c, first_layer, last_layer, rows, cols):
    """(row_bounds, col_bounds): balanced tile boundaries of the group
    [first_layer, last_layer] (lists of rows+1 and cols+1 ints)."""
    rb = (ctypes.c_int32 * (rows + 1))()
    cb = (ctypes.c_int32 * (cols + 1))()
    _check("mafat_balanced_bounds",
           lib().mafat_balanced_bounds(_layer_array(layers), len(layers), in_h, in_w, in_c, first_layer,
                                       last_layer, rows, cols, rb, cb))
    return list(rb), list(cb)


def mafat_plan_destroy(plan):
    lib().mafat_plan_destroy(plan)


def mafat_packed_weights_size(plan, layer, dtype):
    v = ctypes.c_size_t()
    _check("mafat_packed_weights_size",
           lib().mafat_packed_weights_size(plan, layer, DTYPES.get(dtype, dtype), ctypes.byref(v)))
    return v.value


def mafat_pack_weights(plan, layer, dtype, w_krsc_ptr, w_packed_ptr, stream=None):
    _check("mafat_pack_weights",
           lib().mafat_pack_weights(plan, layer, DTYPES.get(dtype, dtype), w_krsc_ptr, w_packed_ptr,
                                    _stream_handle(stream)))


def mafat_plan_layer_shape(plan, layer):
    d = (ctypes.c_int32 * 6)()
    _check("mafat_plan_layer_shape", lib().mafat_plan_layer_shape(plan, layer, d))
    return tuple(d)


def mafat_plan_group(plan, group):
    a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    _check("mafat_plan_group", lib().mafat_plan_group(plan, group, ctypes.byref(a), ctypes.byref(b),
                                                      ctypes.byref(c)))
    return a.value, b.value, c.value


def mafat_plan_num_tiles(plan, group):
    n = ctypes.c_int32()
    _check("mafat_plan_num_tiles", lib().mafat_plan_num_tiles(plan, group, ctypes.byref(n)))
    return n.value


def mafat_plan_regions(plan, group):
    """int32 array (tiles, layers_in_group, 8): in y0,y1,x0,x1 then out y0,y1,x0,x1."""
    _, nl, nt = mafat_plan_group(plan, group)
    ins, outs = (mafat_rect * (nl * nt))(), (mafat_rect * (nl * nt))()
    _check("mafat_plan_regions", lib().mafat_plan_regions(plan, group, ins, outs, nl * nt))
    a = np.ctypeslib.as_array(ctypes.cast(ins, ctypes.POINTER(ctypes.c_int32)), (nl * nt * 4,))
    b = np.ctypeslib.as_array(ctypes.cast(outs, ctypes.POINTER(ctypes.c_int32)), (nl * nt * 4,))
    return np.concatenate([a.reshape(nt, nl, 4), b.reshape(nt, nl, 4)], axis=2).copy()


def mafat_plan_macs(plan, group):
    e, u = ctypes.c_int64(), ctypes.c_int64()
    _check("mafat_plan_macs", lib().mafat_plan_macs(plan, group, ctypes.byref(e), ctypes.byref(u)))
    return e.value, u.value


def mafat_plan_stages(plan, group):
    n = ctypes.c_int32()
    _check("mafat_plan_stages", lib().mafat_plan_stages(plan, group, ctypes.byref(n)))
    out = []
    for s in range(n.value):
        a, b = ctypes.c_int32(), ctypes.c_int32()
        _check("mafat_plan_stage_layers", lib().mafat_plan_stage_layers(plan, group, s, ctypes.byref(a),
                                                                        ctypes.byref(b)))
        out.append((a.value, b.value))
    return out


def mafat_plan_set_tile_batch(plan, tiles):
    _check("mafat_plan_set_tile_batch", lib().mafat_plan_set_tile_batch(plan, tiles))


def mafat_plan_stage_fused(plan, group, stage, batch, dtype):
    f = ctypes.c_int32()
    _check("mafat_plan_stage_fused", lib().mafat_plan_stage_fused(plan, group, stage, batch, DTYPES.get(dtype, dtype),
                                                                  ctypes.byref(f)))
    return bool(f.value)


# mafat_kernel values, by name
KERNELS = ("patch", "patch_first", "patch_1x1", "ring", "mfma_f32", "first_layer", "generic", "pool")


def mafat_plan_stage_kernel(plan, group, stage, batch, dtype):
    """The kernel family (a KERNELS name) that runs a stage in mafat_run_group."""
    out = ctypes.c_int32()
    _check("mafat_plan_stage_kernel", lib().mafat_plan_stage_kernel(plan, group, stage, batch, DTYPES.get(dtype, dtype),
                                                                    ctypes.byref(out)))
    return KERNELS[out.value]


def mafat_workspace_size(plan, batch, dtype):
    n = ctypes.c_size_t()
    _check("mafat_workspace_size", lib().mafat_workspace_size(plan, batch, dtype, ctypes.byref(n)))
    return n.value


def mafat_run_group(plan, group, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes, stream):
    """x, y, workspace: device pointers (int); w/scale/bias: lists of device
    pointers indexed by layer (None for pools); stream: hipStream_t (int)."""
    _check("mafat_run_group",
           lib().mafat_run_group(plan, group, batch, dtype, x, y, _ptrs(w), _ptrs(scale), _ptrs(bias),
                                 workspace, ws_bytes, stream))


def mafat_run_group_timed(plan, group, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes, stream,
                          events):
    """mafat_run_group plus events: a list of 2 * n_stages hipEvent_t
    handles (start and end of each stage's kernels; entries may be None)."""
    _check("mafat_run_group_timed",
           lib().mafat_run_group_timed(plan, group, batch, dtype, x, y, _ptrs(w), _ptrs(scale), _ptrs(bias),
                                       workspace, ws_bytes, stream, _ptrs(events)))


def mafat_run_stage(plan, group, stage, batch, dtype, x, y, w, scale, bias, workspace, ws_bytes, stream):
    """One stage of a group (same pointer conventions as mafat_run_group)."""
    _check("mafat_run_stage",
           lib().mafat_run_stage(plan, group, stage, batch, dtype, x, y, _ptrs(w), _ptrs(scale), _ptrs(bias),
                                 workspace, ws_bytes, stream))


def mafat_run_network(plan, batch, dtype, x, y, cut_bufs, w, scale, bias, workspace, ws_bytes, stream):
    _check("mafat_run_network",
           lib().mafat_run_network(plan, batch, dtype, x, y, _ptrs(cut_bufs), _ptrs(w), _ptrs(scale),
                                   _ptrs(bias), workspace, ws_bytes, stream))


def mafat_run_network_static(plan, batch, dtype, x, y, cut_bufs, w, scale, bias, stream):
    """mafat_run_network with the library's static workspace (no workspace
    argument; allocates nothing)."""
    _check("mafat_run_network_static",
           lib().mafat_run_network_static(plan, batch, dtype, x, y, _ptrs(cut_bufs), _ptrs(w), _ptrs(scale),
                                          _ptrs(bias), stream))


def mafat_predict_mem(plan, model, batch, dtype):
    """Predicted bytes (int) of a plan handle under model 'device' or 'paper'."""
    out = ctypes.c_int64()
    _check("mafat_predict_mem", lib().mafat_predict_mem(plan, MEM_MODELS.get(model, model), batch,
                                                        DTYPES.get(dtype, dtype), ctypes.byref(out)))
    return out.value


def mafat_get_config(layers, in_hwc, limit_bytes, model="paper", batch=1, dtype="f32", bias_bytes=0,
                     cuts=(16, 12, 8), grids=(1, 2, 3, 4, 5), second_grid=2, balanced=False, flags=0):
    """Algorithm 2 (balanced=True: mafat_get_config_balanced, every
    candidate with balanced tile boundaries; flags: plan flags of every
    candidate, mafat_get_config_flags).  Returns (tiling spec in the paper's
    notation, prediction + bias, fits)."""
    h, w, c = in_hwc
    cc = (ctypes.c_int32 * len(cuts))(*cuts)
    gg = (ctypes.c_int32 * len(grids))(*grids)
    oc, o1, o2, fits = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    pred = ctypes.c_int64()
    head = (_layer_array(layers), len(layers), h, w, c, MEM_MODELS.get(model, model), batch, DTYPES.get(dtype, dtype),
            int(bias_bytes), int(limit_bytes), cc, len(cuts), gg, len(grids), second_grid)
    tail = (ctypes.byref(oc), ctypes.byref(o1), ctypes.byref(o2), ctypes.byref(pred), ctypes.byref(fits))
    if flags:
        _check("mafat_get_config_flags", lib().mafat_get_config_flags(*head, int(flags), int(bool(balanced)), *tail))
    else:
        name = "mafat_get_config_balanced" if balanced else "mafat_get_config"
        _check(name, getattr(lib(), name)(*head, *tail))
    if oc.value >= len(layers):
        spec = f"{o1.value}x{o1.value}/NoCut"
    else:
        spec = f"{o1.value}x{o1.value}/{oc.value}/{o2.value}x{o2.value}"
    return spec, pred.value, bool(fits.value)


# ------------------------------------------------------------------ convenience

class Plan:
    """A plan for a layer stack, an input shape and a tiling spec such as
    ``"5x5/8/2x2"`` (section 5.1 notation) or explicit group lists."""

    def __init__(self, layers, in_hwc, tiling="1x1/NoCut", stage_partition=False, packed_weights=False,
                 tile_batch=0, bounds=None, row_reuse=False):
        """bounds: None (even tile boundaries), "balanced" (each group's
        mafat_balanced_bounds) or a pair (row_bounds, col_bounds) of
        per-group boundary lists (mafat_plan_create_bounds).  row_reuse:
        MAFAT_PLAN_ROW_REUSE (tile rows in order, each stage output computed
        once into row bands)."""
        self.layers = list(layers)
        self.stage_partition = bool(stage_partition)
        self.row_reuse = bool(row_reuse)
        self.packed_weights = bool(packed_weights)
        self.tile_batch = int(tile_batch)
        self.h, self.w, self.c = in_hwc
        self.group_start, self.rows, self.cols = W.parse_tiling(tiling, len(layers)) \
            if isinstance(tiling, str) else tiling
        if isinstance(bounds, str):
            if bounds != "balanced":
                raise ValueError(f"bounds: None, 'balanced' or (row_bounds, col_bounds), not {bounds!r}")
            per = [mafat_balanced_bounds(self.layers, self.h, self.w, self.c, g0,
                                         (self.group_start[g + 1] if g + 1 < len(self.group_start)
                                          else len(self.layers)) - 1, self.rows[g], self.cols[g])
                   for g, g0 in enumerate(self.group_start)]
            bounds = ([p[0] for p in per], [p[1] for p in per])
        self.bounds = bounds
        rb, cb = bounds if bounds is not None else (None, None)
        self.handle = mafat_plan_create(self.layers, self.h, self.w, self.c, self.group_start,
                                        self.rows, self.cols,
                                        (MAFAT_PLAN_STAGE_PARTITION if self.stage_partition else 0) |
                                        (MAFAT_PLAN_PACKED_WEIGHTS if self.packed_weights else 0) |
                                        (MAFAT_PLAN_ROW_REUSE if self.row_reuse else 0),
                                        row_bounds=rb, col_bounds=cb)
        self.n_groups = len(self.group_start)
        if self.tile_batch:
            mafat_plan_set_tile_batch(self.handle, self.tile_batch)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                mafat_plan_destroy(h)
            except Exception:
                pass
            self.handle = None

    def shape(self, layer):
        return mafat_plan_layer_shape(self.handle, layer)

    def group(self, g):
        return mafat_plan_group(self.handle, g)

    def num_tiles(self, g):
        return mafat_plan_num_tiles(self.handle, g)

    def regions(self, g):
        return mafat_plan_regions(self.handle, g)

    def macs(self, g):
        return mafat_plan_macs(self.handle, g)

    def stages(self, g):
        return mafat_plan_stages(self.handle, g)

    def stage_fused(self, g, s, batch=1, dtype="bf16"):
        return mafat_plan_stage_fused(self.handle, g, s, batch, dtype)

    def stage_kernel(self, g, s, batch=1, dtype="bf16"):
        return mafat_plan_stage_kernel(self.handle, g, s, batch, dtype)

    def launches(self, g, batch=1, dtype="bf16"):
        """The kernel launches of mafat_run_group for group g: lists of stage
        indices (a fused pair is one launch)."""
        st, out, s = self.stages(g), [], 0
        while s < len(st):
            n = 2 if self.stage_fused(g, s, batch, dtype) else 1
            out.append(list(range(s, s + n)))
            s += n
        return out

    def predict_mem(self, model="device", batch=1, dtype="bf16"):
        return mafat_predict_mem(self.handle, model, batch, dtype)

    def workspace_size(self, batch, dtype):
        return mafat_workspace_size(self.handle, batch, DTYPES.get(dtype, dtype))

    def group_out_shape(self, g):
        first, nl, _ = self.group(g)
        d = self.shape(first + nl - 1)
        return d[3], d[4], d[5]


def _stream_handle(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Network:
    """Device-resident parameters for a plan, plus output / cut / workspace
    buffers, all allocated by torch.  run() enqueues mafat_run_network."""

    def __init__(self, plan: Plan, params, batch: int, dtype: str, device="cuda"):
        import torch
        self.plan, self.batch, self.dtype = plan, batch, dtype
        self.code = DTYPES[dtype]
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        self.tdtype = tdt
        self.w, self.scale, self.bias = [], [], []
        for k, L in enumerate(plan.layers):
            if L["op"] != W.CONV:
                self.w.append(None); self.scale.append(None); self.bias.append(None)
                continue
            w = torch.from_numpy(np.ascontiguousarray(params["w"][k])).to(device=device, dtype=tdt)
            nbytes = mafat_packed_weights_size(plan.handle, k, dtype)
            if nbytes:  # the plan takes this layer's weights packed (mafat_pack_weights)
                wp = torch.empty(nbytes // w.element_size(), dtype=tdt, device=device)
                mafat_pack_weights(plan.handle, k, dtype, w.data_ptr(), wp.data_ptr())
                torch.cuda.synchronize()
                del w
                w = wp
            self.w.append(w)
            self.scale.append(torch.from_numpy(np.ascontiguousarray(params["scale"][k])).to(device))
            self.bias.append(torch.from_numpy(np.ascontiguousarray(params["bias"][k])).to(device))
        self.cuts = [torch.empty((batch,) + plan.group_out_shape(g), dtype=tdt, device=device)
                     for g in range(plan.n_groups - 1)]
        self.y = torch.empty((batch,) + plan.group_out_shape(plan.n_groups - 1), dtype=tdt, device=device)
        self.ws_bytes = plan.workspace_size(batch, dtype)
        self.ws = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)
        self._wp = [None if t is None else t.data_ptr() for t in self.w]
        self._sp = [None if t is None else t.data_ptr() for t in self.scale]
        self._bp = [None if t is None else t.data_ptr() for t in self.bias]

    def input_tensor(self, x_np, device="cuda"):
        import torch
        return torch.from_numpy(np.ascontiguousarray(x_np)).to(device=device, dtype=self.tdtype)

    def run(self, x, stream=None):
        assert x.dtype == self.tdtype and x.is_contiguous()
        assert tuple(x.shape) == (self.batch, self.plan.h, self.plan.w, self.plan.c)
        mafat_run_network(self.plan.handle, self.batch, self.code, x.data_ptr(), self.y.data_ptr(),
                          [c.data_ptr() for c in self.cuts], self._wp, self._sp, self._bp,
                          self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream))
        return self.y

    def run_group(self, g, x, y, stream=None, events=None):
        args = (self.plan.handle, g, self.batch, self.code, x.data_ptr(), y.data_ptr(),
                self._wp, self._sp, self._bp, self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream))
        if events is None:
            mafat_run_group(*args)
        else:
            mafat_run_group_timed(*args, events)

    def run_stage(self, g, s, x, y, stream=None):
        mafat_run_stage(self.plan.handle, g, s, self.batch, self.code, x.data_ptr(), y.data_ptr(),
                        self._wp, self._sp, self._bp, self.ws.data_ptr(), self.ws_bytes,
                        _stream_handle(stream))

    def group_io(self, g, x):
        gin = x if g == 0 else self.cuts[g - 1]
        gout = self.y if g == self.plan.n_groups - 1 else self.cuts[g]
        return gin, gout


def run_network(plan, x, params, out=None, stream=None):
    """One call: the plan's network on the device tensor x (NHWC, batch
    frames, bfloat16 or float32 -- the run dtype), with the parameters
    `params` (per-layer host arrays w / scale / bias, as
    workloads.make_inputs draws them) uploaded for this call
    (mafat_run_network on caller-owned torch buffers).  Returns the output,
    or writes it into `out` and returns that.  For repeated runs keep a
    Network, which uploads the parameters once."""
    import torch
    if x.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("x must be bfloat16 or float32")
    dtype = "bf16" if x.dtype == torch.bfloat16 else "f32"
    net = Network(plan, params, x.shape[0], dtype, device=x.device)
    y = net.run(x.contiguous(), stream=stream)
    if out is None:
        return y
    out.copy_(y)
    return out
