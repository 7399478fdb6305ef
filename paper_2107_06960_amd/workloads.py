"""Workload descriptions and seeded synthetic inputs.

This module is shared by the GPU library's tests/benchmark and by the CPU
oracle's tests.  It holds only *descriptions* (layer lists, tilings, input
recipes) and random draws; it performs none of the method's arithmetic
(no shape inference, no regions, no convolution).

Networks (arXiv 2107.06960):
  * ``YOLOV2_16`` -- the first 16 layers of YOLOv2, the network the paper
    evaluates (section 2 and section 5).  The paper lists the cut candidates
    directly after the max-pools at layers 2, 4, 8 and 12 (section 4), which
    puts the max-pools at layers 1, 3, 7 and 11; the layer types and widths
    are those of YOLOv2's first 16 layers.
  * ``TINY`` -- a three-layer conv / max-pool / conv stack for quick checks.

Tiling notation (section 5.1): ``N1xM1/c/N2xM2`` is a first group tiled
N1xM1, a cut at layer c, and a second group tiled N2xM2; ``NxM/NoCut`` (or
just ``NxM``) is one fused group.  Cuts are 0-based layer indices: group 1 is
layers [0, c) and group 2 is layers [c, n) (section 4).

Input recipe (stated once here, used everywhere): ``numpy.random.default_rng
(seed)`` drawing, in this order, the input (batch, H, W, C) from U[0, 1); then
for every convolution layer in index order its weights (c_out, f, f, c_in)
from N(0, std = sqrt(2 / (c_in * f * f))), its folded batch-norm scale
(c_out) from U[0.5, 1.5) and its bias (c_out) from N(0, 0.1).  All draws are
float32.  For bf16 workloads every array is rounded to the nearest bfloat16
(ties to even) and both the GPU path and the oracle receive those values.
"""
from __future__ import annotations

import re
from dataclasses import dataclass, field

import numpy as np

CONV, MAXPOOL = "conv", "max"
LINEAR, LEAKY = "linear", "leaky"


def conv(c_out: int, f: int = 3, act: str = LEAKY, s: int = 1, p: int = None) -> dict:
    """A convolution with scale/bias + act; by default stride 1 and 'same'
    padding (f-1)/2."""
    return {"op": CONV, "c_out": c_out, "f": f, "s": s, "p": (f - 1) // 2 if p is None else p, "act": act}


def maxpool(f: int = 2, s: int = 2, p: int = 0) -> dict:
    """A max-pool over the in-image elements of each f x f window."""
    return {"op": MAXPOOL, "c_out": 0, "f": f, "s": s, "p": p, "act": LINEAR}


# YOLOv2 layers 0-15.
YOLOV2_16 = [
    conv(32), maxpool(), conv(64), maxpool(),
    conv(128), conv(64, 1), conv(128), maxpool(),
    conv(256), conv(128, 1), conv(256), maxpool(),
    conv(512), conv(256, 1), conv(512), conv(256, 1),
]

TINY = [conv(16), maxpool(), conv(32)]

# Other layer kinds (the generalisation to other CNNs the paper names as
# future work, section 6): a ResNet-style stem (7x7 stride-2 convolution,
# 3x3 stride-2 padded max-pool) followed by 3x3 convolutions, a strided 3x3
# downsampling convolution, a 3x3 stride-1 max-pool and a 5x5 convolution.
OTHER_CNN = [conv(32, 7, s=2, p=3), maxpool(3, 2, 1), conv(32), conv(64, 3, s=2, p=1),
             maxpool(3, 1, 1), conv(64, 5), conv(32, 1), maxpool(), conv(64)]


def parse_tiling(spec: str, n_layers: int):
    """Parses ``"5x5/8/2x2"``, ``"2x2/NoCut"`` or ``"3x3"`` (more groups:
    ``"a/c1/b/c2/d"``).  Returns (group_start, grid_rows, grid_cols)."""
    parts = [p.strip() for p in spec.split("/") if p.strip()]
    if parts and parts[-1].lower() == "nocut":
        parts = parts[:-1]
    if len(parts) % 2 != 1:
        raise ValueError(f"bad tiling spec {spec!r}")
    starts, rows, cols = [0], [], []
    for k, p in enumerate(parts):
        if k % 2 == 0:
            m = re.fullmatch(r"(\d+)\s*[xX]\s*(\d+)", p)
            if not m:
                raise ValueError(f"bad grid {p!r} in {spec!r}")
            rows.append(int(m.group(1)))
            cols.append(int(m.group(2)))
        else:
            c = int(p)
            if not (starts[-1] < c < n_layers):
                raise ValueError(f"cut {c} out of range in {spec!r}")
            starts.append(c)
    return starts, rows, cols


@dataclass
class Workload:
    name: str
    layers: list
    h: int
    w: int
    c: int
    batch: int
    dtype: str          # "f32" or "bf16"
    tiling: str
    seed: int = 0
    note: str = ""
    extra: dict = field(default_factory=dict)

    def groups(self):
        return parse_tiling(self.tiling, len(self.layers))


WORKLOADS = {
    "tiny": Workload("tiny", TINY, 64, 64, 3, 1, "f32", "2x2/NoCut",
                     note="conv3x3 3->16, maxpool, conv3x3 16->32; one group 2x2"),
    "yolo416_ftp3": Workload("yolo416_ftp3", YOLOV2_16, 416, 416, 3, 1, "f32", "3x3/NoCut",
                             note="YOLOv2 layers 0-15, 416x416, one fused group 3x3"),
    "yolo608_5x5_8_2x2": Workload("yolo608_5x5_8_2x2", YOLOV2_16, 608, 608, 3, 1, "bf16", "5x5/8/2x2",
                                  note="YOLOv2 layers 0-15, 608x608, layers 0-7 on 5x5, 8-15 on 2x2"),
    "yolo608_4x4_12_1x1_b8": Workload("yolo608_4x4_12_1x1_b8", YOLOV2_16, 608, 608, 3, 8, "bf16",
                                      "4x4/12/1x1",
                                      note="YOLOv2 layers 0-15, 608x608, batch 8, layers 0-11 on 4x4, 12-15 1x1"),
}

SWEEP6 = ["3x3/4/2x2", "6x6/4/2x2", "3x3/8/2x2", "6x6/8/2x2", "3x3/12/2x2", "6x6/12/2x2"]
for _t in SWEEP6:
    _n = "yolo608_sweep_" + _t.replace("/", "_")
    WORKLOADS[_n] = Workload(_n, YOLOV2_16, 608, 608, 3, 1, "bf16", _t,
                             note=f"YOLOv2 layers 0-15, 608x608, {_t}")


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 (ties to even) of float32 values, kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    nan = np.isnan(a)
    out = r.view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


def conv_channels(layers, c_in: int):
    """Input channel count of every layer (channel bookkeeping for drawing
    weights of the right shape; a conv sets the count, a pool keeps it)."""
    chans = []
    c = c_in
    for L in layers:
        chans.append(c)
        if L["op"] == CONV:
            c = L["c_out"]
    return chans


def make_inputs(layers, h: int, w: int, c: int, batch: int = 1, seed: int = 0,
                dtype: str = "f32"):
    """Draws the seeded synthetic input and parameters (recipe above).
    Returns dict(x, w, scale, bias); per-layer lists hold None for pools."""
    rng = np.random.default_rng(seed)
    x = rng.random((batch, h, w, c), dtype=np.float32)
    ws, ss, bs = [], [], []
    for L, cin in zip(layers, conv_channels(layers, c)):
        if L["op"] != CONV:
            ws.append(None); ss.append(None); bs.append(None)
            continue
        f, co = L["f"], L["c_out"]
        std = np.float32(np.sqrt(2.0 / (cin * f * f)))
        wt = (rng.standard_normal((co, f, f, cin), dtype=np.float32) * std).astype(np.float32)
        sc = rng.uniform(0.5, 1.5, size=co).astype(np.float32)
        bi = (rng.standard_normal(co, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
        ws.append(wt); ss.append(sc); bs.append(bi)
    if dtype == "bf16":
        x = bf16_round(x)
        ws = [None if a is None else bf16_round(a) for a in ws]
        ss = [None if a is None else bf16_round(a) for a in ss]
        bs = [None if a is None else bf16_round(a) for a in bs]
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return {"x": x, "w": ws, "scale": ss, "bias": bs}


def workload_inputs(wl: Workload):
    return make_inputs(wl.layers, wl.h, wl.w, wl.c, wl.batch, wl.seed, wl.dtype)
