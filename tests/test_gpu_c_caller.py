"""The C ABI from a plain C program (tests/c_caller/mafat_c_caller.c, built
by __graft_entry__.build()): plan (with plan flags: packed weights repacked
by mafat_pack_weights, row reuse), regions, workspace size, caller-owned
hipMalloc buffers, mafat_run_network and mafat_run_group on a stream of its
own, the short-workspace error -- no Python or torch in that process.  Its
regions must equal the oracle's and its output the oracle's forward within
each dtype's tolerance."""
import os
import subprocess

import numpy as np
import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import TOL, normwise_err, require_gpu

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c_caller", "mafat_c_caller")
OPS = {W.CONV: 0, W.MAXPOOL: 1}
ACTS = {W.LINEAR: 0, W.LEAKY: 1}


def _bf16_bits(a):
    """float32 values that are bfloat16 numbers -> their 16-bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    assert not np.any(u & 0xFFFF), "not bfloat16 values"
    return (u >> 16).astype(np.uint16)


def _write(d, name, a, dtype):
    a = np.ascontiguousarray(a, dtype=np.float32)
    (_bf16_bits(a) if dtype == "bf16" else a).tofile(os.path.join(d, name))


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,batch,tiling,flags", [("f32", 1, "3x3/8/2x2", 0), ("bf16", 2, "5x5/8/2x2", 0),
                                                     ("bf16", 1, "2x2/4/3x3/12/1x1", 0),
                                                     ("bf16", 1, "5x5/8/2x2", 6),    # row reuse, packed weights
                                                     ("f32", 2, "3x3/NoCut", 4)])    # row reuse
def test_c_caller(orc, tmp_path, dtype, batch, tiling, flags):
    require_gpu()
    assert os.path.exists(EXE), f"{EXE} is missing: run __graft_entry__.build() first"
    layers, (h, w, c) = W.YOLOV2_16, (96, 96, 3)
    gs, rows, cols = W.parse_tiling(tiling, len(layers))
    p = W.make_inputs(layers, h, w, c, batch, 71, dtype)
    d = str(tmp_path)
    with open(os.path.join(d, "config.txt"), "w") as f:
        f.write(f"{h} {w} {c} {batch} {1 if dtype == 'bf16' else 0} {len(layers)} {len(gs)} {flags}\n")
        for L in layers:
            f.write(f"{OPS[L['op']]} {int(L.get('c_out', 0))} {L['f']} {L['s']} {L['p']} {ACTS[L.get('act', W.LINEAR)]}\n")
        for g in range(len(gs)):
            f.write(f"{gs[g]} {rows[g]} {cols[g]}\n")
    _write(d, "x.bin", p["x"], dtype)
    for k, L in enumerate(layers):
        if L["op"] == W.CONV:
            _write(d, f"w{k}.bin", p["w"][k], dtype)
            np.ascontiguousarray(p["scale"][k], dtype=np.float32).tofile(os.path.join(d, f"s{k}.bin"))
            np.ascontiguousarray(p["bias"][k], dtype=np.float32).tofile(os.path.join(d, f"b{k}.bin"))
    print(f"[c caller] {h}x{w}x{c} {tiling} batch={batch} {dtype} flags={flags}", flush=True)
    r = subprocess.run([EXE, d], capture_output=True, text=True, timeout=120)
    print(r.stdout.strip(), r.stderr.strip()[-2000:], flush=True)
    assert r.returncode == 0, r.stderr
    # regions as the C program read them through mafat_plan_regions
    R = orc.regions(layers, h, w, c, gs, rows, cols)
    got = np.loadtxt(os.path.join(d, "regions.txt"), dtype=np.int64, ndmin=2)
    for g in range(len(gs)):
        mine = got[got[:, 0] == g][:, 2:]
        nt, nl = R[g].shape[0], R[g].shape[1]
        assert mine.shape == (nt * nl, 8)
        assert np.array_equal(mine.reshape(nt, nl, 8), R[g])
    dims = orc.shapes(layers, h, w, c)
    shape = (batch, int(dims[-1, 3]), int(dims[-1, 4]), int(dims[-1, 5]))
    raw = np.fromfile(os.path.join(d, "y.bin"), dtype=np.uint16 if dtype == "bf16" else np.float32)
    y = ((raw.astype(np.uint32) << 16).view(np.float32) if dtype == "bf16" else raw).reshape(shape)
    ref = orc.forward_layers(layers, h, w, c, p["x"], p)
    assert not np.isnan(y).any()
    err = normwise_err(y.astype(np.float64), ref)
    print(f"[c caller] normwise error {err:.3e}", flush=True)
    assert err <= TOL[dtype]
