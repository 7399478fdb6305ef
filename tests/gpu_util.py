"""Helpers shared by the GPU tests: run the HIP library on a workload and
compare with the oracle."""
import numpy as np

from paper_2107_06960_amd import workloads as W


def require_gpu():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_gpu(layers, h, w, c, params, tiling, batch, dtype, x=None, want_cuts=True, sentinel=True, part=False,
            bounds=None, reuse=False, packed=False):
    """Runs the library (mafat_run_network) and returns float64 numpy output
    (and the cut tensors).  bounds: tile boundaries of the plan (Plan's
    `bounds`: None, "balanced" or per-group lists); reuse: row reuse;
    packed: packed weights."""
    import torch
    from paper_2107_06960_amd import mafat as M
    plan = M.Plan(layers, (h, w, c), tiling, stage_partition=part, bounds=bounds, row_reuse=reuse,
                  packed_weights=packed)
    net = M.Network(plan, params, batch, dtype)
    xt = net.input_tensor(params["x"] if x is None else x)
    if sentinel:
        net.y.fill_(float("nan"))
        for t in net.cuts:
            t.fill_(float("nan"))
    y = net.run(xt)
    torch.cuda.synchronize()
    out = y.float().cpu().numpy().astype(np.float64)
    cuts = [t.float().cpu().numpy().astype(np.float64) for t in net.cuts]
    return (out, cuts, net, xt) if want_cuts else out


def normwise_err(got, ref):
    """max |got - ref| / max |ref| (NaN if anything is NaN)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if np.isnan(got).any():
        return float("nan")
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


TOL = {"f32": 1e-4, "bf16": 2e-2}
