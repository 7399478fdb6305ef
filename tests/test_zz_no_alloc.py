"""mafat_run_network_static (the entry point for callers that cannot
allocate device memory: its workspace is a static device array of the
library) against mafat_run_network with a caller-owned workspace, through
the C ABI.

Both run the same kernels on the same plan, so their outputs must be
identical bit for bit.  Two calls in a row, the second on a smaller input
(and the static array still holding the first call's intermediates), then a
third plan; the size limit is checked on the host.
"""
import ctypes

import numpy as np
import pytest

from paper_2107_06960_amd import mafat as M
from paper_2107_06960_amd import workloads as W

from gpu_util import require_gpu


def _static_run(plan, net, x):
    M.mafat_run_network_static(plan.handle, net.batch, net.code, x.data_ptr(), net.y.data_ptr(),
                               [c.data_ptr() for c in net.cuts], net._wp, net._sp, net._bp,
                               M._stream_handle(None))


@pytest.mark.gpu
def test_static_workspace_equals_caller_workspace():
    require_gpu()
    import torch
    cases = [  # the benchmark workload, then a smaller input, then another network and dtype,
               # then row reuse (its band take-over copies run on the static array too)
        (W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2", 1, "bf16", 0, False),
        (W.YOLOV2_16, (200, 168, 3), "3x2/8/2x2", 2, "bf16", 1, False),
        (W.TINY, (64, 64, 3), "2x2", 1, "f32", 2, False),
        (W.YOLOV2_16, (608, 608, 3), "5x5/8/2x2", 1, "bf16", 3, True),
    ]
    for layers, hwc, tiling, batch, dtype, seed, reuse in cases:
        print(f"[no-alloc] {len(layers)} layers {hwc} {tiling} batch={batch} {dtype} row_reuse={reuse}", flush=True)
        plan = M.Plan(layers, hwc, tiling, packed_weights=True, row_reuse=reuse)
        assert plan.workspace_size(batch, dtype) <= M.MAFAT_STATIC_WORKSPACE_MIB << 20
        p = W.make_inputs(layers, *hwc, batch, seed, dtype)
        net = M.Network(plan, p, batch, dtype)
        x = net.input_tensor(p["x"])
        ref = net.run(x).clone()
        ref_cuts = [c.clone() for c in net.cuts]
        net.y.fill_(float("nan"))
        for c in net.cuts:
            c.fill_(float("nan"))
        torch.cuda.synchronize()
        _static_run(plan, net, x)
        torch.cuda.synchronize()
        assert torch.equal(net.y, ref)
        for a, b in zip(net.cuts, ref_cuts):
            assert torch.equal(a, b)
        del net, x


def test_static_workspace_limit_is_checked_first():
    # a plan whose workspace exceeds the static array fails before any HIP
    # call, with a message naming both sizes (host-only)
    L = M.lib()
    wl = W.WORKLOADS["yolo608_4x4_12_1x1_b8"]
    plan = M.Plan(wl.layers, (wl.h, wl.w, wl.c), wl.tiling)
    assert plan.workspace_size(wl.batch, wl.dtype) > M.MAFAT_STATIC_WORKSPACE_MIB << 20
    fake = 1 << 20
    w = M._ptrs([fake] * len(wl.layers))
    rc = L.mafat_run_network_static(plan.handle, wl.batch, M.MAFAT_BF16, fake, fake * 4, M._ptrs([fake * 8]),
                                    w, w, w, None)
    assert rc == M.MAFAT_EWORKSPACE
    assert b"static workspace" in L.mafat_last_error()
    assert L.mafat_run_network_static(None, 1, 0, fake, fake, None, w, w, w, None) == M.MAFAT_EINVAL
    assert L.mafat_run_network_static(plan.handle, 0, 0, fake, fake, None, w, w, w, None) == M.MAFAT_EINVAL
