"""GPU: the library used from two host threads at once, each with its own
buffers and stream, one of them sharing its plan object with the other
(plans are read-only after creation).  Every result must equal the result
of the same run made alone, bit for bit (the library keeps no mutable state
between calls besides the thread-local error message)."""
import threading

import pytest

from paper_2107_06960_amd import workloads as W

from gpu_util import require_gpu

pytestmark = pytest.mark.gpu


def _net(M, layers, hwc, tiling, dtype, batch, seed, plan=None):
    p = W.make_inputs(layers, *hwc, batch, seed, dtype)
    plan = plan or M.Plan(layers, hwc, tiling, packed_weights=True)
    net = M.Network(plan, p, batch, dtype)
    return plan, net, net.input_tensor(p["x"])


def test_two_threads_two_streams_bit_identical():
    require_gpu()
    import torch
    from paper_2107_06960_amd import mafat as M
    print("[concurrency] two host threads, two streams, a shared plan", flush=True)
    plan_a, net_a, x_a = _net(M, W.YOLOV2_16, (96, 96, 3), "3x3/8/2x2", "bf16", 2, 81)
    _, net_b, x_b = _net(M, W.YOLOV2_16, (96, 96, 3), "3x3/8/2x2", "bf16", 2, 82, plan=plan_a)
    _, net_c, x_c = _net(M, W.TINY, (64, 64, 3), "2x2", "f32", 1, 83)
    torch.cuda.synchronize()
    ref = [n.run(x).clone() for n, x in ((net_a, x_a), (net_b, x_b), (net_c, x_c))]
    torch.cuda.synchronize()
    for n in (net_a, net_b, net_c):
        n.y.zero_()
    torch.cuda.synchronize()

    errors = []

    def worker(jobs, stream):
        try:
            with torch.cuda.stream(stream):
                for _ in range(25):
                    for n, x in jobs:
                        n.run(x, stream=stream)
            stream.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    t1 = threading.Thread(target=worker, args=([(net_a, x_a), (net_c, x_c)], s1))
    t2 = threading.Thread(target=worker, args=([(net_b, x_b)], s2))
    t1.start(); t2.start()
    t1.join(timeout=120); t2.join(timeout=120)
    assert not t1.is_alive() and not t2.is_alive()
    assert not errors, errors
    torch.cuda.synchronize()
    for got, want in zip((net_a.y, net_b.y, net_c.y), ref):
        assert torch.equal(got, want)
