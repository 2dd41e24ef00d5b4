"""The benchmark's flop accounting against the layer shapes.

One traced step of each workload, run the way bench.py runs it (the
AlexNet-shaped training step at batch 256; the single-layer workload with
its input gradient): the work the library's trace tags on the conv / FC
GEMM kernels must equal the algorithmic flops of the step's conv / FC passes
computed from the workload's layer shapes (2 x the multiply-adds of the
direct definition, padded taps included, every layer's forward pass, filter
gradient and input gradient except the first layer's input gradient), and
every GEMM kernel that ran must be one bench.py counts.
"""
import numpy as np
import pytest
import torch

import bench
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _layer_flops(w, batch):
    """Per conv / FC layer: 2 N P Q K C R S from the listed shapes."""
    out = []
    c, h, ww = w.in_shape
    for l in w.layers:
        if isinstance(l, (wl.Conv, wl.FC)):
            k, p, q = l.out_shape
            r = l.kernel if isinstance(l, wl.Conv) else h
            s = l.kernel if isinstance(l, wl.Conv) else ww
            out.append(2.0 * batch * p * q * k * c * r * s)
        if isinstance(l, (wl.Conv, wl.Pool, wl.FC)):
            c, h, ww = l.out_shape
    return out


@pytest.mark.parametrize("index", [1, 2, 3, 4, 5])
def test_traced_conv_flops_equal_layer_shapes(index):
    from paper_1603_07846_amd import net as gnet
    from paper_1603_07846_amd import singa
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w)
    net = gnet.Net(w, concurrent_wgrad=False)
    net.load_params(inp.params)
    x = net.to_device_input(inp.x)
    labels = torch.from_numpy(inp.labels).cuda() if inp.labels is not None else None
    dy = net.to_device_input(inp.dy) if inp.dy is not None else None
    need_dx = index == 1
    singa.trace_enable(True)
    net.train_one_batch(x, labels=labels, dy_top=dy, need_input_grad=need_dx)
    torch.cuda.synchronize()
    singa.trace_enable(False)
    recs = singa.trace_records()
    traced = sum(r[2] for r in recs if bench.is_conv_kernel(r[0]))
    per_layer = _layer_flops(w, w.batch)
    expected = sum(per_layer) * 3 - (0 if need_dx else per_layer[0])
    assert traced == pytest.approx(expected, rel=1e-12), (traced, expected)
    assert bench.step_conv_flops(w, w.batch, need_dx) == pytest.approx(expected, rel=1e-12)
    gemm = {r[0] for r in recs if r[3] == "flop"}
    assert all(bench.is_conv_kernel(n) for n in gemm), gemm
    if index == 5:
        assert abs(traced / 1e9 - 1689.78) < 0.01, traced
        assert any(n.startswith("conv_wgrad_large_kernel") for n in gemm), gemm
    if index == 4:
        assert abs(traced / 1e9 - 1599.74) < 0.01, traced
    assert np.isfinite(traced)
