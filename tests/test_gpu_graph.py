"""A training step replayed from a HIP graph against the same step run eagerly.

Two nets start from the same parameters.  One runs train_one_batch eagerly
on one stream with every update after the backward loop, the other replays a
graph captured from its own train_one_batch, with the update fused into the
filter-gradient kernel where the net does that and the other filter
gradients on a second stream beside the backward-data passes.  Between
replays the program does eager work of its own (the eager net's step, a copy
into the captured input, synchronizations), and after every replay the
graph's loss, updated master weights, momentum and bf16 shadow must equal the
eager net's bit for bit: both run the same kernels, whose reductions have a
fixed order.  A fresh input is copied into the captured tensor before the
third replay to show that a replay reads the tensor's current contents.
"""
import numpy as np
import pytest
import torch

from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu


# every workload the benchmark times from a graph: the single layer (with its
# input gradient), the CIFAR-shaped net, the two conv stacks (upstream
# gradient given) and the AlexNet-shaped step
@pytest.mark.parametrize("index,batch", [(1, None), (2, 16), (3, 2), (4, 4), (5, 8)])
def test_graph_replay_matches_eager(index, batch):
    from paper_1603_07846_amd import net as gnet
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w, batch=batch, seed_offset=31)
    inp2 = wl.make_inputs(w, batch=batch, seed_offset=32)
    eager = gnet.Net(w, batch=batch, device="cuda:0", fuse_update=False, concurrent_wgrad=False)
    graphed = gnet.Net(w, batch=batch, device="cuda:0")
    if w.dtype == "bf16" and w.classes:
        assert any(l.fused_update for l in graphed.param_layers())
    for n in (eager, graphed):
        n.load_params(inp.params)
    xe = eager.to_device_input(inp.x)
    xg = graphed.to_device_input(inp.x)
    lab = torch.from_numpy(inp.labels).cuda() if inp.labels is not None else None
    dye = eager.to_device_input(inp.dy) if inp.dy is not None else None
    dyg = graphed.to_device_input(inp.dy) if inp.dy is not None else None
    need_dx = index == 1
    torch.cuda.synchronize()
    g = graphed.capture(xg, labels=lab, dy_top=dyg, need_input_grad=need_dx)
    torch.cuda.synchronize()
    for step in range(4):
        if step == 2:
            fresh = eager.to_device_input(inp2.x)
            xe.copy_(fresh)
            xg.copy_(fresh)
        eager.train_one_batch(xe, labels=lab, dy_top=dye, need_input_grad=need_dx)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        if lab is not None:
            assert torch.equal(graphed.layers[-1].loss, eager.layers[-1].loss), step
        assert torch.equal(graphed.w_flat, eager.w_flat), step
        assert torch.equal(graphed.v_flat, eager.v_flat), step
        if eager.wb_flat is not None:
            assert torch.equal(graphed.wb_flat, eager.wb_flat), step
        if lab is not None:
            assert np.isfinite(float(eager.layers[-1].loss[0]))


@pytest.mark.parametrize("index,batch,reduce_update", [(5, 8, False), (5, 32, False), (6, 8, False), (5, 256, False),
                                                       (5, 32, True), (5, 256, True)])
def test_two_stream_eager_matches_one_stream(index, batch, reduce_update):
    """The default step launched eagerly (filter gradients, and the fully
    connected layers' fused gradient + update, on the second stream; with
    reduce_update, the convolutions' updates applied by their split-K
    reductions there too) against one stream with every update after the
    backward loop: bit for bit, over three steps, with no synchronization
    inside a step."""
    from paper_1603_07846_amd import net as gnet
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w, batch=batch, seed_offset=33)
    one = gnet.Net(w, batch=batch, device="cuda:0", fuse_update=False, concurrent_wgrad=False)
    two = gnet.Net(w, batch=batch, device="cuda:0", reduce_update=reduce_update)
    assert two.wgrad_stream is not None and any(l.fused_update for l in two.param_layers())
    assert any(l.reduce_update for l in two.param_layers()) == reduce_update
    for n in (one, two):
        n.load_params(inp.params)
    x = one.to_device_input(inp.x)
    lab = torch.from_numpy(inp.labels).cuda()
    for step in range(3):
        one.train_one_batch(x, labels=lab)
        two.train_one_batch(x, labels=lab)
    torch.cuda.synchronize()
    assert torch.equal(two.layers[-1].loss, one.layers[-1].loss)
    assert torch.equal(two.w_flat, one.w_flat)
    assert torch.equal(two.v_flat, one.v_flat)
    assert torch.equal(two.wb_flat, one.wb_flat)
