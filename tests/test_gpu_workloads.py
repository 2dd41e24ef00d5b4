"""End-to-end parity of the five workloads (BPTrainOneBatch + Updater) on the GPU.

* Workloads 1 and 2 run at full size and every produced tensor is compared
  element by element with the oracle: each layer's output, the Param
  gradients, the input gradients, the loss and the updated parameters and
  momentum.
* Workloads 3-5 (AlexNet-shaped) run the same comparison at batch 2, with
  the same layer shapes and kernels as the full batch.
* At their full batch (128 / 256) they run in the benchmark's launch
  configuration and are checked on what the oracle can evaluate in seconds:
  every layer's output for two sampled images (the forward pass of an image
  depends on that image alone), the loss against its closed form at the
  initial weights, and the batch-sum property of the filter gradient.

bf16 workloads are compared (rel-L2 <= 2e-2) against the oracle run on the
same bf16 inputs with its activations and activation gradients rounded to bf16
where the kernels store bf16, so that ReLU masks and max-pool argmaxes are
decided on the same stored values on both sides; fp32 workloads at 1e-4 with
no rounding.  The forward activations are also checked against the oracle's
unrounded fp64 pass.

The ReLU backward runs in place on the incoming gradient buffer, so after a
step the buffer a layer wrote its input gradient to holds the gradient at the
input of the ReLU below it when there is one; the comparison follows that.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import net as onet
from _helpers import TOL, rel_l2
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    global gnet
    from paper_1603_07846_amd import net as g
    gnet = g
    assert torch.cuda.is_available()
    yield


def _nhwc_to_nchw(t):
    a = t.detach().float().cpu().numpy().astype(np.float64)
    return a.transpose(0, 3, 1, 2) if a.ndim == 4 else a


def _oracle_params(inp, dtype):
    """Values the layers compute with: the bf16 rounding of the master for bf16 workloads."""
    if dtype == "bf16":
        return [(wl.round_bf16(p.w), p.b) for p in inp.params]
    return [(p.w, p.b) for p in inp.params]


def _run_gpu(w, inp, batch, need_input_grad):
    net = gnet.Net(w, batch=batch)
    net.load_params(inp.params)
    x = net.to_device_input(inp.x)
    labels = torch.from_numpy(inp.labels).cuda() if inp.labels is not None else None
    dy = net.to_device_input(inp.dy) if inp.dy is not None else None
    gx = net.train_one_batch(x, labels=labels, dy_top=dy, need_input_grad=need_input_grad)
    torch.cuda.synchronize()
    return net, gx


def _output_of(ref, layers, i):
    """Oracle output that the GPU layer i holds (a fused ReLU's output for a conv followed by ReLU)."""
    l = layers[i]
    if isinstance(l, (wl.Conv, wl.FC)) and i + 1 < len(layers) and isinstance(layers[i + 1], wl.Relu):
        return ref["acts"]["out"][layers[i + 1].name]
    return ref["acts"]["out"][l.name]


def _compare(net, ref, w, tol, need_input_grad):
    errs = {}
    layers = w.layers
    for i, (spec, l) in enumerate(zip(layers, net.layers)):
        if isinstance(spec, wl.SoftmaxCE):
            errs["loss"] = abs(float(l.loss[0].item()) - ref["acts"]["loss"]) / abs(ref["acts"]["loss"])
            continue
        if isinstance(spec, wl.Relu) and l.fused is not None:
            continue
        got = _nhwc_to_nchw(l.y)
        errs["y:" + spec.name] = rel_l2(got, _output_of(ref, layers, i).reshape(got.shape))
    names = [s.name for s in layers if isinstance(s, (wl.Conv, wl.FC))]
    for name, l, (wn, bn) in zip(names, net.param_layers(), ref["params"]):
        K = l.w_shape[0]
        dw = l.dw.detach().cpu().numpy().transpose(0, 3, 1, 2).reshape(ref["grads"]["dw"][name].shape)
        errs["dw:" + name] = rel_l2(dw, ref["grads"]["dw"][name])
        if l.has_bias:
            errs["db:" + name] = rel_l2(l.db.cpu().numpy(), ref["grads"]["db"][name])
        if w.update:
            wnew = l.w.detach().cpu().numpy().transpose(0, 3, 1, 2).reshape(wn.shape)
            errs["w':" + name] = rel_l2(wnew, wn)
    for i, (spec, l) in enumerate(zip(layers, net.layers)):
        if isinstance(spec, (wl.Conv, wl.FC, wl.Pool)) and (i > 0 or need_input_grad):
            got = _nhwc_to_nchw(l.dx)
            # a ReLU below this layer has masked the buffer in place
            below = layers[i - 1] if i > 0 and isinstance(layers[i - 1], wl.Relu) else spec
            errs["dx:" + spec.name] = rel_l2(got, ref["grads"]["grad_in"][below.name].reshape(got.shape))
    bad = {k: v for k, v in errs.items() if not v <= tol}
    return errs, bad


def _train_ref(w, inp, need_input_grad, mirror=True):
    store = oracle.round_bf16 if (w.dtype == "bf16" and mirror) else None
    return onet.train_one_batch(w.layers, inp.x, _oracle_params(inp, w.dtype),
                                master=[(p.w, p.b) for p in inp.params], labels=inp.labels, dy_top=inp.dy,
                                lr=w.lr, momentum=w.momentum, wd=w.weight_decay, need_input_grad=need_input_grad,
                                store=store)


def test_workload1_full():
    w = wl.CFG1
    inp = wl.make_inputs(w)
    net, gx = _run_gpu(w, inp, None, True)
    ref = _train_ref(w, inp, True)
    errs, bad = _compare(net, ref, w, TOL["f32"], True)
    # momentum after one step from zero: v = lr * g
    l = net.param_layers()[0]
    v = net.v_flat[:l.w.numel()].view(l.w_shape).cpu().numpy().transpose(0, 3, 1, 2)
    errs["v'"] = rel_l2(v, ref["velocity"][0][0])
    assert not bad and errs["v'"] <= TOL["f32"], errs


def test_workload2_full():
    w = wl.CFG2
    inp = wl.make_inputs(w)
    net, _ = _run_gpu(w, inp, None, False)
    ref = _train_ref(w, inp, False)
    errs, bad = _compare(net, ref, w, TOL["f32"], False)
    assert not bad, bad
    assert abs(ref["acts"]["loss"] - np.log(10)) < 1e-2


# Free-running bf16 backward: the first ReLU mask in the backward pass is decided
# on forward values that differ from the oracle's by the accumulated bf16
# rounding drift (~1e-3 rel-L2 at the last layers); pre-activations within that
# drift of zero flip, and with random labels / upstream gradients each flip is
# an O(1) change of a gradient element.  Measured effect at batch 2: ~1.5e-2
# (workload 4) and ~7e-2 (workload 5) rel-L2 below the first mask.  The
# free-running bf16 backward is therefore held to this sanity bound, and the
# 2e-2 bound is checked per layer on the real data flow (teacher-forced test).
BF16_FREE_RUNNING_BACKWARD = 1.5e-1


@pytest.mark.parametrize("index", [3, 4, 5])
def test_alexnet_workloads_batch2(index):
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w, batch=2)
    net, gx = _run_gpu(w, inp, 2, True)
    ref = _train_ref(w, inp, True)
    errs, _ = _compare(net, ref, w, TOL[w.dtype], True)
    print("workload %d batch 2 worst rel-L2: %s" % (index, max(errs.items(), key=lambda kv: kv[1])))
    if w.dtype == "f32":
        bad = {k: v for k, v in errs.items() if not v <= TOL["f32"]}
        assert not bad, bad
        return
    # forward, loss, updated weights and every gradient above the first ReLU mask
    # of the backward pass (the last FC layer's Param gradients): 2e-2
    above = set()
    for spec in reversed(w.layers):
        if isinstance(spec, wl.Relu):
            break
        above.add(spec.name)
    strict = {k: v for k, v in errs.items()
              if k.startswith(("y:", "loss", "w':")) or (k.startswith(("dw:", "db:")) and k[3:] in above)}
    bad = {k: v for k, v in strict.items() if not v <= TOL["bf16"]}
    assert not bad, bad
    loose = {k: v for k, v in errs.items() if not v <= BF16_FREE_RUNNING_BACKWARD}
    assert not loose, loose
    # forward activations against the unrounded fp64 oracle as well
    plain = onet.forward(w.layers, inp.x, _oracle_params(inp, w.dtype), labels=inp.labels)
    for i, (spec, l) in enumerate(zip(w.layers, net.layers)):
        if isinstance(spec, wl.SoftmaxCE) or (isinstance(spec, wl.Relu) and l.fused is not None):
            continue
        got = _nhwc_to_nchw(l.y)
        err = rel_l2(got, _output_of({"acts": plain}, w.layers, i).reshape(got.shape))
        assert err <= TOL["bf16"], (spec.name, err)


def _dev(a, dt):
    a = np.asarray(a, np.float32)
    if a.ndim == 4:
        a = a.transpose(0, 2, 3, 1)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda().to(torch.bfloat16 if dt == "bf16" else torch.float32)


@pytest.mark.parametrize("index", [4, 5])
def test_bf16_backward_teacher_forced(index):
    """Each layer's GPU ComputeGradient, fed the oracle's stored (bf16) input
    activation and upstream gradient of the real step, against the oracle's
    gradients from the same inputs: rel-L2 <= 2e-2 for every tensor."""
    from paper_1603_07846_amd import singa
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w, batch=2)
    ref = _train_ref(w, inp, True)
    acts, grads = ref["acts"], ref["grads"]
    params = _oracle_params(inp, w.dtype)
    layers = w.layers
    pi = {s.name: i for i, s in enumerate([l for l in layers if isinstance(l, (wl.Conv, wl.FC))])}
    errs = {}
    for li in range(len(layers) - 1, -1, -1):
        spec = layers[li]
        if isinstance(spec, wl.SoftmaxCE):
            continue
        # upstream gradient = the oracle's gradient at this layer's output
        if li + 1 == len(layers):
            up = inp.dy
        elif isinstance(layers[li + 1], wl.SoftmaxCE):
            up = acts["dlogits"]
        else:
            up = grads["grad_in"][layers[li + 1].name]
        xin = acts["in"][spec.name]
        if isinstance(spec, wl.Relu):
            got = singa.relu_bwd(_dev(acts["out"][spec.name], "bf16"), _dev(up, "bf16"))
            torch.cuda.synchronize()
            np.testing.assert_array_equal(_nhwc_to_nchw(got), grads["grad_in"][spec.name])
            continue
        if isinstance(spec, wl.Pool):
            shape = (xin.shape[0], xin.shape[2], xin.shape[3], xin.shape[1])
            _, am = singa.pool_fwd(_dev(xin, "bf16"), spec.mode, spec.kernel, spec.stride, spec.pad,
                                   spec.ceil_mode)
            got = singa.pool_bwd(_dev(up, "bf16"), am, shape, spec.mode, spec.kernel, spec.stride, spec.pad,
                                 spec.ceil_mode)
            torch.cuda.synchronize()
            errs["dx:" + spec.name] = rel_l2(_nhwc_to_nchw(got), grads["grad_in"][spec.name])
            continue
        wk, bk = params[pi[spec.name]]
        if isinstance(spec, wl.FC):
            N, C, H, W = xin.shape
            wk = np.asarray(wk).reshape(-1, C, H, W)
            pad, stride = 0, 1
            up = np.asarray(up).reshape(N, -1, 1, 1)
        else:
            pad, stride = spec.pad, spec.stride
        wd = _dev(wk, "bf16")
        xd, upd = _dev(xin, "bf16"), _dev(up, "bf16")
        dw, db = singa.conv_bwd_filter(xd, upd, tuple(wd.shape), pad, stride)
        dx = singa.conv_bwd_data(upd, wd, tuple(xd.shape), pad, stride)
        torch.cuda.synchronize()
        rdw = grads["dw"][spec.name]
        errs["dw:" + spec.name] = rel_l2(dw.cpu().numpy().transpose(0, 3, 1, 2).reshape(rdw.shape), rdw)
        errs["db:" + spec.name] = rel_l2(db.cpu().numpy(), grads["db"][spec.name])
        rdx = grads["grad_in"][spec.name]
        if rdx is not None:
            errs["dx:" + spec.name] = rel_l2(_nhwc_to_nchw(dx), rdx.reshape(xin.shape))
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    print("workload %d teacher-forced worst rel-L2: %s" % (index, max(errs.items(), key=lambda kv: kv[1])))
    assert not bad, bad


@pytest.mark.parametrize("index", [3, 4, 5])
def test_alexnet_workloads_full_batch_sampled(index):
    w = wl.WORKLOADS[index]
    inp = wl.make_inputs(w)
    net, _ = _run_gpu(w, inp, None, False)
    # forward of two sampled images through the oracle
    pick = [0, w.batch - 1]
    sub = wl.Inputs(w, 2, inp.x[pick], inp.params,
                    labels=None if inp.labels is None else inp.labels[pick],
                    dy=None if inp.dy is None else inp.dy[pick])
    store = oracle.round_bf16 if w.dtype == "bf16" else None
    acts = onet.forward(w.layers, sub.x, _oracle_params(sub, w.dtype), labels=sub.labels, store=store)
    ref = {"acts": acts}
    tol = TOL[w.dtype]
    for i, (spec, l) in enumerate(zip(w.layers, net.layers)):
        if isinstance(spec, (wl.SoftmaxCE,)) or (isinstance(spec, wl.Relu) and l.fused is not None):
            continue
        got = _nhwc_to_nchw(l.y)[pick]
        err = rel_l2(got, _output_of(ref, w.layers, i).reshape(got.shape))
        assert err <= tol, (spec.name, err)
    if w.classes:
        # at N(0, 0.01) weights the logits are tiny: the loss is ln(classes) to ~1e-3,
        # and each row of dlogits sums to zero
        loss = float(net.layers[-1].loss[0].item())
        assert abs(loss - np.log(w.classes)) < 5e-3, loss
        dz = net.layers[-1].dz.float().reshape(w.batch, -1).sum(dim=1).abs().max().item()
        assert dz < 2e-2 / w.batch
    # batch-sum property of the second conv layer's filter gradient (any tensor of dy's shape will do)
    from paper_1603_07846_amd import singa
    l = net.param_layers()[1]
    half = w.batch // 2
    dw_full, _ = singa.conv_bwd_filter(l.x, l.y, l.w_shape, l.pad, l.stride)
    dw_a, _ = singa.conv_bwd_filter(l.x[:half], l.y[:half], l.w_shape, l.pad, l.stride)
    singa.conv_bwd_filter(l.x[half:], l.y[half:], l.w_shape, l.pad, l.stride, dw=dw_a, accumulate=True)
    torch.cuda.synchronize()
    assert rel_l2(dw_a.cpu().numpy(), dw_full.cpu().numpy()) <= 1e-5
