"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times (NHWC, batch 128 fp32 / 256 bf16).

Every layer shape of the AlexNet-shaped workloads is run on seeded inputs of
exactly that shape.  Convolutions are checked on 1,500 sampled outputs per
pass, each evaluated one by one by the oracle's point evaluators (a filter
gradient point sums over all N*P*Q output pixels); pooling, ReLU,
softmax-CE and the Updater are checked element by element over the whole
tensor.
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import TOL, rel_l2
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu

NPTS = 1500


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    global singa
    from paper_1603_07846_amd import singa as s
    singa = s
    yield


def _conv_layers(w):
    """(name, N, C, H, W, K, R, S, pad, stride) of every conv / FC layer of a workload."""
    out = []
    c, h, ww = w.in_shape
    for l in w.layers:
        if isinstance(l, wl.Conv):
            out.append((l.name, w.batch, c, h, ww, l.out_channels, l.kernel, l.kernel, l.pad, l.stride))
        elif isinstance(l, wl.FC):
            out.append((l.name, w.batch, c, h, ww, l.out_features, h, ww, 0, 1))
        if isinstance(l, (wl.Conv, wl.Pool, wl.FC)):
            c, h, ww = l.out_shape
    return out


CASES = [(3, l) for l in _conv_layers(wl.CFG3)] + [(4, l) for l in _conv_layers(wl.CFG4)] + \
        [(5, l) for l in _conv_layers(wl.CFG5) if l[0].startswith("fc")]


def _nchw_flat_to_nhwc_flat(idx, shape_nchw):
    n, c, h, w = np.unravel_index(idx, shape_nchw)
    N, C, H, W = shape_nchw
    return ((n * H + h) * W + w) * C + c


def _to_dev(a_nchw, dt):
    t = torch.from_numpy(np.ascontiguousarray(a_nchw.transpose(0, 2, 3, 1)))
    return t.cuda().to(torch.bfloat16 if dt == "bf16" else torch.float32)


def _take(t, idx):
    return t.reshape(-1)[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("index,layer", CASES, ids=["w%d-%s" % (i, l[0]) for i, l in CASES])
def test_conv_layer_full_size(index, layer):
    name, N, C, H, W, K, R, S, pad, stride = layer
    dt = wl.WORKLOADS[index].dtype
    seed = 500 + index * 10 + len(name) + K
    x = wl.random_array((N, C, H, W), seed, "normal", 1.0, dt)
    w = wl.random_array((K, C, R, S), seed + 1, "normal", 0.01, dt)
    b = wl.random_array((K,), seed + 2, "normal", 0.01, "f32")
    P, Q = oracle.conv_out(H, R, pad, stride), oracle.conv_out(W, S, pad, stride)
    dy = wl.random_array((N, K, P, Q), seed + 3, "normal", 1.0, dt)
    xd, dyd = _to_dev(x, dt), _to_dev(dy, dt)
    wd = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 2, 3, 1))).cuda().to(xd.dtype)
    y = singa.conv_fwd(xd, wd, torch.from_numpy(b).cuda(), pad, stride, relu=False)
    dx = singa.conv_bwd_data(dyd, wd, (N, H, W, C), pad, stride)
    dw, db = singa.conv_bwd_filter(xd, dyd, (K, R, S, C), pad, stride)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed)
    iy = rng.choice(N * K * P * Q, NPTS, replace=False)
    ix = rng.choice(N * C * H * W, NPTS, replace=False)
    iw = rng.choice(K * C * R * S, min(NPTS, K * C * R * S), replace=False)
    ref_y = oracle.conv_fwd_points(x, w, b, iy, pad=pad, stride=stride)
    ref_dx = oracle.conv_bwd_data_points(dy, w, x.shape, ix, pad=pad, stride=stride)
    ref_dw = oracle.conv_bwd_filter_points(x, dy, w.shape, iw, pad=pad, stride=stride)
    got_y = _take(y, _nchw_flat_to_nhwc_flat(iy, (N, K, P, Q)))
    got_dx = _take(dx, _nchw_flat_to_nhwc_flat(ix, (N, C, H, W)))
    k, c, r, s = np.unravel_index(iw, (K, C, R, S))
    got_dw = _take(dw, ((k * R + r) * S + s) * C + c)
    errs = {"y": rel_l2(got_y, ref_y), "dx": rel_l2(got_dx, ref_dx), "dw": rel_l2(got_dw, ref_dw),
            "db": rel_l2(db.cpu().numpy(), dy.astype(np.float64).sum(axis=(0, 2, 3)))}
    tol = TOL[dt]
    # dw and db are fp32 sums of exact products of representable inputs
    assert errs["y"] <= tol and errs["dx"] <= tol and errs["dw"] <= TOL["f32"] and errs["db"] <= TOL["f32"], errs


POOLS = [(3, (128, 96, 55, 55)), (3, (128, 256, 27, 27)), (4, (256, 96, 55, 55)), (4, (256, 256, 27, 27)),
         (5, (256, 256, 13, 13))]


@pytest.mark.parametrize("index,shape", POOLS, ids=["w%d-%dx%dx%dx%d" % ((i,) + s) for i, s in POOLS])
def test_maxpool_full_size(index, shape):
    dt = wl.WORKLOADS[index].dtype
    x = wl.random_array(shape, 700 + shape[1], "normal", 1.0, dt)
    x = np.maximum(x, 0)  # pooling follows a ReLU in these stacks: many all-zero windows (ties)
    ref_y, ref_am = oracle.pool_fwd(x, oracle.MAX, 3, 2, 0, True)
    y, am = singa.pool_fwd(_to_dev(x, dt), "max", 3, 2, 0, True)
    dy = wl.random_array(ref_y.shape, 701 + shape[1], "normal", 1.0, dt)
    dx = singa.pool_bwd(_to_dev(dy, dt), am, (shape[0], shape[2], shape[3], shape[1]), "max", 3, 2, 0, True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(am.cpu().numpy().transpose(0, 3, 1, 2), ref_am)
    np.testing.assert_array_equal(y.float().cpu().numpy().transpose(0, 3, 1, 2), ref_y)
    ref_dx = oracle.pool_bwd(dy, ref_am, shape, oracle.MAX, 3, 2, 0, True)
    assert rel_l2(dx.float().cpu().numpy().transpose(0, 3, 1, 2), ref_dx) <= TOL[dt]


def test_relu_full_size():
    n = 256 * 96 * 55 * 55
    x = wl.random_array((n,), 800, "normal", 1.0, "bf16")
    dy = wl.random_array((n,), 801, "normal", 1.0, "bf16")
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    y = singa.relu_fwd(xd)
    dx = singa.relu_bwd(y, torch.from_numpy(dy).cuda().to(torch.bfloat16))
    torch.cuda.synchronize()
    ref_y = oracle.relu_fwd(x)
    np.testing.assert_array_equal(y.float().cpu().numpy(), ref_y)
    np.testing.assert_array_equal(dx.float().cpu().numpy(), oracle.relu_bwd(ref_y, dy))


def test_softmax_ce_full_size():
    z = wl.random_array((256, 1000), 810, "normal", 0.05, "bf16")
    lab = np.random.default_rng(811).integers(0, 1000, 256).astype(np.int32)
    ref_loss, ref_dz = oracle.softmax_ce(z, lab)
    loss, dz = singa.softmax_ce(torch.from_numpy(z).cuda().to(torch.bfloat16), torch.from_numpy(lab).cuda())
    torch.cuda.synchronize()
    assert abs(loss[0].item() - ref_loss) <= 1e-5 * ref_loss
    assert rel_l2(dz.float().cpu().numpy(), ref_dz) <= TOL["bf16"]


def test_adagrad_full_size():
    n = 62378344
    w = wl.random_array((n,), 822, "normal", 0.01)
    g = wl.random_array((n,), 823, "normal", 1e-3)
    h = wl.random_array((n,), 824, "uniform01", 1e-6)  # a running sum of squares: non-negative
    wd, gd, hd = (torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda() for a in (w, g, h))
    wb = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    singa.adagrad_update(wd, gd, hd, wb, 0.01, 1e-6, 5e-4)
    torch.cuda.synchronize()
    w1, h1 = oracle.adagrad(w, g, h, 0.01, 1e-6, 5e-4)
    assert rel_l2(wd.cpu().numpy(), w1) <= TOL["f32"]
    assert rel_l2(hd.cpu().numpy(), h1) <= TOL["f32"]
    np.testing.assert_array_equal(wb.cpu().view(torch.int16).numpy().view(np.uint16), wl.bf16_bits(wd.cpu().numpy()))


def test_sgd_full_size():
    n = 62378344
    w = wl.random_array((n,), 820, "normal", 0.01)
    g = wl.random_array((n,), 821, "normal", 1e-3)
    v = np.zeros(n, np.float32)
    wd, gd, vd = (torch.from_numpy(a).cuda() for a in (w, g, v))
    wb = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    singa.sgd_momentum_update(wd, gd, vd, wb, 0.01, 0.9, 5e-4)
    torch.cuda.synchronize()
    w1, v1 = oracle.sgd_momentum(w, g, v, 0.01, 0.9, 5e-4)
    assert rel_l2(wd.cpu().numpy(), w1) <= TOL["f32"]
    assert rel_l2(vd.cpu().numpy(), v1) <= TOL["f32"]
    np.testing.assert_array_equal(wb.cpu().view(torch.int16).numpy().view(np.uint16), wl.bf16_bits(wd.cpu().numpy()))
