"""Parity at the workloads' full sizes, in the launch configuration the
benchmark times (NHWC, batch 128 fp32 / 256 bf16).

Every conv / FC layer shape of the AlexNet-shaped workloads is run on seeded
inputs of exactly that shape.  Each pass is a GEMM over an output matrix
(forward: output pixels x filters; input gradient: input pixels x channels,
or images x (h, w, c) for a fully connected layer; filter gradient: filters x
taps); every tile any of the kernels uses starts at a multiple of 128 rows
and of 32 columns of that matrix and spans at least 128 x 96, so one sampled
point in every 128 x 32 block, plus the four corners, puts at least one
point in every output tile of whatever tiling ran (and every split-K
partition adds into every point of its tile).  The strided first layer's
input gradient is a GEMM over its space-to-depth form, whose rows are 4 x 4
blocks of input pixels: there one such block per 128 rows is checked whole.
Each point is evaluated one by one by the oracle's point evaluators and held
to a per-point bound (the output rounding plus fp32 accumulation error over
the sum of absolute products, which the same evaluators give on |x| and |w|),
and the sampled set to rel-L2.  The bias gradient is checked against the
oracle over the whole vector, and the full filter gradients of the bf16
stack's conv3-5 and of fc6-8 element by element.  Pooling, ReLU, softmax-CE
and the Updater are checked element by element over the whole tensor.
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import TOL, rel_l2, to_gpu
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu

BM, BN = 128, 32  # block grid that every kernel's output tiles are unions of
EPS32 = 2.0 ** -24
OUT_ROUND = {"f32": 2.0 ** -23, "bf16": 2.0 ** -7}  # twice the largest relative rounding error of a stored output


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
# filter gradients checked over every element (the bf16 benchmark stack's
# 3x3 layers and the fully connected layers)
FULL_DW = {(4, "conv3"), (4, "conv4"), (4, "conv5"), (5, "fc6"), (5, "fc7"), (5, "fc8")}


def block_points(rows, cols, rng, bm=BM, bn=BN):
    """(row, col) of one random element in every bm x bn block of a rows x
    cols matrix (ragged last blocks included) and of its four corners."""
    r0 = np.arange(0, rows, bm)
    c0 = np.arange(0, cols, bn)
    hr = np.minimum(bm, rows - r0)
    hc = np.minimum(bn, cols - c0)
    R = (r0[:, None] + (rng.random((len(r0), len(c0))) * hr[:, None]).astype(np.int64)).ravel()
    C = (c0[None, :] + (rng.random((len(r0), len(c0))) * hc[None, :]).astype(np.int64)).ravel()
    R = np.concatenate([R, [0, 0, rows - 1, rows - 1]])
    C = np.concatenate([C, [0, cols - 1, 0, cols - 1]])
    return R.astype(np.int64), C.astype(np.int64)


def _to_dev(a_nchw, dt):
    return to_gpu(np.ascontiguousarray(a_nchw.transpose(0, 2, 3, 1)), torch.bfloat16 if dt == "bf16" else torch.float32)


def _take(t, idx):
    return t.reshape(-1)[torch.from_numpy(idx).cuda()].float().cpu().numpy().astype(np.float64)


def _check_points(name, got, ref, absum, n_acc, dt_out):
    """rel-L2 over the sample and the per-point bound
    |got - ref| <= OUT_ROUND |ref| + 8 sqrt(n_acc) 2^-24 sum|a b|."""
    bound = OUT_ROUND[dt_out] * np.abs(ref) + 8.0 * np.sqrt(n_acc) * EPS32 * absum
    worst = float(np.max(np.abs(got - ref) / np.maximum(bound, 1e-300)))
    assert worst <= 1.0, (name, "per-point bound exceeded", worst)
    return rel_l2(got, ref), worst


@pytest.mark.parametrize("index,layer", CASES, ids=["w%d-%s" % (i, l[0]) for i, l in CASES])
def test_conv_layer_full_size(index, layer):
    name, N, C, H, W, K, R, S, pad, stride = layer
    dt = wl.WORKLOADS[index].dtype
    fc = R == H and S == W and pad == 0 and H > 1 and name.startswith("fc")
    seed = 500 + index * 10 + len(name) + K
    x = wl.random_array((N, C, H, W), seed, "normal", 1.0, dt)
    w = wl.random_array((K, C, R, S), seed + 1, "normal", 0.01, dt)
    b = wl.random_array((K,), seed + 2, "normal", 0.01, "f32")
    P, Q = oracle.conv_out(H, R, pad, stride), oracle.conv_out(W, S, pad, stride)
    dy = wl.random_array((N, K, P, Q), seed + 3, "normal", 1.0, dt)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    xd = to_gpu(np.ascontiguousarray(x.transpose(0, 2, 3, 1)), tdt)
    dyd = to_gpu(np.ascontiguousarray(dy.transpose(0, 2, 3, 1)), tdt)
    wd = to_gpu(np.ascontiguousarray(w.transpose(0, 2, 3, 1)), tdt)
    y = singa.conv_fwd(xd, wd, to_gpu(b), pad, stride, relu=False)
    dx = singa.conv_bwd_data(dyd, wd, (N, H, W, C), pad, stride)
    dw, db = singa.conv_bwd_filter(xd, dyd, (K, R, S, C), pad, stride)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed)
    ax, aw, ady, ab = np.abs(x), np.abs(w), np.abs(dy), np.abs(b)
    errs, worst = {}, {}

    # forward: rows (n, p, q), columns k
    r, c = block_points(N * P * Q, K, rng)
    n, p, q = r // (P * Q), (r // Q) % P, r % Q
    iy = ((n * K + c) * P + p) * Q + q
    ref = oracle.conv_fwd_points(x, w, b, iy, pad=pad, stride=stride)
    absum = oracle.conv_fwd_points(ax, aw, ab, iy, pad=pad, stride=stride)
    errs["y"], worst["y"] = _check_points(name + " y", _take(y, r * K + c), ref, absum, C * R * S, dt)

    # input gradient
    if fc:  # rows n, columns (h, w, c)
        r, c = block_points(N, H * W * C, rng)
        hh, ww_, cc = c // (W * C), (c // C) % W, c % C
        nn = r
    elif stride == 1:  # rows (n, h, w), columns c
        r, cc = block_points(N * H * W, C, rng)
        nn, hh, ww_ = r // (H * W), (r // W) % H, r % W
    else:  # space-to-depth rows: whole stride x stride pixel blocks, every channel
        Hs, Ws = P + (R + stride - 1) // stride - 1, Q + (S + stride - 1) // stride - 1
        rows = N * Hs * Ws
        r0 = np.arange(0, rows, BM)
        rr = np.concatenate([r0 + (rng.random(len(r0)) * np.minimum(BM, rows - r0)).astype(np.int64),
                             [0, rows - 1]])
        nb, hb, wb = rr // (Hs * Ws), (rr // Ws) % Hs, rr % Ws
        dh, dw_, cg = np.meshgrid(np.arange(stride), np.arange(stride), np.arange(C), indexing="ij")
        nn = np.repeat(nb, dh.size)
        hh = (hb[:, None] * stride + dh.ravel()[None, :]).ravel()
        ww_ = (wb[:, None] * stride + dw_.ravel()[None, :]).ravel()
        cc = np.tile(cg.ravel(), len(rr))
        keep = (hh < H) & (ww_ < W)
        nn, hh, ww_, cc = nn[keep], hh[keep], ww_[keep], cc[keep]
    ix = ((nn * C + cc) * H + hh) * W + ww_
    ref = oracle.conv_bwd_data_points(dy, w, x.shape, ix, pad=pad, stride=stride)
    absum = oracle.conv_bwd_data_points(ady, aw, x.shape, ix, pad=pad, stride=stride)
    got = _take(dx, ((nn * H + hh) * W + ww_) * C + cc)
    errs["dx"], worst["dx"] = _check_points(name + " dx", got, ref, absum, K * R * S, dt)

    # filter gradient: rows k, columns (r, s, c); every element where it is cheap enough
    if (index, name) in FULL_DW:
        ref_dw = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride, with_bias=False)
        abs_dw = oracle.conv_bwd_filter(ax, ady, w.shape, pad=pad, stride=stride, with_bias=False)
        got = dw.cpu().numpy().astype(np.float64).transpose(0, 3, 1, 2)
        errs["dw"], worst["dw"] = _check_points(name + " dw", got.ravel(), ref_dw.ravel(), abs_dw.ravel(),
                                                N * P * Q, "f32")
    else:
        if stride == 1:
            k, j = block_points(K, R * S * C, rng)
        else:  # space-to-depth taps: every tap of eight filters and of the last one
            ks = np.concatenate([rng.choice(K, min(K, 8), replace=False), [K - 1]])
            k = np.repeat(ks, R * S * C)
            j = np.tile(np.arange(R * S * C), len(ks))
        rr_, ss, cc = j // (S * C), (j // C) % S, j % C
        iw = ((k * C + cc) * R + rr_) * S + ss
        ref = oracle.conv_bwd_filter_points(x, dy, w.shape, iw, pad=pad, stride=stride)
        absum = oracle.conv_bwd_filter_points(ax, ady, w.shape, iw, pad=pad, stride=stride)
        errs["dw"], worst["dw"] = _check_points(name + " dw", _take(dw, k * R * S * C + j), ref, absum,
                                                N * P * Q, "f32")
    # bias gradient, every element: the oracle's filter gradient of a one-channel
    # all-ones input under a 1x1 filter is the sum of dy over (n, p, q), as is its db
    _, ref_db = oracle.conv_bwd_filter(np.ones((N, 1, P, Q)), dy, (K, 1, 1, 1), with_bias=True)
    abs_db = oracle.conv_bwd_filter(np.ones((N, 1, P, Q)), ady, (K, 1, 1, 1), with_bias=False).ravel()
    errs["db"], worst["db"] = _check_points(name + " db", db.cpu().numpy().astype(np.float64), ref_db, abs_db,
                                            N * P * Q, "f32")
    tol = TOL[dt]
    print("%s w%d: rel-L2 %s, worst point / bound %s" % (name, index, errs, worst))
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
    wd, gd, hd = (to_gpu(np.ascontiguousarray(a, np.float32)) for a in (w, g, h))
    wb = singa.empty((n,), torch.bfloat16, "cuda")
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
    wd, gd, vd = (to_gpu(a) for a in (w, g, v))
    wb = singa.empty((n,), torch.bfloat16, "cuda")
    singa.sgd_momentum_update(wd, gd, vd, wb, 0.01, 0.9, 5e-4)
    torch.cuda.synchronize()
    w1, v1 = oracle.sgd_momentum(w, g, v, 0.01, 0.9, 5e-4)
    assert rel_l2(wd.cpu().numpy(), w1) <= TOL["f32"]
    assert rel_l2(vd.cpu().numpy(), v1) <= TOL["f32"]
    np.testing.assert_array_equal(wb.cpu().view(torch.int16).numpy().view(np.uint16), wl.bf16_bits(wd.cpu().numpy()))
