"""GPU parity of every C-ABI operation against the CPU oracle.

Each case draws seeded inputs (representable in the tested dtype), runs the
HIP library through the Python binding and the fp64 oracle on the same values,
and compares element by element: rel-L2 <= 1e-4 (fp32) or 2e-2 (bf16, fp32
accumulation); integer outputs (max-pool argmax) must match exactly.
Shapes are chosen to span several 128 x 128 tiles and ragged tails in M, N
and K, channel counts that do and do not allow vector loads, strides 1/2/4 and
the dense fully connected geometry.
"""
import numpy as np
import pytest
import torch

import oracle
from _helpers import TOL, dev_to_nchw, filt_to_kcrs, fphys, gpu_full, kcrs_to_dev, nchw_to_dev, phys, rel_l2, to_gpu
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _singa():
    global singa
    from paper_1603_07846_amd import singa as s
    singa = s
    assert torch.cuda.is_available()
    yield


# N, C, H, W, K, R, S, pad, stride
CONV_CASES = [
    (2, 3, 13, 13, 5, 3, 3, 1, 1),       # C=3: element-wise tap loads, K tail
    (2, 8, 9, 9, 16, 5, 5, 2, 1),        # vector loads in both dtypes
    (3, 32, 17, 17, 40, 3, 3, 1, 2),     # stride 2, M and N tails
    (2, 3, 35, 35, 8, 11, 11, 0, 4),     # AlexNet conv1 geometry, shrunk
    (4, 64, 7, 7, 130, 3, 3, 1, 1),      # two N tiles
    (2, 96, 27, 27, 256, 5, 5, 2, 1),    # AlexNet conv2 shape at batch 2
    (3, 24, 3, 3, 10, 3, 3, 0, 1),       # fully connected as whole-input conv
    (7, 40, 1, 1, 20, 1, 1, 0, 1),       # 1x1 on 1x1 (FC)
    (1, 16, 6, 5, 12, 1, 1, 0, 1),       # 1x1, non-square
    (2, 12, 8, 8, 9, 3, 3, 2, 1),        # pad 2 with a 3x3 kernel
    (4, 64, 4, 4, 200, 4, 4, 0, 1),      # FC, few rows, long reduction: split-K forward
    (5, 256, 2, 2, 520, 2, 2, 0, 1),     # FC: split-K forward and split-K backward-data
    (3, 5, 9, 9, 16, 3, 3, 1, 1),        # C=5: zero-padded channels in the forward pass
    (2, 12, 10, 10, 24, 3, 3, 1, 1),     # C=12: bf16 8-byte tap halves that wrap to the next tap
    (3, 4, 19, 19, 16, 5, 5, 2, 2),      # C=4, filter rows of 100 taps: 8-byte halves for both operands
    (3, 5, 3, 3, 16, 3, 3, 0, 1),        # FC with 45 inputs: backward-data through a transposed copy
    (2, 3, 33, 33, 8, 7, 7, 3, 4),       # space-to-depth rewrite with padding
    (1, 3, 6, 1400, 4, 3, 3, 1, 2),      # stride 2 on 3 channels: space-to-depth (f32), padded channels (bf16)
]


def _ids(cases):
    return ["x".join(str(v) for v in c) for c in cases]


def _conv_inputs(case, dt, seed):
    N, C, H, W, K, R, S, pad, stride = case
    x = wl.random_array((N, C, H, W), seed, "normal", 1.0, dt)
    w = wl.random_array((K, C, R, S), seed + 1, "normal", 0.1, dt)
    b = wl.random_array((K,), seed + 2, "normal", 0.5, "f32")
    P = oracle.conv_out(H, R, pad, stride)
    Q = oracle.conv_out(W, S, pad, stride)
    dy = wl.random_array((N, K, P, Q), seed + 3, "normal", 1.0, dt)
    return x, w, b, dy


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", CONV_CASES, ids=_ids(CONV_CASES))
def test_conv_fwd(case, layout, dt):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, _ = _conv_inputs(case, dt, 10)
    for relu in (False, True):
        ref = oracle.conv_fwd(x, w, b, pad=pad, stride=stride)
        if relu:
            ref = oracle.relu_fwd(ref)
        y = singa.conv_fwd(nchw_to_dev(x, dt, layout), kcrs_to_dev(w, dt, layout),
                           torch.from_numpy(b).cuda(), pad, stride, relu=relu, layout=layout)
        torch.cuda.synchronize()
        got = dev_to_nchw(y, layout)
        assert got.shape == ref.shape
        err = rel_l2(got, ref)
        assert err <= TOL[dt], (case, relu, err)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", CONV_CASES, ids=_ids(CONV_CASES))
def test_conv_bwd_data(case, layout, dt):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 20)
    ref = oracle.conv_bwd_data(dy, w, x.shape, pad=pad, stride=stride)
    dx = singa.conv_bwd_data(nchw_to_dev(dy, dt, layout), kcrs_to_dev(w, dt, layout), phys(x.shape, layout),
                             pad, stride, layout=layout)
    torch.cuda.synchronize()
    err = rel_l2(dev_to_nchw(dx, layout), ref)
    assert err <= TOL[dt], (case, err)


# dense (fully connected) backward-data in bf16: the GEMM reads the weight
# matrix as stored when the input width is a multiple of 8, else a transposed copy
FC_BWD_CASES = [((16, 256, 6, 6, 96, 6, 6, 0, 1), True), ((8, 64, 4, 4, 520, 4, 4, 0, 1), True),
                ((256, 1024, 1, 1, 4096, 1, 1, 0, 1), True), ((6, 7, 2, 2, 40, 2, 2, 0, 1), False)]


@pytest.mark.parametrize("case,direct", FC_BWD_CASES, ids=[_ids([c])[0] for c, _ in FC_BWD_CASES])
def test_fc_bwd_data_reads_weights_as_stored(case, direct):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, "bf16", 25)
    xr = np.maximum(x, 0.0)
    singa.trace_enable(True)
    dx = singa.conv_bwd_data(nchw_to_dev(dy, "bf16"), kcrs_to_dev(w, "bf16"), phys(x.shape), pad, stride,
                             relu_y=nchw_to_dev(xr, "bf16"))
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    assert any(n.startswith("conv_fwd_kernel<bf16,2,3,1>") for n in names) == direct, names
    assert (not any(n.startswith("transpose") for n in names)) == direct, names
    ref = oracle.relu_bwd(xr, oracle.conv_bwd_data(dy, w, x.shape, pad=pad, stride=stride))
    got = dev_to_nchw(dx)
    np.testing.assert_array_equal(got[xr <= 0], 0.0)
    assert rel_l2(got, ref) <= TOL["bf16"], case


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", CONV_CASES, ids=_ids(CONV_CASES))
def test_conv_bwd_filter(case, layout, dt):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 30)
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    dw, db = singa.conv_bwd_filter(nchw_to_dev(x, dt, layout), nchw_to_dev(dy, dt, layout), fphys(w.shape, layout),
                                   pad, stride, layout=layout)
    torch.cuda.synchronize()
    # inputs are exact in dt and dw/db accumulate in fp32: fp32 tolerance applies to both dtypes
    assert rel_l2(filt_to_kcrs(dw, layout), ref_dw) <= TOL["f32"]
    assert rel_l2(db.cpu().numpy(), ref_db) <= TOL["f32"]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_conv_bwd_filter_accumulate_shards(dt):
    # dim-0 partitioning: the gradient of the batch is the sum of the shards'
    case = (6, 16, 12, 12, 24, 3, 3, 1, 1)
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 40)
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    xd, dyd = nchw_to_dev(x, dt), nchw_to_dev(dy, dt)
    dw, db = singa.conv_bwd_filter(xd[:2], dyd[:2], fphys(w.shape), pad, stride)
    singa.conv_bwd_filter(xd[2:], dyd[2:], fphys(w.shape), pad, stride, dw=dw, db=db, accumulate=True)
    full_dw, full_db = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), pad, stride)
    torch.cuda.synchronize()
    assert rel_l2(filt_to_kcrs(dw), ref_dw) <= TOL["f32"]
    assert rel_l2(db.cpu().numpy(), ref_db) <= TOL["f32"]
    assert rel_l2(dw.cpu().numpy(), full_dw.cpu().numpy()) <= 1e-6


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", [(16, 16, 24, 24, 24, 3, 3, 1, 1), (8, 3, 35, 35, 8, 11, 11, 0, 4)],
                         ids=["split-K", "padded-channels"])
def test_conv_bwd_filter_accumulate_split(case, dt):
    # accumulate through the split-K reduction (and the channel-padded path)
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 41)
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    xd, dyd = nchw_to_dev(x, dt), nchw_to_dev(dy, dt)
    h = N // 2
    dw, db = singa.conv_bwd_filter(xd[:h], dyd[:h], fphys(w.shape), pad, stride)
    singa.conv_bwd_filter(xd[h:], dyd[h:], fphys(w.shape), pad, stride, dw=dw, db=db, accumulate=True)
    torch.cuda.synchronize()
    assert rel_l2(filt_to_kcrs(dw), ref_dw) <= TOL["f32"]
    assert rel_l2(db.cpu().numpy(), ref_db) <= TOL["f32"]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_conv_bwd_filter_without_bias(layout, dt):
    case = (4, 8, 11, 11, 16, 3, 3, 1, 1)
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 42)
    ref_dw, _ = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    dw, db = singa.conv_bwd_filter(nchw_to_dev(x, dt, layout), nchw_to_dev(dy, dt, layout), fphys(w.shape, layout),
                                   pad, stride, layout=layout, with_bias=False)
    torch.cuda.synchronize()
    assert db is None
    assert rel_l2(filt_to_kcrs(dw, layout), ref_dw) <= TOL["f32"]


# the 128 x 256 filter-gradient tile: several row tiles, direct and split
# reductions, image-fastest order with accumulation, no bias
LARGE_WGRAD_CASES = [
    ((8, 32, 15, 15, 512, 3, 3, 1, 1), True, False),    # two row tiles, ragged taps + bias, split reduction
    ((4, 64, 9, 9, 256, 3, 3, 1, 1), True, False),      # short reduction: one split, written directly
    ((32, 16, 12, 12, 256, 3, 3, 1, 1), True, True),    # image-fastest order, accumulated in two halves
    ((8, 32, 15, 15, 256, 3, 3, 1, 1), False, False),   # without bias
    ((6, 24, 13, 13, 304, 3, 3, 1, 1), True, False),    # 304 filters: ragged row tile
]


@pytest.mark.parametrize("case,bias,halves", LARGE_WGRAD_CASES,
                         ids=["x".join(map(str, c)) + ("-bias" if b else "") + ("-acc" if h else "")
                              for c, b, h in LARGE_WGRAD_CASES])
def test_conv_bwd_filter_large_tile(case, bias, halves):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, "bf16", 43)
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    xd, dyd = nchw_to_dev(x, "bf16"), nchw_to_dev(dy, "bf16")
    singa.trace_enable(True)
    if halves:
        h = N // 2
        dw, db = singa.conv_bwd_filter(xd[:h], dyd[:h], fphys(w.shape), pad, stride, with_bias=bias)
        singa.conv_bwd_filter(xd[h:], dyd[h:], fphys(w.shape), pad, stride, dw=dw, db=db, accumulate=True,
                              with_bias=bias)
    else:
        dw, db = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), pad, stride, with_bias=bias)
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    assert any(n.startswith("conv_wgrad_large_kernel") for n in names), names
    assert rel_l2(filt_to_kcrs(dw), ref_dw) <= TOL["f32"]
    if bias:
        assert rel_l2(db.cpu().numpy(), ref_db) <= TOL["f32"]
    else:
        assert db is None


# the 128 x 256 filter-gradient kernel with K-tiles of 32 images at one
# output pixel (batches that are multiples of 32, as in the benchmark):
# ragged rows and taps, the bias column in a ragged column tile, direct and
# split reductions, a strided padded layer, the space-to-depth first layer, a
# whole-input (fully connected) layer, and accumulation over two batches
PIXEL_WGRAD_CASES = [
    (32, 32, 15, 15, 512, 3, 3, 1, 1, True),     # two row tiles, ragged taps + bias, split reduction
    (32, 64, 3, 3, 256, 3, 3, 1, 1, True),       # nine K-tiles: one split, written directly
    (32, 24, 13, 13, 304, 3, 3, 1, 1, True),     # 304 filters: ragged row tile
    (64, 48, 7, 7, 96, 3, 3, 1, 1, False),       # 96 filters, no bias
    (32, 16, 20, 20, 256, 5, 5, 2, 2, True),     # stride 2, pad 2
    (32, 64, 4, 4, 520, 4, 4, 0, 1, True),       # whole-input layer, three column tiles
    (32, 3, 35, 35, 96, 11, 11, 0, 4, True),     # AlexNet conv1 geometry on its space-to-depth form
]


@pytest.mark.parametrize("case", PIXEL_WGRAD_CASES, ids=["x".join(map(str, c[:9])) + ("-bias" if c[9] else "")
                                                         for c in PIXEL_WGRAD_CASES])
def test_conv_bwd_filter_pixel_order(case):
    case, bias = case[:9], case[9]
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, "bf16", 44)
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    xd, dyd = nchw_to_dev(x, "bf16"), nchw_to_dev(dy, "bf16")
    singa.trace_enable(True)
    dw, db = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), pad, stride, with_bias=bias)
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    assert "conv_wgrad_large_kernel<1,0>" in names, names
    assert rel_l2(filt_to_kcrs(dw), ref_dw) <= TOL["f32"]
    if bias:
        assert rel_l2(db.cpu().numpy(), ref_db) <= TOL["f32"]
    else:
        assert db is None
    # bitwise reproducible: the partial tiles are summed in a fixed order
    dw2, db2 = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), pad, stride, with_bias=bias)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and (db is None or torch.equal(db, db2))


def test_conv_bwd_filter_pixel_order_accumulate():
    # the gradients of two batches of 32 added through the accumulate flag
    case = (32, 32, 9, 9, 384, 3, 3, 1, 1)
    N, C, H, W, K, R, S, pad, stride = case
    x1, w, b, dy1 = _conv_inputs(case, "bf16", 45)
    x2, _, _, dy2 = _conv_inputs(case, "bf16", 46)
    r1 = oracle.conv_bwd_filter(x1, dy1, w.shape, pad=pad, stride=stride)
    r2 = oracle.conv_bwd_filter(x2, dy2, w.shape, pad=pad, stride=stride)
    singa.trace_enable(True)
    dw, db = singa.conv_bwd_filter(nchw_to_dev(x1, "bf16"), nchw_to_dev(dy1, "bf16"), fphys(w.shape), pad, stride)
    singa.conv_bwd_filter(nchw_to_dev(x2, "bf16"), nchw_to_dev(dy2, "bf16"), fphys(w.shape), pad, stride, dw=dw,
                          db=db, accumulate=True)
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    assert names.count("conv_wgrad_large_kernel<1,0>") == 2, names
    assert rel_l2(filt_to_kcrs(dw), r1[0] + r2[0]) <= TOL["f32"]
    assert rel_l2(db.cpu().numpy(), r1[1] + r2[1]) <= TOL["f32"]


def test_conv_bwd_filter_deterministic():
    case = (4, 32, 15, 15, 48, 3, 3, 1, 1)
    x, w, b, dy = _conv_inputs(case, "f32", 50)
    xd, dyd = nchw_to_dev(x), nchw_to_dev(dy)
    a = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), 1, 1)
    c = singa.conv_bwd_filter(xd, dyd, fphys(w.shape), 1, 1)
    torch.cuda.synchronize()
    assert torch.equal(a[0], c[0]) and torch.equal(a[1], c[1])


def _s2d_reference(x_nhwc, R, S, pad, stride):
    """The space-to-depth input written out from its definition (NHWC)."""
    n, H, W, C = x_nhwc.shape
    P, Q = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1
    Rs, Ss = -(-R // stride), -(-S // stride)
    out = np.zeros((n, P + Rs - 1, Q + Ss - 1, stride * stride * C), x_nhwc.dtype)
    for hq in range(P + Rs - 1):
        for wq in range(Q + Ss - 1):
            for dh in range(stride):
                for dw in range(stride):
                    h, w = stride * hq + dh - pad, stride * wq + dw - pad
                    if 0 <= h < H and 0 <= w < W:
                        c0 = (dh * stride + dw) * C
                        out[:, hq, wq, c0:c0 + C] = x_nhwc[:, h, w, :]
    return out


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", [(2, 3, 35, 35, 8, 11, 11, 0, 4), (2, 3, 33, 33, 8, 7, 7, 3, 4)],
                         ids=["conv1-shrunk", "padded"])
def test_space_to_depth_input_layout(case, dt):
    """The caller-side space-to-depth input: its layout follows the
    definition, and the forward pass and filter gradient computed from it are
    bitwise those of the NHWC calls (which build the same form themselves)."""
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 71)
    xd, wd = nchw_to_dev(x, dt), kcrs_to_dev(w, dt)
    xs = singa.space_to_depth(xd, tuple(wd.shape), pad, stride)
    torch.cuda.synchronize()
    ref = _s2d_reference(np.ascontiguousarray(np.asarray(x, np.float32).transpose(0, 2, 3, 1)), R, S, pad, stride)
    assert np.array_equal(xs.float().cpu().numpy(), ref)
    bias = torch.from_numpy(b).cuda()
    y0 = singa.conv_fwd(xd, wd, bias, pad, stride, relu=True)
    y1 = singa.conv_fwd(xs, wd, bias, pad, stride, relu=True, layout="NHWC_S2D", x_shape=tuple(xd.shape))
    dyd = nchw_to_dev(dy, dt)
    dw0, db0 = singa.conv_bwd_filter(xd, dyd, tuple(wd.shape), pad, stride)
    dw1, db1 = singa.conv_bwd_filter(xs, dyd, tuple(wd.shape), pad, stride, layout="NHWC_S2D",
                                     x_shape=tuple(xd.shape))
    torch.cuda.synchronize()
    assert torch.equal(y0, y1) and torch.equal(dw0, dw1) and torch.equal(db0, db1)
    ref_y = oracle.relu_fwd(oracle.conv_fwd(x, w, b, pad=pad, stride=stride))
    assert rel_l2(dev_to_nchw(y1), ref_y) <= TOL[dt]
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, w.shape, pad=pad, stride=stride)
    assert rel_l2(filt_to_kcrs(dw1), ref_dw) <= TOL["f32"]
    assert rel_l2(db1.cpu().numpy(), ref_db) <= TOL["f32"]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("batch", [1, 3])
def test_space_to_depth_alexnet_conv1_layout(batch, dt):
    """AlexNet's first layer (227 x 227 x 3, 11 x 11 stride 4): the rewritten
    input at full image size, bit for bit against the definition; an odd
    batch puts the end of x inside a 16-byte chunk."""
    x = wl.random_array((batch, 3, 227, 227), 72, "normal", 1.0, dt)
    xd = nchw_to_dev(x, dt)
    xs = singa.space_to_depth(xd, (96, 11, 11, 3), 0, 4)
    torch.cuda.synchronize()
    ref = _s2d_reference(np.ascontiguousarray(np.asarray(x, np.float32).transpose(0, 2, 3, 1)), 11, 11, 0, 4)
    assert xs.shape == (batch, 57, 57, 48)
    assert np.array_equal(xs.float().cpu().numpy(), ref)


# N, C, H, W, mode, k, stride, pad
POOL_CASES = [
    (2, 32, 32, 32, "max", 3, 2, 0),   # CIFAR pool1 (ceil-mode edge windows)
    (2, 32, 16, 16, "avg", 3, 2, 0),
    (2, 64, 8, 8, "avg", 3, 2, 0),
    (2, 96, 55, 55, "max", 3, 2, 0),   # AlexNet pool1
    (3, 5, 13, 13, "max", 3, 2, 0),
    (2, 7, 9, 10, "max", 3, 2, 1),     # padded ceil mode
    (2, 7, 9, 10, "avg", 3, 2, 1),
    (1, 3, 7, 7, "avg", 2, 2, 0),
    (2, 16, 9, 10, "max", 3, 2, 1),    # padded, vector channels
    (2, 16, 9, 10, "avg", 3, 2, 1),
    (2, 8, 6, 6, "max", 3, 1, 1),      # overlapping stride-1 windows
]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", POOL_CASES, ids=_ids(POOL_CASES))
def test_pool(case, layout, dt):
    N, C, H, W, mode, k, s, p = case
    x = wl.random_array((N, C, H, W), 60, "normal", 1.0, dt)
    m = oracle.MAX if mode == "max" else oracle.AVG
    ref_y, ref_am = oracle.pool_fwd(x, m, k, s, p, True)
    y, am = singa.pool_fwd(nchw_to_dev(x, dt, layout), mode, k, s, p, True, layout=layout)
    dy = wl.random_array(ref_y.shape, 61, "normal", 1.0, dt)
    dx = singa.pool_bwd(nchw_to_dev(dy, dt, layout), am, phys(x.shape, layout), mode, k, s, p, True, layout=layout)
    torch.cuda.synchronize()
    assert rel_l2(dev_to_nchw(y, layout), ref_y) <= (TOL[dt] if mode == "avg" else 0.0)
    if mode == "max":
        got_am = am.cpu().numpy()
        if layout == "NHWC":
            got_am = got_am.transpose(0, 3, 1, 2)
        # same values compared in the same order: the argmax is exact
        np.testing.assert_array_equal(got_am, ref_am)
    ref_dx = oracle.pool_bwd(dy, ref_am, x.shape, m, k, s, p, True)
    assert rel_l2(dev_to_nchw(dx, layout), ref_dx) <= TOL[dt]


# ReLU backward folded into the pooling backward: the pooling's input is a
# ReLU output (many zeros, hence all-zero windows whose maximum is 0).
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", [c for c in POOL_CASES if c[4] == "max"], ids=_ids([c for c in POOL_CASES
                                                                                      if c[4] == "max"]))
def test_pool_bwd_relu_folded(case, layout, dt):
    N, C, H, W, mode, k, s, p = case
    x = np.maximum(wl.random_array((N, C, H, W), 62, "normal", 1.0, dt), 0.0)
    ref_y, ref_am = oracle.pool_fwd(x, oracle.MAX, k, s, p, True)
    y, am = singa.pool_fwd(nchw_to_dev(x, dt, layout), mode, k, s, p, True, layout=layout)
    dy = wl.random_array(ref_y.shape, 63, "normal", 1.0, dt)
    dx = singa.pool_bwd(nchw_to_dev(dy, dt, layout), am, phys(x.shape, layout), mode, k, s, p, True, layout=layout,
                        relu_y=y)
    torch.cuda.synchronize()
    ref_dx = oracle.relu_bwd(x, oracle.pool_bwd(dy, ref_am, x.shape, oracle.MAX, k, s, p, True))
    got = dev_to_nchw(dx, layout)
    np.testing.assert_array_equal(got[x <= 0], 0.0)
    assert rel_l2(got, ref_dx) <= TOL[dt]


def test_pool_bwd_relu_folded_rejects_avg():
    x = nchw_to_dev(np.ones((1, 8, 5, 5)), "f32")
    y, _ = singa.pool_fwd(x, "avg", 3, 2, 0, True)
    with pytest.raises(singa.SingaError):
        singa.pool_bwd(y, None, tuple(x.shape), "avg", 3, 2, 0, True, relu_y=y)


# ReLU backward folded into the backward-data pass: the layer's input is a
# ReLU output.  Covers the GEMM path (3x3 and 1x1), the dense geometry with
# split-K, the strided gather kernel and the 256 x 128 bf16 kernel.
RELU_FOLD_CASES = [
    (2, 12, 9, 9, 20, 3, 3, 1, 1),
    (5, 256, 2, 2, 520, 2, 2, 0, 1),
    (3, 32, 17, 17, 40, 3, 3, 1, 2),
    (2, 16, 6, 5, 12, 1, 1, 0, 1),
]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", RELU_FOLD_CASES, ids=_ids(RELU_FOLD_CASES))
def test_conv_bwd_data_relu_folded(case, layout, dt):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, dt, 90)
    xr = np.maximum(x, 0.0)
    ref = oracle.relu_bwd(xr, oracle.conv_bwd_data(dy, w, x.shape, pad=pad, stride=stride))
    dx = singa.conv_bwd_data(nchw_to_dev(dy, dt, layout), kcrs_to_dev(w, dt, layout), phys(x.shape, layout),
                             pad, stride, layout=layout, relu_y=nchw_to_dev(xr, dt, layout))
    torch.cuda.synchronize()
    got = dev_to_nchw(dx, layout)
    np.testing.assert_array_equal(got[xr <= 0], 0.0)
    assert rel_l2(got, ref) <= TOL[dt], case


@pytest.mark.parametrize("case", [(15, 200, 47, 47, 128, 3, 3, 1, 1), (30, 96, 47, 47, 40, 3, 3, 1, 1)])
def test_conv_bwd_data_relu_folded_large_tile(case):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, "bf16", 91)
    xr = np.maximum(x, 0.0)
    singa.trace_enable(True)
    dx = singa.conv_bwd_data(nchw_to_dev(dy, "bf16"), kcrs_to_dev(w, "bf16"), phys(x.shape), pad, stride,
                             relu_y=nchw_to_dev(xr, "bf16"))
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    assert any(n.startswith("conv_fwd_large_kernel") for n in names), names
    ref = oracle.relu_bwd(xr, oracle.conv_bwd_data(dy, w, x.shape, pad=pad, stride=stride))
    got = dev_to_nchw(dx)
    np.testing.assert_array_equal(got[xr <= 0], 0.0)
    assert rel_l2(got, ref) <= TOL["bf16"]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("n", [1, 7, 8, 1000, 4099, 1 << 20])
def test_relu(n, dt):
    x = wl.random_array((n,), 70, "normal", 1.0, dt)
    x[: min(n, 3)] = 0.0
    dy = wl.random_array((n,), 71, "normal", 1.0, dt)
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16 if dt == "bf16" else torch.float32)
    y = singa.relu_fwd(xd)
    dx = singa.relu_bwd(y, torch.from_numpy(dy).cuda().to(xd.dtype))
    inplace = xd.clone()
    singa.relu_fwd(inplace, out=inplace)
    torch.cuda.synchronize()
    ref_y = oracle.relu_fwd(x)
    np.testing.assert_array_equal(y.float().cpu().numpy(), ref_y)
    np.testing.assert_array_equal(inplace.float().cpu().numpy(), ref_y)
    np.testing.assert_array_equal(dx.float().cpu().numpy(), oracle.relu_bwd(ref_y, dy))


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(100, 10), (256, 1000), (3, 7), (1, 1)])
def test_softmax_ce(shape, dt):
    B, classes = shape
    z = wl.random_array(shape, 80, "normal", 2.0, dt)
    lab = np.random.default_rng(81).integers(0, classes, B).astype(np.int32)
    ref_loss, ref_dz = oracle.softmax_ce(z, lab)
    zd = torch.from_numpy(z).cuda().to(torch.bfloat16 if dt == "bf16" else torch.float32)
    loss, dz = singa.softmax_ce(zd, torch.from_numpy(lab).cuda())
    torch.cuda.synchronize()
    assert abs(loss[0].item() - ref_loss) <= 1e-5 * max(1.0, abs(ref_loss))
    assert rel_l2(dz.float().cpu().numpy(), ref_dz) <= TOL[dt]
    # per-row losses: the oracle's loss of each row as a batch of one
    rows = np.array([oracle.softmax_ce(z[n:n + 1], lab[n:n + 1])[0] for n in range(B)])
    assert rel_l2(loss[1:].cpu().numpy(), rows) <= 1e-5


@pytest.mark.parametrize("n", [1, 5, 2400, 89578, 1 << 20])
@pytest.mark.parametrize("shadow", [False, True])
def test_sgd_momentum(n, shadow):
    w = wl.random_array((n,), 90, "normal", 0.01)
    g = wl.random_array((n,), 91, "normal", 1.0)
    v = wl.random_array((n,), 92, "normal", 0.01)
    wd, vd, gd = to_gpu(w), to_gpu(v), to_gpu(g)
    wb = gpu_full((n,), 0.0, torch.bfloat16) if shadow else None
    for step in range(3):
        singa.sgd_momentum_update(wd, gd, vd, wb, lr=0.01, momentum=0.9, weight_decay=5e-4)
        w, v = oracle.sgd_momentum(w, g, v, 0.01, 0.9, 5e-4)
    torch.cuda.synchronize()
    assert rel_l2(wd.cpu().numpy(), w) <= TOL["f32"]
    assert rel_l2(vd.cpu().numpy(), v) <= TOL["f32"]
    if shadow:
        # the shadow is exactly the rounded master
        np.testing.assert_array_equal(wb.cpu().view(torch.int16).numpy().view(np.uint16),
                                      wl.bf16_bits(wd.cpu().numpy()))


@pytest.mark.parametrize("n", [1, 5, 7, 8, 2400, 89578, 1 << 20])
@pytest.mark.parametrize("shadow", [False, True])
def test_adagrad(n, shadow):
    w = wl.random_array((n,), 93, "normal", 0.01)
    g = wl.random_array((n,), 94, "normal", 1.0)
    h = np.zeros(n)
    wd, hd, gd = to_gpu(w), gpu_full((n,), 0.0), to_gpu(g)
    wb = gpu_full((n,), 0.0, torch.bfloat16) if shadow else None
    for step in range(3):
        singa.adagrad_update(wd, gd, hd, wb, lr=0.01, delta=1e-6, weight_decay=5e-4)
        w, h = oracle.adagrad(w, g, h, 0.01, 1e-6, 5e-4)
    torch.cuda.synchronize()
    assert rel_l2(wd.cpu().numpy(), w) <= TOL["f32"]
    assert rel_l2(hd.cpu().numpy(), h) <= TOL["f32"]
    if shadow:
        np.testing.assert_array_equal(wb.cpu().view(torch.int16).numpy().view(np.uint16),
                                      wl.bf16_bits(wd.cpu().numpy()))


def test_adagrad_errors():
    w = torch.zeros(64, device="cuda")
    with pytest.raises(singa.SingaError) as e:
        singa.adagrad_update(w, w, w, delta=0.0)
    assert e.value.status == -3
    with pytest.raises(singa.SingaError) as e:
        singa.adagrad_update(w[1:], w[1:], w[1:])
    assert e.value.status == -5


def test_abi_errors_launch_nothing():
    x = torch.zeros((2, 8, 8, 4), device="cuda")
    w = torch.zeros((4, 3, 3, 4), device="cuda")
    with pytest.raises(singa.SingaError) as e:
        singa.conv_fwd(x, torch.zeros((4, 3, 3, 5), device="cuda"))
    assert e.value.status == -2
    ws = torch.zeros(16, dtype=torch.uint8, device="cuda")
    xs = torch.zeros((16, 24, 24, 16), device="cuda")  # long reduction: split-K partial sums need workspace
    with pytest.raises(singa.SingaError) as e:
        singa.conv_bwd_filter(xs, torch.zeros((16, 24, 24, 4), device="cuda"), (4, 3, 3, 16), 1, 1, workspace=ws)
    assert e.value.status == -4
    with pytest.raises(singa.SingaError) as e:
        singa.relu_fwd(x.view(-1)[1:])
    assert e.value.status == -5


# Shapes big enough (>= 256 tiles, a long reduction) that the bf16 forward /
# backward-data passes take the 256 x 128 direct-to-LDS kernel (checked
# through the kernel trace), with ragged M, N and K tails and stride 2;
# compared element by element.
LARGE_CASES = [
    ("fwd", (10, 128, 47, 47, 300, 3, 3, 1, 1)),
    ("bwd_data", (15, 200, 47, 47, 128, 3, 3, 1, 1)),
    ("fwd", (40, 128, 59, 59, 136, 3, 3, 1, 2)),
    ("fwd", (15, 512, 47, 47, 136, 3, 3, 1, 1)),       # 4608 taps: 64-tap K-tiles
    ("bwd_data", (15, 136, 47, 47, 512, 3, 3, 1, 1)),
    # at most 96 output columns: the 256 x 96 wave layout
    ("fwd", (40, 48, 57, 57, 96, 3, 3, 0, 1)),   # the space-to-depth first layer's shape: 472.7 row tiles
    ("fwd", (100, 128, 27, 27, 96, 3, 3, 1, 1)),
    ("bwd_data", (30, 96, 47, 47, 128, 3, 3, 1, 1)),
    ("fwd", (30, 64, 47, 47, 96, 3, 3, 1, 1)),
    ("fwd", (30, 32, 47, 47, 90, 3, 3, 1, 1)),   # ragged columns, element-wise epilogue
    ("fwd", (30, 32, 47, 47, 40, 3, 3, 1, 1)),
    ("bwd_data", (30, 96, 47, 47, 40, 3, 3, 1, 1)),
    ("fwd", (32, 24, 64, 64, 96, 3, 3, 1, 1)),   # 512 row tiles of 256 x 96: one full round
    # 256 columns and enough row tiles: the 256 x 256 layout of 8 waves, or its
    # 192 x 256 form where that saves a round (the first two: 346 ragged tiles
    # of 192 rows in two rounds against 259 of 256 in two; the third: 216
    # tiles of 256 rows in one round)
    ("fwd", (30, 64, 47, 47, 256, 3, 3, 1, 1)),
    ("bwd_data", (30, 256, 47, 47, 64, 3, 3, 1, 1)),
    ("fwd", (25, 64, 47, 47, 250, 3, 3, 1, 1)),  # ragged columns, element-wise epilogue
    ("fwd", (256, 64, 13, 13, 256, 3, 3, 1, 1)),  # the 13 x 13 layers at batch 256: 226 tiles of 192 rows
    # stride 1 with 32-channel slices: the input-patch variant (tiles of 13 x 13
    # images span up to three images; odd and even slice counts; pad 0 and 2;
    # a non-square kernel; ragged rows and columns)
    ("fwd", (400, 64, 13, 13, 128, 3, 3, 1, 1)),
    ("bwd_data", (400, 128, 13, 13, 96, 3, 3, 1, 1)),
    ("fwd", (401, 64, 13, 13, 120, 3, 3, 1, 1)),
    ("fwd", (400, 32, 15, 15, 128, 3, 3, 0, 1)),
    ("fwd", (400, 64, 13, 13, 128, 3, 2, 1, 1)),
    ("fwd", (100, 96, 27, 27, 256, 5, 5, 2, 1)),
    ("bwd_data", (400, 256, 13, 13, 384, 3, 3, 1, 1)),
]


def _patch_fits(N, H, W, R, S, pad, cap):
    P, Q = H + 2 * pad - R + 1, W + 2 * pad - S + 1
    Hp, Wp, M = H + 2 * pad, W + 2 * pad, N * P * Q
    for m0 in range(0, M, 256):
        m1 = min(m0 + 256, M) - 1
        n0, p0 = m0 // (P * Q), (m0 % (P * Q)) // Q
        n1, p1 = m1 // (P * Q), (m1 % (P * Q)) // Q
        if (n1 * Hp + p1 + R - (n0 * Hp + p0)) * Wp > cap:
            return False
    return True


@pytest.mark.parametrize("op,case", LARGE_CASES, ids=[o + "-" + "x".join(map(str, c)) for o, c in LARGE_CASES])
def test_conv_large_tile_path(op, case):
    N, C, H, W, K, R, S, pad, stride = case
    x, w, b, dy = _conv_inputs(case, "bf16", 50)
    singa.trace_enable(True)
    if op == "fwd":
        out = singa.conv_fwd(nchw_to_dev(x, "bf16"), kcrs_to_dev(w, "bf16"), torch.from_numpy(b).cuda(), pad, stride,
                             relu=True)
    else:
        out = singa.conv_bwd_data(nchw_to_dev(dy, "bf16"), kcrs_to_dev(w, "bf16"), phys(x.shape), pad, stride)
    torch.cuda.synchronize()
    names = [r[0] for r in singa.trace_records()]
    singa.trace_enable(False)
    large = [n for n in names if n.startswith("conv_fwd_large_kernel")]
    assert large, names
    # template arguments: <bwd, taps per K-tile, wave layout[, 1 = input patch]>
    targs = [n[n.index("<") + 1:-1].split(",") for n in large]
    cols = K if op == "fwd" else C  # GEMM columns: filters, or input channels for the data gradient
    slice_c = C if op == "fwd" else K  # channels of the operand the taps gather
    narrow = cols <= 96
    assert all((t[2] == "4") == narrow for t in targs), large
    wide = 192 < cols <= 256  # 256-column tiles at least 3/4 used (every case here has enough row tiles)
    assert all((t[2] in ("6", "8")) == wide for t in targs), large
    # 192 x 256 instead of 256 x 256 when its rounds of 256 workgroups (one per CU) take at most 90 % of the time
    rows = N * (H + 2 * pad - R + 1) * (W + 2 * pad - S + 1) if op == "fwd" else N * H * W
    t256, t192 = -(-rows // 256), -(-rows // 192)
    short = wide and 10 * (-(-t192 // 256)) * 192 <= 9 * (-(-t256 // 256)) * 256
    assert all((t[2] == "6") == short for t in targs), large
    deep = not narrow and not wide and R * S * slice_c >= 4096  # reduction length
    assert all((t[1] == "64") == deep for t in targs), large
    # the input patch: stride 1, 32-channel slices, at least 4 taps, the 256 x 128 layout with 32-tap
    # K-tiles, and every 256-row tile's padded input rows x padded width within 448 entries
    patch = (stride == 1 and slice_c % 32 == 0 and R * S >= 4 and not narrow and not wide and not deep
             and _patch_fits(N, H, W, R, S, pad, 448))
    assert all((len(t) == 4 and t[3] == "1") == patch for t in targs), large
    if op == "fwd":
        ref = oracle.relu_fwd(oracle.conv_fwd(x, w, b, pad=pad, stride=stride))
    else:
        ref = oracle.conv_bwd_data(dy, w, x.shape, pad=pad, stride=stride)
    err = rel_l2(dev_to_nchw(out), ref)
    assert err <= TOL["bf16"], (case, err)


# (N, C, H, W, K, R, S, pad, stride, dtype, layout, bias): the first five take
# the fused kernel (one pass over the reduction), the rest the gradient-then-
# update path (long reduction split over the batch, fp32, NCHW, K % 8 != 0)
SGD_CASES = [
    (64, 32, 6, 6, 40, 6, 6, 0, 1, "bf16", "NHWC", True),      # fully connected, ragged taps (1152 + bias)
    (16, 256, 1, 1, 1000, 1, 1, 0, 1, "bf16", "NHWC", True),   # 1000 filters: ragged rows
    (16, 256, 1, 1, 1000, 1, 1, 0, 1, "bf16", "NHWC", False),
    (4, 16, 8, 8, 24, 3, 3, 1, 1, "bf16", "NHWC", True),       # convolution with a one-pass reduction
    (8, 64, 3, 3, 96, 3, 3, 0, 1, "bf16", "NHWC", True),
    (16, 16, 16, 16, 32, 3, 3, 1, 1, "bf16", "NHWC", True),    # split reduction
    (64, 32, 6, 6, 40, 6, 6, 0, 1, "f32", "NHWC", True),
    (64, 32, 6, 6, 40, 6, 6, 0, 1, "bf16", "NCHW", True),
    (16, 64, 1, 1, 30, 1, 1, 0, 1, "bf16", "NHWC", True),
    (32, 96, 27, 27, 256, 5, 5, 2, 1, "bf16", "NHWC", True),   # AlexNet conv2 shape, pixel-ordered split reduction
    (16, 16, 16, 16, 32, 3, 3, 1, 1, "bf16", "NHWC", False),   # split reduction without bias
    (16, 16, 16, 16, 32, 3, 3, 1, 1, "f32", "NHWC", True),     # fp32 split reduction (128 x 128 kernel)
    (4, 3, 35, 35, 8, 11, 11, 0, 4, "bf16", "NHWC", True),     # space-to-depth first layer: gradient, then update
]
# the cases whose update the split-K reduction applies
SGD_REDUCE = {5, 9, 10, 11}


def _sgd_state(K, C, R, S, layout, seed):
    w = wl.random_array((K, C, R, S), seed, "normal", 0.1, "f32")
    v = wl.random_array((K, C, R, S), seed + 1, "normal", 0.01, "f32")
    b = wl.random_array((K,), seed + 2, "normal", 0.1, "f32")
    vb = wl.random_array((K,), seed + 3, "normal", 0.01, "f32")
    return (kcrs_to_dev(w, "f32", layout), kcrs_to_dev(v, "f32", layout), to_gpu(b), to_gpu(vb))


@pytest.mark.parametrize("case", SGD_CASES, ids=["x".join(map(str, c)) for c in SGD_CASES])
def test_conv_bwd_filter_sgd_matches_gradient_then_update(case):
    """The fused call leaves w, v, the bf16 copies and the gradients bit for
    bit as singa_conv_bwd_filter followed by singa_sgd_momentum_update."""
    N, C, H, W, K, R, S, pad, stride, dt, layout, bias = case
    x, _, _, dy = _conv_inputs((N, C, H, W, K, R, S, pad, stride), dt, 120)
    xd, dyd = nchw_to_dev(x, dt, layout), nchw_to_dev(dy, dt, layout)
    wshape = fphys((K, C, R, S), layout)
    lr, mom, wd = 0.01, 0.9, 5e-4
    fused_expected = singa.conv_workspace_bytes(singa.OP_BWD_FILTER_SGD, singa.BF16 if dt == "bf16" else singa.F32,
                                                phys((N, C, H, W), layout), wshape, pad, stride, layout) == 0
    assert fused_expected == (case in SGD_CASES[:5])
    # reference: gradient, then the flat update
    w0, v0, b0, vb0 = _sgd_state(K, C, R, S, layout, 130)
    dw, db = singa.conv_bwd_filter(xd, dyd, wshape, pad, stride, layout=layout, with_bias=bias)
    wr, vr, br, vbr = to_gpu(w0), to_gpu(v0), to_gpu(b0), to_gpu(vb0)
    wbr = gpu_full(wr.shape, 0.0, torch.bfloat16)
    bbr = gpu_full(br.shape, 0.0, torch.bfloat16)
    singa.sgd_momentum_update(wr, dw, vr, wbr, lr, mom, wd)
    if bias:
        singa.sgd_momentum_update(br, db, vbr, bbr, lr, mom, wd)
    # the gradient also stored: 16-byte aligned (vector epilogue), or 4 bytes
    # off (element-wise epilogue); or not stored
    for mode in ("keep", "keep_unaligned", "none"):
        keep = mode != "none"
        wf, vf, bf, vbf = to_gpu(w0), to_gpu(v0), to_gpu(b0), to_gpu(vb0)
        wbf = gpu_full(wf.shape, 0.0, torch.bfloat16)
        bbf = gpu_full(bf.shape, 0.0, torch.bfloat16)
        gw = None
        if mode == "keep":
            gw = gpu_full(dw.shape, float("nan"))
        elif mode == "keep_unaligned":
            gw = gpu_full((dw.numel() + 1,), float("nan"))[1:].view(dw.shape)
        gb = gpu_full((K,), float("nan")) if keep and bias else None
        singa.trace_enable(True)
        singa.conv_bwd_filter_sgd(xd, dyd, wshape, wf, vf, wbf, b=bf if bias else None, vb=vbf if bias else None,
                                  b_bf16=bbf if bias else None, lr=lr, momentum=mom, weight_decay=wd, pad=pad,
                                  stride=stride, layout=layout, dw=gw, db=gb)
        torch.cuda.synchronize()
        names = [r[0] for r in singa.trace_records()]
        singa.trace_enable(False)
        assert any(n.endswith(",1>") and n.startswith("conv_wgrad_large") for n in names) == fused_expected, names
        assert ("splitk_reduce_sgd_kernel" in names) == (SGD_CASES.index(case) in SGD_REDUCE), names
        assert ("sgd_kernel" in names) == (not fused_expected and SGD_CASES.index(case) not in SGD_REDUCE), names
        assert torch.equal(wf, wr) and torch.equal(vf, vr) and torch.equal(wbf, wbr), (case, mode)
        if bias:
            assert torch.equal(bf, br) and torch.equal(vbf, vbr) and torch.equal(bbf, bbr), (case, mode)
        else:
            assert torch.equal(bf, b0) and torch.equal(vbf, vb0)  # untouched
        if keep:
            assert torch.equal(gw, dw), case
            if bias:
                assert torch.equal(gb, db), case
    # and the update itself against the oracle's, from the oracle's gradient
    ref_dw, ref_db = oracle.conv_bwd_filter(x, dy, (K, C, R, S), pad=pad, stride=stride)
    w_np, v_np = filt_to_kcrs(w0, layout), filt_to_kcrs(v0, layout)
    ref_w, ref_v = oracle.sgd_momentum(w_np, ref_dw, v_np, lr, mom, wd)
    assert rel_l2(filt_to_kcrs(wr, layout), ref_w) <= TOL["f32"]
    assert rel_l2(filt_to_kcrs(vr, layout), ref_v) <= TOL["f32"]


# local response normalization: (N, C, H, W, size); sizes 3 and 5 with C a
# multiple of the vector width take the vector kernel (NHWC), the rest the
# element-wise one
LRN_CASES = [(2, 96, 13, 13, 5), (3, 64, 7, 9, 3), (2, 16, 5, 5, 5), (2, 8, 4, 4, 5), (1, 3, 6, 6, 5),
             (2, 12, 5, 4, 4), (2, 20, 3, 3, 7), (1, 5, 2, 2, 9)]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("case", LRN_CASES, ids=_ids(LRN_CASES))
def test_lrn(case, layout, dt):
    N, C, H, W, size = case
    x = wl.random_array((N, C, H, W), 110, "normal", 4.0, dt)
    dy = wl.random_array((N, C, H, W), 111, "normal", 1.0, dt)
    args = (size, 2e-2, 0.75, 1.0)  # alpha large enough that the window matters
    y = singa.lrn_fwd(nchw_to_dev(x, dt, layout), *args, layout=layout)
    dx = singa.lrn_bwd(nchw_to_dev(x, dt, layout), nchw_to_dev(dy, dt, layout), *args, layout=layout)
    torch.cuda.synchronize()
    assert rel_l2(dev_to_nchw(y, layout), oracle.lrn_fwd(x, *args)) <= TOL[dt], case
    assert rel_l2(dev_to_nchw(dx, layout), oracle.lrn_bwd(x, dy, *args)) <= TOL[dt], case


def test_lrn_alexnet_shapes():
    # the two layers of AlexNet (after conv1 and conv2), Krizhevsky's constants in Caffe's form
    for C, H in ((96, 55), (256, 27)):
        x = np.maximum(wl.random_array((4, C, H, H), 112, "normal", 1.0, "bf16"), 0.0)
        dy = wl.random_array((4, C, H, H), 113, "normal", 1.0, "bf16")
        y = singa.lrn_fwd(nchw_to_dev(x, "bf16"), 5, 1e-4, 0.75, 1.0)
        dx = singa.lrn_bwd(nchw_to_dev(x, "bf16"), nchw_to_dev(dy, "bf16"), 5, 1e-4, 0.75, 1.0)
        torch.cuda.synchronize()
        assert rel_l2(dev_to_nchw(y), oracle.lrn_fwd(x, 5, 1e-4, 0.75, 1.0)) <= TOL["bf16"]
        assert rel_l2(dev_to_nchw(dx), oracle.lrn_bwd(x, dy, 5, 1e-4, 0.75, 1.0)) <= TOL["bf16"]


def test_lrn_errors():
    x = torch.zeros((2, 4, 4, 8), device="cuda")
    for bad in ((0, 1e-4, 0.75, 1.0), (5, -1.0, 0.75, 1.0), (5, 1e-4, 0.75, 0.0)):
        with pytest.raises(singa.SingaError) as e:
            singa.lrn_fwd(x, *bad)
        assert e.value.status == -3


# The folded ReLU backward keeps an element exactly where the mask value is
# > 0: not at +0 or -0, not at negative values or NaNs (any payload), yes at
# +inf and at positive subnormals.  The epilogue decides that from the bit
# patterns; the masks here hold every such class, and the masked output must
# equal the unmasked one zeroed where !(mask > 0), bit for bit.  Cases: the
# 256 x 96, 192 x 256 and input-patch layouts, the 128 x 128 kernel in both
# dtypes, and the dense layer through its split-K epilogue.
MASK_CASES = [("bf16", (30, 96, 47, 47, 40, 3, 3, 1, 1)), ("bf16", (30, 256, 47, 47, 64, 3, 3, 1, 1)),
              ("bf16", (400, 128, 13, 13, 96, 3, 3, 1, 1)), ("bf16", (4, 16, 8, 8, 24, 3, 3, 1, 1)),
              ("f32", (4, 16, 8, 8, 24, 3, 3, 1, 1)), ("bf16", (256, 1024, 1, 1, 4096, 1, 1, 0, 1))]


def _special_mask(shape, dt, seed):
    """Mask values of every class, as the raw bits of dt."""
    rng = np.random.default_rng(seed)
    if dt == "bf16":
        specials = np.array([0x0000, 0x8000, 0x3f80, 0xbf80, 0x7f80, 0xff80, 0x7fc0, 0x7f81, 0xffc1, 0x0001,
                             0x007f, 0x8001, 0x4120, 0x0080], np.uint16)
        bits = rng.choice(specials, size=shape).astype(np.uint16)
        vals = (bits.astype(np.uint32) << 16).view(np.float32)
        return bits, vals
    specials = np.array([0x00000000, 0x80000000, 0x3f800000, 0xbf800000, 0x7f800000, 0xff800000, 0x7fc00000,
                         0x7f800001, 0xffc00001, 0x00000001, 0x007fffff, 0x80000001, 0x41200000, 0x00800000],
                        np.uint32)
    bits = rng.choice(specials, size=shape).astype(np.uint32)
    return bits, bits.view(np.float32)


@pytest.mark.parametrize("dt,case", MASK_CASES, ids=[d + "-" + "x".join(map(str, c)) for d, c in MASK_CASES])
def test_folded_relu_backward_special_mask_values(dt, case):
    N, C, H, W, K, R, S, pad, stride = case
    _, w, _, dy = _conv_inputs(case, dt, 140)
    bits, vals = _special_mask((N, H, W, C), dt, 141)  # NHWC, the layout of the input gradient
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    ibits = bits.view(np.int16) if dt == "bf16" else bits.view(np.int32)
    mask = to_gpu(torch.from_numpy(np.ascontiguousarray(ibits))).view(tdt)
    dyd, wd = nchw_to_dev(dy, dt), kcrs_to_dev(w, dt)
    plain = singa.conv_bwd_data(dyd, wd, phys((N, C, H, W)), pad, stride)
    masked = singa.conv_bwd_data(dyd, wd, phys((N, C, H, W)), pad, stride, relu_y=mask)
    torch.cuda.synchronize()
    keep = torch.from_numpy(vals > 0).to(plain.device)
    want = torch.where(keep, plain, torch.zeros_like(plain))
    assert torch.equal(masked.view(torch.int16 if dt == "bf16" else torch.int32),
                       want.view(torch.int16 if dt == "bf16" else torch.int32)), case
