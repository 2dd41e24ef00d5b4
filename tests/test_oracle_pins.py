"""Pins for the CPU oracle: each check ties it to something other than itself.

Kinds of pin used here (CPU only, no GPU):
  * hand-worked examples stored under tests/golden/ (derivations in the files);
  * brute-force operator matrices built from an independent zero-pad-and-slice
    formulation, whose transposes must equal the backward routines;
  * the adjoint identities of a bilinear map, to fp64 rounding;
  * central finite differences;
  * library routines on special cases (torch CPU float64 conv2d, pooling,
    cross-entropy and SGD, including autograd for gradients);
  * closed forms (SGD-momentum, softmax-CE at equal logits).
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import AVG, MAX

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
torch.set_num_threads(4)


def _rng(seed):
    return np.random.default_rng(424242 + seed)


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b.ravel())
    return np.linalg.norm((a - b).ravel()) / (nb if nb > 0 else 1.0)


def _read_cases(fname):
    cases, cur = [], None
    with open(os.path.join(GOLDEN, fname)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            if key == "case":
                cur = {"name": vals[0]}
                cases.append(cur)
            elif cur is not None:
                cur[key] = [float(v) for v in vals]
            else:
                cases.append({key: [float(v) for v in vals]})
    return cases


# ----------------------------------------------------------------- sizes

def test_conv_and_pool_output_sizes():
    # AlexNet-shaped stack: 227 -> 55 (11x11 s4), pools 55 -> 27 -> 13 -> 6
    assert oracle.conv_out(227, 11, 0, 4) == 55
    assert oracle.conv_out(27, 5, 2, 1) == 27
    assert oracle.conv_out(13, 3, 1, 1) == 13
    assert [oracle.pool_out(n, 3, 0, 2, True) for n in (55, 27, 13)] == [27, 13, 6]
    # CIFAR-shaped stack: ceil mode is what makes the FC input 64*4*4 = 1024
    assert [oracle.pool_out(n, 3, 0, 2, True) for n in (32, 16, 8)] == [16, 8, 4]
    assert [oracle.pool_out(n, 3, 0, 2, False) for n in (32, 16, 8)] == [15, 7, 3]
    # padded ceil mode drops a window that would start inside the right padding
    for n in range(3, 20):
        for pad in (0, 1):
            for stride in (1, 2, 3):
                ref = torch.nn.functional.max_pool2d(torch.zeros(1, 1, n, n), 3, stride, pad,
                                                     ceil_mode=True).shape[-1]
                assert oracle.pool_out(n, 3, pad, stride, True) == ref


# ------------------------------------------------------- convolution pins

def test_conv_hand_examples():
    x = np.arange(1, 17, dtype=np.float64).reshape(1, 1, 4, 4)
    cases = [c for c in _read_cases("conv_hand_4x4.txt") if "name" in c]
    assert len(cases) == 3
    for c in cases:
        w = np.array(c["filter"]).reshape(1, 1, 3, 3)
        y = oracle.conv_fwd(x, w, None, pad=int(c["pad"][0]), stride=int(c["stride"][0]))
        np.testing.assert_array_equal(y.ravel(), np.array(c["y"]), err_msg=c["name"])


def _conv_slices(x, w, pad, stride):
    """Independent forward: zero-pad explicitly, then take window slices."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    ph, pw = pad
    sh, sw = stride
    xp = np.zeros((N, C, H + 2 * ph, W + 2 * pw))
    xp[:, :, ph:ph + H, pw:pw + W] = x
    P = (H + 2 * ph - R) // sh + 1
    Q = (W + 2 * pw - S) // sw + 1
    y = np.zeros((N, K, P, Q))
    for p in range(P):
        for q in range(Q):
            win = xp[:, :, p * sh:p * sh + R, q * sw:q * sw + S]  # N C R S
            y[:, :, p, q] = np.tensordot(win, w, axes=([1, 2, 3], [1, 2, 3]))
    return y


BRUTE_SHAPES = [
    # N, C, H, W, K, R, S, ph, pw, sh, sw
    (1, 1, 5, 5, 1, 3, 3, 0, 0, 1, 1),
    (2, 3, 7, 6, 2, 3, 3, 1, 1, 1, 1),
    (1, 2, 7, 7, 3, 5, 5, 2, 2, 1, 1),
    (2, 2, 7, 7, 2, 3, 3, 1, 1, 2, 2),
    (1, 3, 7, 7, 2, 3, 3, 0, 1, 2, 1),
    (1, 2, 7, 7, 2, 1, 1, 0, 0, 1, 1),
    (1, 1, 7, 7, 2, 3, 3, 2, 2, 4, 4),
    (2, 1, 6, 7, 1, 5, 3, 2, 1, 1, 2),
]


@pytest.mark.parametrize("shape", BRUTE_SHAPES)
def test_conv_brute_force_operator(shape):
    N, C, H, W, K, R, S, ph, pw, sh, sw = shape
    rng = _rng(sum(shape))
    x = rng.standard_normal((N, C, H, W))
    w = rng.standard_normal((K, C, R, S))
    y = oracle.conv_fwd(x, w, None, pad=(ph, pw), stride=(sh, sw))
    np.testing.assert_allclose(y, _conv_slices(x, w, (ph, pw), (sh, sw)), rtol=1e-13, atol=1e-13)
    # explicit operator matrix A (vec y = A vec x) from unit inputs of the slice formulation
    nx = x.size
    A = np.stack([_conv_slices(np.eye(nx)[i].reshape(x.shape), w, (ph, pw), (sh, sw)).ravel()
                  for i in range(nx)], axis=1)
    dy = rng.standard_normal(y.shape)
    dx = oracle.conv_bwd_data(dy, w, x.shape, pad=(ph, pw), stride=(sh, sw))
    np.testing.assert_allclose(dx.ravel(), A.T @ dy.ravel(), rtol=1e-12, atol=1e-12)
    # operator in the filter (vec y = B vec w); dw must equal B^T vec dy
    nw = w.size
    Bm = np.stack([_conv_slices(x, np.eye(nw)[j].reshape(w.shape), (ph, pw), (sh, sw)).ravel()
                   for j in range(nw)], axis=1)
    dw, db = oracle.conv_bwd_filter(x, dy, w.shape, pad=(ph, pw), stride=(sh, sw))
    np.testing.assert_allclose(dw.ravel(), Bm.T @ dy.ravel(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2, 3)), rtol=1e-13, atol=1e-13)


TORCH_SHAPES = [
    (2, 3, 32, 32, 8, 5, 5, 2, 2, 1, 1),     # CIFAR-style conv1
    (1, 3, 35, 35, 4, 11, 11, 0, 0, 4, 4),   # AlexNet conv1 geometry, shrunk
    (2, 6, 9, 9, 5, 5, 5, 2, 2, 1, 1),
    (2, 5, 13, 13, 7, 3, 3, 1, 1, 1, 1),
    (3, 4, 8, 11, 3, 3, 2, 1, 0, 2, 3),
    (2, 8, 6, 6, 6, 6, 6, 0, 0, 1, 1),       # a dense "FC as full-extent conv"
    (4, 16, 1, 1, 5, 1, 1, 0, 0, 1, 1),      # 1x1 on 1x1 (FC)
]


@pytest.mark.parametrize("shape", TORCH_SHAPES)
def test_conv_against_torch_float64(shape):
    N, C, H, W, K, R, S, ph, pw, sh, sw = shape
    rng = _rng(7 + sum(shape))
    x = rng.standard_normal((N, C, H, W))
    w = rng.standard_normal((K, C, R, S))
    b = rng.standard_normal(K)
    y = oracle.conv_fwd(x, w, b, pad=(ph, pw), stride=(sh, sw))
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    ty = F.conv2d(tx, tw, tb, stride=(sh, sw), padding=(ph, pw))
    np.testing.assert_allclose(y, ty.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal(y.shape)
    ty.backward(torch.tensor(dy))
    dx = oracle.conv_bwd_data(dy, w, x.shape, pad=(ph, pw), stride=(sh, sw))
    dw, db = oracle.conv_bwd_filter(x, dy, w.shape, pad=(ph, pw), stride=(sh, sw))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, tw.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("shape", [(2, 5, 11, 11, 4, 3, 3, 1, 1, 1, 1),
                                   (2, 3, 13, 12, 6, 5, 5, 2, 2, 2, 2),
                                   (1, 3, 27, 27, 4, 11, 11, 0, 0, 4, 4)])
def test_conv_adjoint_identities(shape):
    N, C, H, W, K, R, S, ph, pw, sh, sw = shape
    rng = _rng(99 + sum(shape))
    x = rng.standard_normal((N, C, H, W))
    w = rng.standard_normal((K, C, R, S))
    y = oracle.conv_fwd(x, w, None, pad=(ph, pw), stride=(sh, sw))
    dy = rng.standard_normal(y.shape)
    lhs = float(np.vdot(dy, y))
    dx = oracle.conv_bwd_data(dy, w, x.shape, pad=(ph, pw), stride=(sh, sw))
    dw = oracle.conv_bwd_filter(x, dy, w.shape, pad=(ph, pw), stride=(sh, sw), with_bias=False)
    assert abs(lhs - float(np.vdot(dx, x))) <= 1e-12 * max(1.0, abs(lhs)) * 10
    assert abs(lhs - float(np.vdot(dw, w))) <= 1e-12 * max(1.0, abs(lhs)) * 10


def test_conv_finite_differences():
    rng = _rng(5)
    x = rng.standard_normal((2, 3, 9, 9))
    w = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    dy = rng.standard_normal((2, 4, 5, 5))
    kw = dict(pad=1, stride=2)

    def L(xx, ww, bb):
        return float(np.vdot(dy, oracle.conv_fwd(xx, ww, bb, **kw)))

    dx = oracle.conv_bwd_data(dy, w, x.shape, **kw)
    dw, db = oracle.conv_bwd_filter(x, dy, w.shape, **kw)
    eps = 1e-6
    for idx in [(0, 0, 0, 0), (1, 2, 4, 5), (0, 1, 8, 8), (1, 0, 3, 7)]:
        e = np.zeros_like(x)
        e[idx] = eps
        fd = (L(x + e, w, b) - L(x - e, w, b)) / (2 * eps)
        assert abs(fd - dx[idx]) < 1e-6 * max(1, abs(fd))
    for idx in [(0, 0, 0, 0), (3, 2, 2, 1), (1, 1, 1, 1)]:
        e = np.zeros_like(w)
        e[idx] = eps
        fd = (L(x, w + e, b) - L(x, w - e, b)) / (2 * eps)
        assert abs(fd - dw[idx]) < 1e-6 * max(1, abs(fd))
    for k in range(4):
        e = np.zeros_like(b)
        e[k] = eps
        fd = (L(x, w, b + e) - L(x, w, b - e)) / (2 * eps)
        assert abs(fd - db[k]) < 1e-6 * max(1, abs(fd))


def test_conv_special_cases():
    rng = _rng(11)
    # 1x1, stride 1, pad 0 is a plain matrix product over channels
    x = rng.standard_normal((2, 6, 4, 5))
    w = rng.standard_normal((3, 6, 1, 1))
    y = oracle.conv_fwd(x, w, None)
    ref = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0], x)
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)
    # a centred delta filter with "same" padding copies its channel
    x = rng.standard_normal((1, 2, 6, 6))
    w = np.zeros((2, 2, 5, 5))
    w[0, 0, 2, 2] = 1.0
    w[1, 1, 2, 2] = 1.0
    np.testing.assert_array_equal(oracle.conv_fwd(x, w, None, pad=2), x)


def test_conv_points_match_full():
    rng = _rng(12)
    x = rng.standard_normal((2, 3, 11, 11))
    w = rng.standard_normal((5, 3, 3, 3))
    b = rng.standard_normal(5)
    kw = dict(pad=1, stride=2)
    y = oracle.conv_fwd(x, w, b, **kw)
    dy = rng.standard_normal(y.shape)
    dx = oracle.conv_bwd_data(dy, w, x.shape, **kw)
    dw, _ = oracle.conv_bwd_filter(x, dy, w.shape, **kw)
    for full, fn, args in [(y, oracle.conv_fwd_points, (x, w, b)),
                           (dx, oracle.conv_bwd_data_points, (dy, w, x.shape)),
                           (dw, oracle.conv_bwd_filter_points, (x, dy, w.shape))]:
        idx = rng.choice(full.size, size=min(50, full.size), replace=False)
        np.testing.assert_array_equal(fn(*args, idx, **kw), full.ravel()[idx])


def test_bwd_filter_shard_sum():
    # dim-0 (batch) partitioning (Sec. 5.3): the full-batch parameter gradient is
    # the sum of the shards' gradients
    rng = _rng(13)
    x = rng.standard_normal((6, 3, 8, 8))
    dy = rng.standard_normal((6, 4, 8, 8))
    full = oracle.conv_bwd_filter(x, dy, (4, 3, 3, 3), pad=1)
    a = oracle.conv_bwd_filter(x[:2], dy[:2], (4, 3, 3, 3), pad=1)
    b = oracle.conv_bwd_filter(x[2:], dy[2:], (4, 3, 3, 3), pad=1)
    np.testing.assert_allclose(full[0], a[0] + b[0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(full[1], a[1] + b[1], rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------- FC pins

def test_fc_against_matmul_conv_and_torch():
    rng = _rng(21)
    x = rng.standard_normal((5, 12))
    w = rng.standard_normal((7, 12))
    b = rng.standard_normal(7)
    y = oracle.fc_fwd(x, w, b)
    np.testing.assert_allclose(y, x @ w.T + b, rtol=1e-13, atol=1e-13)
    yc = oracle.conv_fwd(x.reshape(5, 12, 1, 1), w.reshape(7, 12, 1, 1), b)
    np.testing.assert_allclose(y, yc.reshape(5, 7), rtol=1e-13, atol=1e-13)
    dy = rng.standard_normal((5, 7))
    dx, dw, db = oracle.fc_bwd(x, w, dy)
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    F.linear(tx, tw, tb).backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, tw.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ pooling pins

def test_pool_hand_examples():
    g = {k: v for c in _read_cases("pool_hand_4x4.txt") for k, v in c.items()}
    x = np.arange(1, 17, dtype=np.float64).reshape(1, 1, 4, 4)
    y, am = oracle.pool_fwd(x, MAX, 3, 2, 0, True)
    np.testing.assert_array_equal(y.ravel(), g["max_y"])
    np.testing.assert_array_equal(am.ravel(), np.array(g["max_argmax"], np.uint8))
    ya, _ = oracle.pool_fwd(x, AVG, 3, 2, 0, True)
    np.testing.assert_array_equal(ya.ravel(), g["avg_y"])
    dx = oracle.pool_bwd(np.array([1, 10, 100, 1000.0]).reshape(1, 1, 2, 2), am, x.shape, MAX, 3, 2, 0, True)
    np.testing.assert_array_equal(dx.ravel(), g["max_dx"])
    dx = oracle.pool_bwd(np.array([9, 6, 6, 4.0]).reshape(1, 1, 2, 2), None, x.shape, AVG, 3, 2, 0, True)
    np.testing.assert_array_equal(dx.ravel(), g["avg_dx"])


def test_maxpool_tie_break_first_maximum():
    x = np.zeros((1, 1, 3, 3))
    _, am = oracle.pool_fwd(x, MAX, 3, 2, 0, True)
    assert am.ravel().tolist() == [0]
    x[0, 0, 0, 1] = 2.0
    x[0, 0, 1, 2] = 2.0  # equal second maximum later in the scan
    y, am = oracle.pool_fwd(x, MAX, 3, 2, 0, True)
    assert y.ravel().tolist() == [2.0] and am.ravel().tolist() == [1]
    x = -np.ones((1, 1, 3, 3))  # all-negative window: maximum -1 at cell 0
    y, am = oracle.pool_fwd(x, MAX, 3, 2, 0, True)
    assert y.ravel().tolist() == [-1.0] and am.ravel().tolist() == [0]


@pytest.mark.parametrize("geom", [(2, 3, 32, 32, 3, 2, 0), (1, 2, 16, 16, 3, 2, 0), (2, 2, 8, 8, 3, 2, 0),
                                  (1, 3, 55, 55, 3, 2, 0), (1, 2, 13, 13, 3, 2, 0), (2, 2, 9, 10, 3, 2, 1),
                                  (1, 2, 7, 7, 2, 2, 0), (1, 1, 12, 9, 3, 3, 1)])
def test_pool_against_torch_float64(geom):
    N, C, H, W, k, s, p = geom
    rng = _rng(31 + sum(geom))
    x = rng.standard_normal((N, C, H, W))  # continuous: no ties
    tx = torch.tensor(x, requires_grad=True)
    ty, tidx = F.max_pool2d(tx, k, s, p, ceil_mode=True, return_indices=True)
    y, am = oracle.pool_fwd(x, MAX, k, s, p, True)
    np.testing.assert_array_equal(y, ty.detach().numpy())
    # torch returns the flat plane index; convert ours to the same
    P, Q = y.shape[2:]
    pp, qq = np.meshgrid(np.arange(P), np.arange(Q), indexing="ij")
    hh = pp * s - p + am // k
    ww = qq * s - p + am % k
    np.testing.assert_array_equal(hh * W + ww, tidx.numpy())
    dy = rng.standard_normal(y.shape)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(oracle.pool_bwd(dy, am, x.shape, MAX, k, s, p, True), tx.grad.numpy(),
                               rtol=1e-14, atol=1e-14)
    tx.grad = None
    ta = F.avg_pool2d(tx, k, s, p, ceil_mode=True, count_include_pad=True)
    ya, _ = oracle.pool_fwd(x, AVG, k, s, p, True)
    np.testing.assert_allclose(ya, ta.detach().numpy(), rtol=1e-13, atol=1e-13)
    ta.backward(torch.tensor(dy))
    np.testing.assert_allclose(oracle.pool_bwd(dy, None, x.shape, AVG, k, s, p, True), tx.grad.numpy(),
                               rtol=1e-13, atol=1e-13)


def test_pool_adjoints_and_block_mean():
    rng = _rng(41)
    x = rng.standard_normal((2, 3, 16, 16))
    for mode in (MAX, AVG):
        y, am = oracle.pool_fwd(x, mode, 3, 2, 0, True)
        dy = rng.standard_normal(y.shape)
        dx = oracle.pool_bwd(dy, am, x.shape, mode, 3, 2, 0, True)
        assert abs(np.vdot(dy, y) - np.vdot(dx, x)) < 1e-11 * abs(np.vdot(dy, y))
    ya, _ = oracle.pool_fwd(x, AVG, 2, 2, 0, True)
    np.testing.assert_allclose(ya, x.reshape(2, 3, 8, 2, 8, 2).mean(axis=(3, 5)), rtol=1e-14)


# --------------------------------------------------------------- ReLU pins

def test_relu_definition_and_fd():
    x = np.array([-2.0, -1e-9, 0.0, 1e-9, 3.5])
    np.testing.assert_array_equal(oracle.relu_fwd(x), [0, 0, 0, 1e-9, 3.5])
    y = oracle.relu_fwd(x)
    np.testing.assert_array_equal(oracle.relu_bwd(y, np.ones(5) * 7), [0, 0, 0, 7, 7])
    rng = _rng(51)
    x = rng.standard_normal(50)
    x[np.abs(x) < 1e-3] = 0.5
    dy = rng.standard_normal(50)
    dx = oracle.relu_bwd(oracle.relu_fwd(x), dy)
    eps = 1e-7
    fd = (np.vdot(dy, oracle.relu_fwd(x + eps)) - np.vdot(dy, oracle.relu_fwd(x - eps))) / (2 * eps)
    assert abs(fd - dx.sum()) < 1e-6


# --------------------------------------------------------- softmax-CE pins

def test_softmax_ce_closed_forms_and_torch():
    for classes in (10, 1000):
        z = np.full((4, classes), 0.37)
        loss, dz = oracle.softmax_ce(z, np.arange(4) % classes)
        assert abs(loss - math.log(classes)) < 1e-13
    rng = _rng(61)
    z = rng.standard_normal((8, 10)) * 3
    lab = rng.integers(0, 10, 8)
    loss, dz = oracle.softmax_ce(z, lab)
    np.testing.assert_allclose(dz.sum(axis=1), 0, atol=1e-15)
    loss2, dz2 = oracle.softmax_ce(z + rng.standard_normal((8, 1)) * 50, lab)
    assert abs(loss - loss2) < 1e-12
    np.testing.assert_allclose(dz, dz2, atol=1e-14)
    tz = torch.tensor(z, requires_grad=True)
    tl = F.cross_entropy(tz, torch.tensor(lab, dtype=torch.long))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-13
    np.testing.assert_allclose(dz, tz.grad.numpy(), rtol=1e-12, atol=1e-15)
    # finite differences of the loss
    eps = 1e-6
    for idx in [(0, 0), (3, 7), (7, 9)]:
        e = np.zeros_like(z)
        e[idx] = eps
        fd = (oracle.softmax_ce(z + e, lab)[0] - oracle.softmax_ce(z - e, lab)[0]) / (2 * eps)
        assert abs(fd - dz[idx]) < 1e-8


# ------------------------------------------------------ bf16 storage rounding

def test_round_bf16_against_torch():
    rng = _rng(81)
    x = rng.standard_normal(200000) * np.exp(rng.uniform(-40, 40, 200000))
    x[:6] = [0.0, -0.0, 1.0, -1.5, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]  # exact and tie cases
    ref = torch.tensor(x).float().bfloat16().double().numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x), ref)
    # ties go to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert oracle.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert oracle.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6


# --------------------------------------------------------------- SGD pins

def test_sgd_momentum_closed_forms():
    rng = _rng(71)
    w0 = rng.standard_normal(100)
    g = rng.standard_normal(100)
    lr, mu, wd = 0.01, 0.9, 5e-4
    w1, v1 = oracle.sgd_momentum(w0, g, np.zeros(100), lr, mu, wd)
    np.testing.assert_allclose(w1, w0 - lr * (g + wd * w0), rtol=1e-15, atol=1e-16)
    np.testing.assert_allclose(v1, lr * (g + wd * w0), rtol=1e-15)
    # constant gradient, no decay: w_t = w0 - lr g sum_{i=1..t} (1 - mu^i)/(1 - mu)
    w, v = w0, np.zeros(100)
    for t in range(1, 8):
        w, v = oracle.sgd_momentum(w, g, v, lr, mu, 0.0)
        coef = sum((1 - mu ** i) / (1 - mu) for i in range(1, t + 1))
        np.testing.assert_allclose(w, w0 - lr * g * coef, rtol=1e-13, atol=1e-15)


def test_adagrad_closed_forms():
    """AdaGrad (Duchi et al. 2011, diagonal form): closed forms of the first
    step and of a constant gradient; the sign step at delta = 0."""
    rng = _rng(73)
    w0 = rng.standard_normal(100)
    g = rng.standard_normal(100)
    lr, delta, wd = 0.01, 1e-6, 5e-4
    w1, h1 = oracle.adagrad(w0, g, np.zeros(100), lr, delta, wd)
    g1 = g + wd * w0
    np.testing.assert_allclose(h1, g1 * g1, rtol=1e-15)
    np.testing.assert_allclose(w1, w0 - lr * g1 / (delta + np.abs(g1)), rtol=1e-14, atol=1e-16)
    w1, _ = oracle.adagrad(w0, g, np.zeros(100), lr, 0.0, 0.0)
    np.testing.assert_allclose(w1, w0 - lr * np.sign(g), rtol=1e-15, atol=1e-16)
    # constant gradient, no decay: h_t = t g^2, w_t = w0 - lr g sum_{i=1..t} 1 / (delta + sqrt(i) |g|)
    w, h = w0, np.zeros(100)
    for t in range(1, 8):
        w, h = oracle.adagrad(w, g, h, lr, delta, 0.0)
        np.testing.assert_allclose(h, t * g * g, rtol=1e-14)
        coef = sum(1.0 / (delta + np.sqrt(i) * np.abs(g)) for i in range(1, t + 1))
        np.testing.assert_allclose(w, w0 - lr * g * coef, rtol=1e-13, atol=1e-15)


def test_adagrad_against_torch_optim():
    # torch's Adagrad with no learning-rate decay and a zero initial sum:
    # sum += g'^2, w -= lr g' / (sqrt(sum) + eps), g' = g + wd w
    rng = _rng(74)
    w0 = rng.standard_normal(64)
    tw = torch.tensor(w0.copy(), requires_grad=True)
    opt = torch.optim.Adagrad([tw], lr=0.01, lr_decay=0.0, weight_decay=5e-4, initial_accumulator_value=0.0,
                              eps=1e-6)
    w, h = w0, np.zeros(64)
    for step in range(5):
        g = rng.standard_normal(64)
        tw.grad = torch.tensor(g)
        opt.step()
        w, h = oracle.adagrad(w, g, h, 0.01, 1e-6, 5e-4)
        np.testing.assert_allclose(w, tw.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_sgd_momentum_against_torch_optim():
    # torch keeps v' = mu v' + g', w -= lr v'; with a constant lr that is the
    # same trajectory as v = mu v + lr g', w -= v
    rng = _rng(72)
    w0 = rng.standard_normal(64)
    tw = torch.tensor(w0.copy(), requires_grad=True)
    opt = torch.optim.SGD([tw], lr=0.01, momentum=0.9, weight_decay=5e-4)
    w, v = w0, np.zeros(64)
    for step in range(5):
        g = rng.standard_normal(64)
        tw.grad = torch.tensor(g)
        opt.step()
        w, v = oracle.sgd_momentum(w, g, v, 0.01, 0.9, 5e-4)
        np.testing.assert_allclose(w, tw.detach().numpy(), rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------ LRN
# Local response normalization across channels (Caffe's form, the reading of
# the layer Sec. 5.4.1 names): pinned by torch's local_response_norm and its
# autograd in float64, closed forms, and finite differences.

@pytest.mark.parametrize("shape,size", [((2, 7, 3, 4), 5), ((1, 3, 2, 2), 5), ((2, 8, 2, 3), 4), ((1, 6, 1, 1), 3),
                                        ((1, 1, 3, 3), 1)])
def test_lrn_against_torch(shape, size):
    rng = _rng(80)
    x = rng.standard_normal(shape) * 3.0
    dy = rng.standard_normal(shape)
    alpha, beta, k = 0.3, 0.75, 1.5
    tx = torch.tensor(x, requires_grad=True)
    ty = torch.nn.functional.local_response_norm(tx, size, alpha=alpha, beta=beta, k=k)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(oracle.lrn_fwd(x, size, alpha, beta, k), ty.detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(oracle.lrn_bwd(x, dy, size, alpha, beta, k), tx.grad.numpy(), rtol=1e-11, atol=1e-13)


def test_lrn_closed_forms():
    rng = _rng(81)
    x = rng.standard_normal((2, 5, 3, 3))
    dy = rng.standard_normal(x.shape)
    # alpha = 0: a constant scale k^-beta
    np.testing.assert_allclose(oracle.lrn_fwd(x, 5, 0.0, 0.75, 2.0), x * 2.0 ** -0.75, rtol=1e-15)
    np.testing.assert_allclose(oracle.lrn_bwd(x, dy, 5, 0.0, 0.75, 2.0), dy * 2.0 ** -0.75, rtol=1e-15)
    # one channel in the window: y = x (k + alpha x^2)^-beta, dy/dx = s^-beta - 2 alpha beta x^2 s^(-beta-1)
    s = 1.0 + 0.5 * x * x
    np.testing.assert_allclose(oracle.lrn_fwd(x, 1, 0.5, 0.75, 1.0), x * s ** -0.75, rtol=1e-14)
    np.testing.assert_allclose(oracle.lrn_bwd(x, dy, 1, 0.5, 0.75, 1.0),
                               dy * (s ** -0.75 - 2 * 0.5 * 0.75 * x * x * s ** -1.75), rtol=1e-13)


def test_lrn_finite_differences():
    rng = _rng(82)
    x = rng.standard_normal((1, 6, 2, 2)) * 2.0
    dy = rng.standard_normal(x.shape)
    args = (5, 0.4, 0.75, 1.0)
    dx = oracle.lrn_bwd(x, dy, *args)
    eps = 1e-6
    for idx in [(0, 0, 0, 0), (0, 2, 1, 0), (0, 5, 1, 1), (0, 3, 0, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (np.sum(dy * oracle.lrn_fwd(xp, *args)) - np.sum(dy * oracle.lrn_fwd(xm, *args))) / (2 * eps)
        assert abs(fd - dx[idx]) <= 1e-7 * max(1.0, abs(fd)), (idx, fd, dx[idx])
