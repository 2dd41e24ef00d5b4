"""Host-side checks of the C ABI (no GPU needed, no compute call made).

* the built library loads and exports every function include/singa_mi.h declares;
* the host-only helpers (output shapes, workspace sizes, status strings)
  agree with the oracle's shape arithmetic and reject bad arguments.
"""
import ctypes
import os
import re

import pytest

import oracle
from paper_1603_07846_amd import singa

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "singa_mi.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(singa_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) == 23
    lib = ctypes.CDLL(singa.lib()._name)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(singa.EXPORTS) == names


def test_status_strings():
    for code in range(-7, 1):
        assert singa.lib().singa_strerror(code)
    assert singa.lib().singa_strerror(-4) == b"workspace too small"


@pytest.mark.parametrize("geom", [(227, 11, 0, 4), (27, 5, 2, 1), (13, 3, 1, 1), (32, 5, 2, 1), (7, 7, 0, 1),
                                  (9, 2, 0, 3), (10, 3, 2, 2)])
def test_conv_out_shape_matches_oracle(geom):
    n, k, p, s = geom
    y = singa.conv_out_shape((3, n, n + 1, 5), (4, k, k, 5), p, s)
    assert y == (3, oracle.conv_out(n, k, p, s), oracle.conv_out(n + 1, k, p, s), 4)
    y2 = singa.conv_out_shape((3, 5, n, n + 1), (4, 5, k, k), p, s, layout="NCHW")
    assert y2 == (3, 4, y[1], y[2])


@pytest.mark.parametrize("n", list(range(3, 40)))
def test_pool_out_shape_matches_oracle(n):
    for pad in (0, 1):
        for stride in (1, 2, 3):
            for ceil in (True, False):
                y = singa.pool_out_shape((1, n, n, 2), "max", 3, stride, pad, ceil)
                assert y[1] == oracle.pool_out(n, 3, pad, stride, ceil)


def test_shape_errors():
    with pytest.raises(singa.SingaError) as e:
        singa.conv_out_shape((1, 8, 8, 3), (4, 3, 3, 5))  # channel mismatch
    assert e.value.status == -2
    with pytest.raises(singa.SingaError) as e:
        singa.conv_out_shape((1, 2, 2, 3), (4, 5, 5, 3))  # output would be empty
    assert e.value.status == -2
    with pytest.raises(singa.SingaError) as e:
        singa.conv_out_shape((0, 8, 8, 3), (4, 3, 3, 3))
    assert e.value.status == -2
    with pytest.raises(singa.SingaError) as e:
        singa.pool_out_shape((1, 40, 40, 3), "max", 17, 1)  # 289 cells do not fit a uint8 argmax
    assert e.value.status == -3
    with pytest.raises(singa.SingaError) as e:
        singa.pool_out_shape((1, 8, 8, 3), "max", 3, 2, 3)  # pad >= window
    assert e.value.status == -3
    with pytest.raises(singa.SingaError) as e:
        singa.conv_out_shape((1 << 16, 256, 256, 64), (4, 3, 3, 64), 1, 1)  # 32-bit index limit
    assert e.value.status == -3


def test_workspace_sizes():
    x, w = (256, 27, 27, 96), (256, 5, 5, 96)
    assert singa.conv_workspace_bytes(singa.OP_FWD, singa.BF16, x, w, 2, 1) == 0
    # stride 1 backward-data keeps one flipped filter copy
    assert singa.conv_workspace_bytes(singa.OP_BWD_DATA, singa.BF16, x, w, 2, 1) >= 256 * 25 * 96 * 2
    # strided backward-data: the space-to-depth filter, its flipped transpose and the rewritten input gradient
    # (11x11/4 on 3 channels -> 3x3/1 on 48 channels, 9x9 rewritten input)
    assert singa.conv_workspace_bytes(singa.OP_BWD_DATA, singa.F32, (2, 35, 35, 3), (8, 11, 11, 3), 0, 4) >= \
        2 * (8 * 3 * 3 * 48 * 4) + 2 * 9 * 9 * 48 * 4
    assert singa.conv_workspace_bytes(singa.OP_BWD_FILTER, singa.F32, x, w, 2, 1) >= 256 * 25 * 96 * 4
    nchw = singa.conv_workspace_bytes(singa.OP_FWD, singa.F32, (2, 96, 27, 27), (256, 96, 5, 5), 2, 1,
                                      layout="NCHW")
    assert nchw >= 4 * (2 * 96 * 27 * 27 + 256 * 96 * 25 + 2 * 256 * 27 * 27)
    with pytest.raises(singa.SingaError) as e:
        singa.conv_workspace_bytes(7, singa.F32, x, w, 2, 1)
    assert e.value.status == -3


def test_bwd_filter_sgd_workspace_says_when_the_update_is_fused():
    """0 bytes exactly for the fused case: bf16, NHWC, K and C multiples of 8,
    no input rewrite, one pass over the reduction (fully connected layers at
    batch 256); otherwise staging for the gradient plus the gradient's own."""
    op = singa.OP_BWD_FILTER_SGD
    fc6, w6 = (256, 6, 6, 256), (4096, 6, 6, 256)
    assert singa.conv_workspace_bytes(op, singa.BF16, fc6, w6, 0, 1) == 0
    assert singa.conv_workspace_bytes(op, singa.BF16, (256, 1, 1, 4096), (1000, 1, 1, 4096), 0, 1) == 0
    g6 = 4096 * 6 * 6 * 256 * 4 + 4096 * 4
    assert singa.conv_workspace_bytes(op, singa.F32, fc6, w6, 0, 1) >= g6          # fp32: no fused kernel
    assert singa.conv_workspace_bytes(op, singa.BF16, (256, 256, 6, 6), (4096, 256, 6, 6), 0, 1,
                                      layout="NCHW") >= g6                                # NCHW
    # a convolution with a long reduction (split over the batch) is not fused
    conv2 = singa.conv_workspace_bytes(op, singa.BF16, (256, 27, 27, 96), (256, 5, 5, 96), 2, 1)
    assert conv2 >= 256 * 25 * 96 * 4 + singa.conv_workspace_bytes(singa.OP_BWD_FILTER, singa.BF16,
                                                                    (256, 27, 27, 96), (256, 5, 5, 96), 2, 1)
    # K or C not a multiple of 8
    assert singa.conv_workspace_bytes(op, singa.BF16, (8, 1, 1, 256), (1001, 1, 1, 256), 0, 1) > 0
    assert singa.conv_workspace_bytes(op, singa.BF16, (8, 1, 1, 250), (1000, 1, 1, 250), 0, 1) > 0


def test_bwd_filter_sgd_argument_errors():
    """Validation before anything is enqueued (fake, never dereferenced device addresses)."""
    lib = singa.lib()
    x = singa._act_shape4((4, 1, 1, 64), singa.NHWC)
    w = singa._filt4((16, 1, 1, 64), singa.NHWC)
    d = singa._cdesc(0, 1)
    A = ctypes.c_void_p(1 << 20)  # 16-byte aligned stand-in pointers
    B = ctypes.c_void_p((1 << 20) + 4)
    N = None

    def call(*ptrs, dt=singa.BF16):
        xp, dyp, wm, vm, wb, bm, vb, bb = ptrs
        return lib.singa_conv_bwd_filter_sgd(dt, singa.NHWC, ctypes.byref(x), xp, ctypes.byref(w), ctypes.byref(d),
                                             dyp, N, N, wm, vm, wb, bm, vb, bb, 0.01, 0.9, 0.0005, N, 0, N)
    assert call(A, A, N, A, N, N, N, N) == -1       # no master weights
    assert call(A, A, A, N, N, N, N, N) == -1       # no momentum
    assert call(A, A, A, A, N, A, N, N) == -1       # bias without its momentum
    assert call(A, A, A, A, N, N, N, A) == -1       # bias shadow without the bias
    assert call(A, A, B, A, N, N, N, N) == -5       # update arrays need 16 bytes
    assert call(A, A, A, A, B, N, N, N) == -5
    assert call(B, A, A, A, N, N, N, N) == -5       # fused case: x needs 16 bytes
    assert call(A, A, A, A, N, N, N, N, dt=singa.F32) == -4  # unfused: staging workspace required


def test_space_to_depth_layout_sizes_and_errors():
    """The space-to-depth input form exists exactly for the convolutions the
    library rewrites that way (strided, channels too few for vector loads,
    rewritten channels enough); its size is N (P + ceil(R/s) - 1)
    (Q + ceil(S/s) - 1) s^2 C elements; workspaces shrink by the rewritten
    input the call no longer builds; other entry points reject the layout."""
    conv1x, conv1w = (256, 227, 227, 3), (96, 11, 11, 3)
    nbytes = singa.space_to_depth_bytes(singa.BF16, conv1x, conv1w, 0, 4)
    assert nbytes == 256 * 57 * 57 * 48 * 2
    assert singa.space_to_depth_shape(conv1x, conv1w, 0, 4) == (256, 57, 57, 48)
    assert singa.space_to_depth_bytes(singa.BF16, (2, 33, 33, 3), (8, 7, 7, 3), 3, 4) == 2 * 10 * 10 * 48 * 2
    # no rewrite: stride 1, or vector-friendly channels
    assert singa.space_to_depth_bytes(singa.BF16, (256, 27, 27, 96), (256, 5, 5, 96), 2, 1) == 0
    assert singa.space_to_depth_bytes(singa.BF16, (2, 35, 35, 16), (8, 11, 11, 16), 0, 4) == 0
    for op in (singa.OP_FWD, singa.OP_BWD_FILTER):
        nhwc = singa.conv_workspace_bytes(op, singa.BF16, conv1x, conv1w, 0, 4)
        s2d = singa.conv_workspace_bytes(op, singa.BF16, conv1x, conv1w, 0, 4, layout="NHWC_S2D")
        assert nhwc - s2d == nbytes
    for op in (singa.OP_BWD_DATA, singa.OP_BWD_FILTER_SGD):
        with pytest.raises(singa.SingaError) as e:
            singa.conv_workspace_bytes(op, singa.BF16, conv1x, conv1w, 0, 4, layout="NHWC_S2D")
        assert e.value.status == -3
    with pytest.raises(singa.SingaError) as e:  # a convolution that is not rewritten
        singa.conv_workspace_bytes(singa.OP_FWD, singa.BF16, (256, 27, 27, 96), (256, 5, 5, 96), 2, 1,
                                   layout="NHWC_S2D")
    assert e.value.status == -3
    lib = singa.lib()
    x, w, d = singa._act_shape4(conv1x, singa.NHWC), singa._filt4(conv1w, singa.NHWC), singa._cdesc(0, 4)
    A, B = ctypes.c_void_p(1 << 20), ctypes.c_void_p((1 << 20) + 4)
    assert lib.singa_space_to_depth(singa.BF16, ctypes.byref(x), A, ctypes.byref(w), ctypes.byref(d), None,
                                    None) == -1
    assert lib.singa_space_to_depth(singa.BF16, ctypes.byref(x), A, ctypes.byref(w), ctypes.byref(d), B,
                                    None) == -5
    d1 = singa._cdesc(2, 1)
    x2, w2 = singa._act_shape4((256, 27, 27, 96), singa.NHWC), singa._filt4((256, 5, 5, 96), singa.NHWC)
    assert lib.singa_space_to_depth(singa.BF16, ctypes.byref(x2), A, ctypes.byref(w2), ctypes.byref(d1), A,
                                    None) == -3
    # pooling and LRN do not take the layout
    pd = singa._pdesc("max", 3, 2, 0, True)
    assert lib.singa_pool_fwd(singa.BF16, singa.NHWC_S2D, ctypes.byref(x), A, ctypes.byref(pd), A, A, None) == -3


def test_empty_and_degenerate_sizes_answered_before_any_launch():
    """n = 0 element-wise calls and updates succeed without touching a
    pointer (here NULL) or the GPU; an empty batch or class count, and every
    NULL pointer of a non-empty call, are rejected before any launch."""
    lib = singa.lib()
    null = ctypes.c_void_p(0)
    for dt in (singa.F32, singa.BF16):
        assert lib.singa_relu_fwd(dt, ctypes.c_size_t(0), null, null, null) == 0
        assert lib.singa_relu_bwd(dt, ctypes.c_size_t(0), null, null, null, null) == 0
        assert lib.singa_relu_fwd(dt, ctypes.c_size_t(8), null, null, null) == -1
        for batch, classes in ((0, 10), (4, 0), (-1, 10)):
            assert lib.singa_softmax_ce(dt, batch, classes, null, null, null, null, null) == -2
        assert lib.singa_softmax_ce(dt, 4, 10, null, null, null, null, null) == -1
    f = ctypes.c_float
    assert lib.singa_sgd_momentum_update(ctypes.c_size_t(0), null, null, null, null, f(0.01), f(0.9), f(5e-4),
                                         null) == 0
    assert lib.singa_sgd_momentum_update(ctypes.c_size_t(8), null, null, null, null, f(0.01), f(0.9), f(5e-4),
                                         null) == -1
    assert lib.singa_adagrad_update(ctypes.c_size_t(0), null, null, null, null, f(0.01), f(1e-6), f(5e-4),
                                    null) == 0
    assert lib.singa_adagrad_update(ctypes.c_size_t(8), null, null, null, null, f(0.01), f(1e-6), f(5e-4),
                                    null) == -1
