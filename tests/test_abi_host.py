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
    assert len(names) == 16
    lib = ctypes.CDLL(singa.lib()._name)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(singa.EXPORTS) == names


def test_status_strings():
    for code in range(-6, 1):
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
