"""singa_conv_bwd_filter_noalloc (the filter gradient with the library's
fixed scratch array) against singa_conv_bwd_filter (caller workspace) on the
same inputs: two calls in a row on one GPU, the second with a smaller input
(and another kernel path) than the first, each bit for bit equal to the
allocating call, whose results the other GPU tests hold to the oracle.  A
call whose workspace would exceed the array is rejected before any launch."""
import numpy as np
import pytest
import torch

from _helpers import gpu_full, to_gpu
from paper_1603_07846_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (N, C, H, W, K, R, S, pad, stride, dtype): an AlexNet conv2-shaped layer
# (split-K partial tiles in the scratch array), then a smaller strided first
# layer (space-to-depth input and fp32 gradient staging in it as well)
CALLS = [(32, 96, 27, 27, 256, 5, 5, 2, 1, "bf16"), (4, 3, 227, 227, 96, 11, 11, 0, 4, "bf16")]


def _inputs(N, C, H, W, K, R, S, pad, stride, dt, seed):
    P, Q = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    x = wl.random_array((N, H, W, C), seed, "normal", 1.0, dt)
    dy = wl.random_array((N, P, Q, K), seed + 1, "normal", 1.0, dt)
    return to_gpu(x, tdt), to_gpu(dy, tdt)


def test_noalloc_matches_workspace_call_twice():
    from paper_1603_07846_amd import singa
    for i, (N, C, H, W, K, R, S, pad, stride, dt) in enumerate(CALLS):
        xd, dyd = _inputs(N, C, H, W, K, R, S, pad, stride, dt, 40 + 5 * i)
        need = singa.conv_workspace_bytes(singa.OP_BWD_FILTER, singa.BF16 if dt == "bf16" else singa.F32,
                                          (N, H, W, C), (K, R, S, C), pad, stride)
        assert 0 < need <= singa.NOALLOC_SCRATCH_BYTES
        ref_dw, ref_db = singa.conv_bwd_filter(xd, dyd, (K, R, S, C), pad, stride)
        dw = gpu_full((K, R, S, C), float("nan"))
        db = gpu_full((K,), float("nan"))
        singa.conv_bwd_filter_noalloc(xd, dyd, (K, R, S, C), pad, stride, dw=dw, db=db)
        torch.cuda.synchronize()
        assert torch.equal(dw, ref_dw), ("call", i)
        assert torch.equal(db, ref_db), ("call", i)
        assert np.isfinite(dw.cpu().numpy()).all()


def test_noalloc_rejects_more_than_the_scratch_array():
    from paper_1603_07846_amd import singa
    # an NCHW call at AlexNet's full first layer stages its input and output
    # gradient in the workspace: more than the array holds
    N, C, H, W, K, R, S = 256, 3, 227, 227, 96, 11, 11
    need = singa.conv_workspace_bytes(singa.OP_BWD_FILTER, singa.BF16, (N, C, H, W), (K, C, R, S), 0, 4, "NCHW")
    assert need > singa.NOALLOC_SCRATCH_BYTES
    x = gpu_full((N, C, H, W), 0.0, torch.bfloat16)
    dy = gpu_full((N, K, 55, 55), 0.0, torch.bfloat16)
    dw = gpu_full((K, C, R, S), 7.0)
    with pytest.raises(singa.SingaError) as e:
        singa.conv_bwd_filter_noalloc(x, dy, (K, C, R, S), 0, 4, layout="NCHW", dw=dw, with_bias=False)
    assert e.value.status == -7
    torch.cuda.synchronize()
    assert bool((dw == 7.0).all())  # nothing was launched
