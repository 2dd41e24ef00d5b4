"""Shared test helpers: layout marshalling and error metrics (no method arithmetic)."""
import numpy as np
import torch

# rel-L2 tolerances, fp32 and bf16 (fp32 accumulation)
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_l2(got, ref) -> float:
    """||got - ref||_2 / ||ref||_2 in fp64 (||got||_2 itself if ref is all zero)."""
    g = np.asarray(got, np.float64).ravel()
    r = np.asarray(ref, np.float64).ravel()
    assert g.shape == r.shape, (g.shape, r.shape)
    nr = np.linalg.norm(r)
    if nr == 0.0:
        return float(np.linalg.norm(g))
    return float(np.linalg.norm(g - r) / nr)


def torch_dtype(dt: str):
    return torch.bfloat16 if dt == "bf16" else torch.float32


def to_gpu(t, dtype=None):
    """A device copy of host tensor / array t (optionally converted to dtype),
    allocated through the binding's allocator: inside a GPU test it carries
    guard bands that are checked when the test ends."""
    from paper_1603_07846_amd import singa
    if not isinstance(t, torch.Tensor):
        t = torch.from_numpy(np.ascontiguousarray(t))
    t = t.contiguous()
    dtype = t.dtype if dtype is None else dtype
    out = singa.empty(tuple(t.shape), dtype, "cuda")
    out.copy_(t.to(dtype))
    return out


def gpu_full(shape, value, dtype=torch.float32):
    """A device tensor filled with value, through the binding's allocator."""
    from paper_1603_07846_amd import singa
    return singa.empty(tuple(shape), dtype, "cuda").fill_(value)


def nchw_to_dev(a, dt="f32", layout="NHWC"):
    """numpy NCHW (values already representable in dt) -> device tensor in layout."""
    a = np.asarray(a, np.float32)
    if layout == "NHWC" and a.ndim == 4:
        a = a.transpose(0, 2, 3, 1)
    return to_gpu(a, torch_dtype(dt))


def kcrs_to_dev(w, dt="f32", layout="NHWC"):
    w = np.asarray(w, np.float32)
    if layout == "NHWC":
        w = w.transpose(0, 2, 3, 1)
    return to_gpu(w, torch_dtype(dt))


def dev_to_nchw(t, layout="NHWC"):
    a = t.detach().float().cpu().numpy().astype(np.float64)
    if layout == "NHWC" and a.ndim == 4:
        a = a.transpose(0, 3, 1, 2)
    return np.ascontiguousarray(a)


def filt_to_kcrs(t, layout="NHWC"):
    a = t.detach().float().cpu().numpy().astype(np.float64)
    if layout == "NHWC":
        a = a.transpose(0, 3, 1, 2)
    return np.ascontiguousarray(a)


def phys(shape_nchw, layout="NHWC"):
    n, c, h, w = shape_nchw
    return (n, h, w, c) if layout == "NHWC" else (n, c, h, w)


def fphys(shape_kcrs, layout="NHWC"):
    k, c, r, s = shape_kcrs
    return (k, r, s, c) if layout == "NHWC" else (k, c, r, s)
