"""ctypes binding of ``libsinga_mi.so`` (declared in include/singa_mi.h).

Argument marshalling only: every function builds the C shape/descriptor
structs from tensor shapes, allocates outputs and workspaces with torch (device
memory plumbing), and calls the C entry point of the same name on torch's
current HIP stream.  All arithmetic runs in the library's HIP kernels; there
is no fallback: if the library is missing, importing this module raises.

Tensor conventions: NHWC tensors have torch shape (N, H, W, C) and KRSC
filters (K, R, S, C); NCHW tensors (N, C, H, W) with KCRS filters (K, C, R, S).
fp32 tensors are torch.float32, bf16 tensors torch.bfloat16.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

from .build import LIB_PATH

OK = 0
ERRORS = {-1: "SINGA_ERR_NULL", -2: "SINGA_ERR_SHAPE", -3: "SINGA_ERR_UNSUPPORTED", -4: "SINGA_ERR_WORKSPACE",
          -5: "SINGA_ERR_ALIGN", -6: "SINGA_ERR_HIP", -7: "SINGA_ERR_SCRATCH"}
NOALLOC_SCRATCH_BYTES = 128 << 20
F32, BF16 = 0, 1
NCHW, NHWC, NHWC_S2D = 0, 1, 2
POOL_MAX, POOL_AVG = 0, 1
OP_FWD, OP_BWD_DATA, OP_BWD_FILTER, OP_BWD_FILTER_SGD = 0, 1, 2, 3

# every exported symbol of the C ABI (checked by the CPU tests against the header)
EXPORTS = ["singa_strerror", "singa_conv_out_shape", "singa_pool_out_shape", "singa_conv_workspace_bytes",
           "singa_conv_fwd", "singa_conv_bwd_data", "singa_conv_bwd_filter", "singa_conv_bwd_filter_noalloc",
           "singa_conv_bwd_filter_sgd",
           "singa_pool_fwd", "singa_pool_bwd",
           "singa_relu_fwd", "singa_relu_bwd", "singa_softmax_ce", "singa_sgd_momentum_update",
           "singa_adagrad_update", "singa_lrn_fwd", "singa_lrn_bwd", "singa_space_to_depth_bytes",
           "singa_space_to_depth",
           "singa_trace_enable", "singa_trace_count", "singa_trace_get"]


class LrnDesc(ctypes.Structure):
    _fields_ = [("size", ctypes.c_int), ("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("k", ctypes.c_float)]


class Shape4(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int), ("c", ctypes.c_int), ("h", ctypes.c_int), ("w", ctypes.c_int)]


class Filter4(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int), ("c", ctypes.c_int), ("r", ctypes.c_int), ("s", ctypes.c_int)]


class ConvDesc(ctypes.Structure):
    _fields_ = [("pad_h", ctypes.c_int), ("pad_w", ctypes.c_int), ("stride_h", ctypes.c_int),
                ("stride_w", ctypes.c_int)]


class PoolDesc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("kh", ctypes.c_int), ("kw", ctypes.c_int), ("stride_h", ctypes.c_int),
                ("stride_w", ctypes.c_int), ("pad_h", ctypes.c_int), ("pad_w", ctypes.c_int),
                ("ceil_mode", ctypes.c_int)]


class SingaError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__("%s failed: %s (%d): %s" % (fn, ERRORS.get(status, "?"), status,
                                                      _lib().singa_strerror(status).decode()))
        self.status = status


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("%s is not built; run `python -m paper_1603_07846_amd.build`" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
        S4, F4, CD, PD = (ctypes.POINTER(Shape4), ctypes.POINTER(Filter4), ctypes.POINTER(ConvDesc),
                          ctypes.POINTER(PoolDesc))
        lib.singa_strerror.restype = ctypes.c_char_p
        lib.singa_strerror.argtypes = [i32]
        lib.singa_conv_out_shape.argtypes = [S4, F4, CD, S4]
        lib.singa_pool_out_shape.argtypes = [S4, PD, S4]
        lib.singa_conv_workspace_bytes.argtypes = [i32, i32, i32, S4, F4, CD, ctypes.POINTER(sz)]
        lib.singa_conv_fwd.argtypes = [i32, i32, S4, vp, F4, vp, vp, CD, vp, i32, vp, sz, vp]
        lib.singa_conv_bwd_data.argtypes = [i32, i32, S4, F4, vp, CD, vp, vp, vp, vp, sz, vp]
        lib.singa_conv_bwd_filter.argtypes = [i32, i32, S4, vp, F4, CD, vp, vp, vp, i32, vp, sz, vp]
        lib.singa_conv_bwd_filter_noalloc.argtypes = [i32, i32, S4, vp, F4, CD, vp, vp, vp, i32, vp]
        f32 = ctypes.c_float
        lib.singa_conv_bwd_filter_sgd.argtypes = [i32, i32, S4, vp, F4, CD, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                  f32, f32, f32, vp, sz, vp]
        lib.singa_pool_fwd.argtypes = [i32, i32, S4, vp, PD, vp, vp, vp]
        lib.singa_pool_bwd.argtypes = [i32, i32, S4, PD, vp, vp, vp, vp, vp]
        lib.singa_relu_fwd.argtypes = [i32, sz, vp, vp, vp]
        lib.singa_relu_bwd.argtypes = [i32, sz, vp, vp, vp, vp]
        lib.singa_softmax_ce.argtypes = [i32, i32, i32, vp, vp, vp, vp, vp]
        LD = ctypes.POINTER(LrnDesc)
        lib.singa_lrn_fwd.argtypes = [i32, i32, S4, vp, LD, vp, vp]
        lib.singa_lrn_bwd.argtypes = [i32, i32, S4, vp, vp, LD, vp, vp]
        lib.singa_adagrad_update.argtypes = [sz, vp, vp, vp, vp, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                             vp]
        lib.singa_sgd_momentum_update.argtypes = [sz, vp, vp, vp, vp, ctypes.c_float, ctypes.c_float,
                                                  ctypes.c_float, vp]
        lib.singa_trace_enable.argtypes = [i32]
        lib.singa_trace_count.argtypes = []
        lib.singa_trace_get.argtypes = [i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]
        for name in EXPORTS:
            if name != "singa_strerror":
                getattr(lib, name).restype = i32
        _LIB = lib
    return _LIB


def lib():
    """The loaded ctypes library (raises ImportError if it is not built)."""
    return _lib()


def _torch_empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


_ALLOC = _torch_empty


def empty(shape, dtype, device):
    """Device memory for an output or workspace tensor.  Every output and
    workspace this module (and the step driver) allocates comes from here,
    so a test can substitute an allocator that surrounds each tensor with
    guard bands (set_allocator)."""
    return _ALLOC(tuple(int(d) for d in shape), dtype, device)


def set_allocator(fn=None):
    """Replace the tensor allocator behind empty() (fn(shape, dtype, device)
    -> a contiguous tensor of that shape); None restores torch.empty."""
    global _ALLOC
    _ALLOC = _torch_empty if fn is None else fn


def _check(fn, status):
    if status != OK:
        raise SingaError(fn, status)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("unsupported dtype %s" % t.dtype)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _pair(v) -> Tuple[int, int]:
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def _layout(layout) -> int:
    if layout in (NHWC, "NHWC"):
        return NHWC
    if layout in (NCHW, "NCHW"):
        return NCHW
    if layout in (NHWC_S2D, "NHWC_S2D"):
        return NHWC_S2D
    raise ValueError(layout)


def _act_shape4(shape, layout) -> Shape4:
    """Shape4 from a physical activation shape (NHWC_S2D: the NHWC shape of
    the input before its space-to-depth rewrite)."""
    if layout in (NHWC, NHWC_S2D):
        n, h, w, c = shape
    else:
        n, c, h, w = shape
    return Shape4(n, c, h, w)


def _filt4(shape, layout) -> Filter4:
    if layout in (NHWC, NHWC_S2D):
        k, r, s, c = shape
    else:
        k, c, r, s = shape
    return Filter4(k, c, r, s)


def _phys(s: Shape4, layout):
    return (s.n, s.h, s.w, s.c) if layout in (NHWC, NHWC_S2D) else (s.n, s.c, s.h, s.w)


def _cdesc(pad, stride) -> ConvDesc:
    ph, pw = _pair(pad)
    sh, sw = _pair(stride)
    return ConvDesc(ph, pw, sh, sw)


def conv_out_shape(x_shape, w_shape, pad=0, stride=1, layout="NHWC"):
    """Physical output shape of a convolution."""
    lay = _layout(layout)
    y = Shape4()
    _check("singa_conv_out_shape", _lib().singa_conv_out_shape(
        ctypes.byref(_act_shape4(x_shape, lay)), ctypes.byref(_filt4(w_shape, lay)),
        ctypes.byref(_cdesc(pad, stride)), ctypes.byref(y)))
    return _phys(y, lay)


def pool_out_shape(x_shape, mode, k=3, stride=2, pad=0, ceil_mode=True, layout="NHWC"):
    lay = _layout(layout)
    y = Shape4()
    _check("singa_pool_out_shape", _lib().singa_pool_out_shape(
        ctypes.byref(_act_shape4(x_shape, lay)), ctypes.byref(_pdesc(mode, k, stride, pad, ceil_mode)),
        ctypes.byref(y)))
    return _phys(y, lay)


def conv_workspace_bytes(op, dtype, x_shape, w_shape, pad=0, stride=1, layout="NHWC") -> int:
    lay = _layout(layout)
    dt = dtype if isinstance(dtype, int) else (BF16 if dtype == torch.bfloat16 else F32)
    out = ctypes.c_size_t(0)
    _check("singa_conv_workspace_bytes", _lib().singa_conv_workspace_bytes(
        op, dt, lay, ctypes.byref(_act_shape4(x_shape, lay)), ctypes.byref(_filt4(w_shape, lay)),
        ctypes.byref(_cdesc(pad, stride)), ctypes.byref(out)))
    return int(out.value)


def _workspace(nbytes, device, ws):
    if nbytes == 0:
        return None
    if ws is not None:
        return ws
    return empty((nbytes,), torch.uint8, device)


def space_to_depth_shape(x_shape, w_shape, pad=0, stride=1):
    """NHWC shape of the space-to-depth form of a convolution's NHWC input:
    (N, P + ceil(R/sh) - 1, Q + ceil(S/sw) - 1, sh sw C)."""
    n, _, _, c = x_shape
    _, r, s_, _ = w_shape
    sh, sw = _pair(stride)
    p, q = conv_out_shape(x_shape, w_shape, pad, stride)[1:3]
    return (n, p + (r + sh - 1) // sh - 1, q + (s_ + sw - 1) // sw - 1, c * sh * sw)


def space_to_depth_bytes(dtype, x_shape, w_shape, pad=0, stride=1) -> int:
    dt = dtype if isinstance(dtype, int) else (BF16 if dtype == torch.bfloat16 else F32)
    out = ctypes.c_size_t(0)
    _check("singa_space_to_depth_bytes", _lib().singa_space_to_depth_bytes(
        dt, ctypes.byref(_act_shape4(x_shape, NHWC)), ctypes.byref(_filt4(w_shape, NHWC)),
        ctypes.byref(_cdesc(pad, stride)), ctypes.byref(out)))
    return int(out.value)


def space_to_depth(x, w_shape, pad=0, stride=1, out=None):
    """The space-to-depth form of the NHWC input x of a strided convolution
    (layout "NHWC_S2D" of conv_fwd / conv_bwd_filter, with x_shape=x.shape)."""
    shape = space_to_depth_shape(tuple(x.shape), tuple(w_shape), pad, stride)
    xs = empty(shape, x.dtype, x.device) if out is None else out
    _check("singa_space_to_depth", _lib().singa_space_to_depth(
        _dt(x), ctypes.byref(_act_shape4(x.shape, NHWC)), _ptr(x), ctypes.byref(_filt4(w_shape, NHWC)),
        ctypes.byref(_cdesc(pad, stride)), _ptr(xs), _stream()))
    return xs


def conv_fwd(x, w, bias=None, pad=0, stride=1, relu=False, layout="NHWC", out=None, workspace=None, x_shape=None):
    """Convolution ComputeFeature: y = [relu](conv(x, w) + bias).  With layout
    "NHWC_S2D", x is space_to_depth()'s output and x_shape the NHWC shape of
    the input it was made from."""
    lay = _layout(layout)
    xs = tuple(x.shape) if lay != NHWC_S2D else tuple(x_shape)
    yshape = conv_out_shape(xs, tuple(w.shape), pad, stride, NHWC if lay == NHWC_S2D else lay)
    y = empty(yshape, x.dtype, x.device) if out is None else out
    nbytes = conv_workspace_bytes(OP_FWD, _dt(x), xs, tuple(w.shape), pad, stride, lay)
    ws = _workspace(nbytes, x.device, workspace)
    _check("singa_conv_fwd", _lib().singa_conv_fwd(
        _dt(x), lay, ctypes.byref(_act_shape4(xs, lay)), _ptr(x), ctypes.byref(_filt4(w.shape, lay)), _ptr(w),
        _ptr(bias), ctypes.byref(_cdesc(pad, stride)), _ptr(y), int(bool(relu)), _ptr(ws),
        0 if ws is None else ws.numel(), _stream()))
    return y


def conv_bwd_data(dy, w, x_shape, pad=0, stride=1, layout="NHWC", out=None, workspace=None, relu_y=None):
    """Convolution ComputeGradient, gradient w.r.t. the source layer's blob.

    relu_y: the output of a ReLU that is the source layer (shape x_shape); the
    result is then the gradient at that ReLU's input (its ComputeGradient
    folded into this call)."""
    lay = _layout(layout)
    dx = empty(tuple(x_shape), dy.dtype, dy.device) if out is None else out
    nbytes = conv_workspace_bytes(OP_BWD_DATA, _dt(dy), tuple(x_shape), tuple(w.shape), pad, stride, lay)
    ws = _workspace(nbytes, dy.device, workspace)
    _check("singa_conv_bwd_data", _lib().singa_conv_bwd_data(
        _dt(dy), lay, ctypes.byref(_act_shape4(x_shape, lay)), ctypes.byref(_filt4(w.shape, lay)), _ptr(w),
        ctypes.byref(_cdesc(pad, stride)), _ptr(dy), _ptr(relu_y), _ptr(dx), _ptr(ws),
        0 if ws is None else ws.numel(), _stream()))
    return dx


def conv_bwd_filter(x, dy, w_shape, pad=0, stride=1, layout="NHWC", with_bias=True, dw=None, db=None,
                    accumulate=False, workspace=None, x_shape=None):
    """Convolution ComputeGradient, Param gradients (fp32 dw and db).  With
    layout "NHWC_S2D", x is space_to_depth()'s output and x_shape the NHWC
    shape of the input it was made from."""
    lay = _layout(layout)
    xs = tuple(x.shape) if lay != NHWC_S2D else tuple(x_shape)
    if dw is None:
        dw = empty(tuple(w_shape), torch.float32, x.device)
    if with_bias and db is None:
        k = w_shape[0]
        db = empty((k,), torch.float32, x.device)
    nbytes = conv_workspace_bytes(OP_BWD_FILTER, _dt(x), xs, tuple(w_shape), pad, stride, lay)
    ws = _workspace(nbytes, x.device, workspace)
    _check("singa_conv_bwd_filter", _lib().singa_conv_bwd_filter(
        _dt(x), lay, ctypes.byref(_act_shape4(xs, lay)), _ptr(x), ctypes.byref(_filt4(w_shape, lay)),
        ctypes.byref(_cdesc(pad, stride)), _ptr(dy), _ptr(dw), _ptr(db if with_bias else None),
        int(bool(accumulate)), _ptr(ws), 0 if ws is None else ws.numel(), _stream()))
    return dw, (db if with_bias else None)


def conv_bwd_filter_noalloc(x, dy, w_shape, pad=0, stride=1, layout="NHWC", with_bias=True, dw=None, db=None,
                            accumulate=False, x_shape=None):
    """conv_bwd_filter with the library's fixed scratch array instead of a
    workspace (dw / db, when not given, are still allocated here; a caller
    that must not allocate passes them)."""
    lay = _layout(layout)
    xs = tuple(x.shape) if lay != NHWC_S2D else tuple(x_shape)
    if dw is None:
        dw = empty(tuple(w_shape), torch.float32, x.device)
    if with_bias and db is None:
        db = empty((w_shape[0],), torch.float32, x.device)
    _check("singa_conv_bwd_filter_noalloc", _lib().singa_conv_bwd_filter_noalloc(
        _dt(x), lay, ctypes.byref(_act_shape4(xs, lay)), _ptr(x), ctypes.byref(_filt4(w_shape, lay)),
        ctypes.byref(_cdesc(pad, stride)), _ptr(dy), _ptr(dw), _ptr(db if with_bias else None),
        int(bool(accumulate)), _stream()))
    return dw, (db if with_bias else None)


def conv_bwd_filter_sgd(x, dy, w_shape, w, v, w_bf16=None, b=None, vb=None, b_bf16=None, lr=0.01, momentum=0.9,
                        weight_decay=0.0, pad=0, stride=1, layout="NHWC", dw=None, db=None, workspace=None):
    """Param gradients of a convolution with the momentum SGD step applied to
    them at once: w, v (fp32, filter shape) and w_bf16 updated in place, the
    bias likewise when b is given; dw / db, if given, also receive the
    gradient.  Returns (w, v)."""
    lay = _layout(layout)
    nbytes = conv_workspace_bytes(OP_BWD_FILTER_SGD, _dt(x), tuple(x.shape), tuple(w_shape), pad, stride, lay)
    ws = _workspace(nbytes, x.device, workspace)
    _check("singa_conv_bwd_filter_sgd", _lib().singa_conv_bwd_filter_sgd(
        _dt(x), lay, ctypes.byref(_act_shape4(x.shape, lay)), _ptr(x), ctypes.byref(_filt4(w_shape, lay)),
        ctypes.byref(_cdesc(pad, stride)), _ptr(dy), _ptr(dw), _ptr(db), _ptr(w), _ptr(v), _ptr(w_bf16), _ptr(b),
        _ptr(vb), _ptr(b_bf16), float(lr), float(momentum), float(weight_decay), _ptr(ws),
        0 if ws is None else ws.numel(), _stream()))
    return w, v


def _pdesc(mode, k, stride, pad, ceil_mode) -> PoolDesc:
    kh, kw = _pair(k)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    m = POOL_MAX if mode in (POOL_MAX, "max") else POOL_AVG
    return PoolDesc(m, kh, kw, sh, sw, ph, pw, int(bool(ceil_mode)))


def pool_fwd(x, mode, k=3, stride=2, pad=0, ceil_mode=True, layout="NHWC", out=None, argmax=None):
    """Pooling ComputeFeature; returns (y, argmax) (argmax is None for AVG)."""
    lay = _layout(layout)
    d = _pdesc(mode, k, stride, pad, ceil_mode)
    yshape = pool_out_shape(tuple(x.shape), mode, k, stride, pad, ceil_mode, lay)
    y = empty(yshape, x.dtype, x.device) if out is None else out
    if d.mode == POOL_MAX and argmax is None:
        argmax = empty(yshape, torch.uint8, x.device)
    _check("singa_pool_fwd", _lib().singa_pool_fwd(
        _dt(x), lay, ctypes.byref(_act_shape4(x.shape, lay)), _ptr(x), ctypes.byref(d), _ptr(y),
        _ptr(argmax if d.mode == POOL_MAX else None), _stream()))
    return y, (argmax if d.mode == POOL_MAX else None)


def pool_bwd(dy, argmax, x_shape, mode, k=3, stride=2, pad=0, ceil_mode=True, layout="NHWC", out=None, relu_y=None):
    """Pooling ComputeGradient.  relu_y (max pooling): the pooling's own output,
    when its input is a ReLU's output; the result is then the gradient at that
    ReLU's input."""
    lay = _layout(layout)
    d = _pdesc(mode, k, stride, pad, ceil_mode)
    dx = empty(tuple(x_shape), dy.dtype, dy.device) if out is None else out
    _check("singa_pool_bwd", _lib().singa_pool_bwd(
        _dt(dy), lay, ctypes.byref(_act_shape4(x_shape, lay)), ctypes.byref(d), _ptr(dy),
        _ptr(argmax if d.mode == POOL_MAX else None), _ptr(relu_y), _ptr(dx), _stream()))
    return dx


def relu_fwd(x, out=None):
    y = empty(x.shape, x.dtype, x.device) if out is None else out
    _check("singa_relu_fwd", _lib().singa_relu_fwd(_dt(x), x.numel(), _ptr(x), _ptr(y), _stream()))
    return y


def relu_bwd(y, dy, out=None):
    dx = empty(dy.shape, dy.dtype, dy.device) if out is None else out
    _check("singa_relu_bwd", _lib().singa_relu_bwd(_dt(y), y.numel(), _ptr(y), _ptr(dy), _ptr(dx), _stream()))
    return dx


def softmax_ce(z, labels, loss=None, dz=None):
    """Softmax cross-entropy over rows of z (batch, classes); returns (loss, dz) where
    loss is an fp32 tensor of batch + 1 values: the mean, then each row's loss."""
    B, classes = z.shape[0], z[0].numel()
    loss = empty((B + 1,), torch.float32, z.device) if loss is None else loss
    dz = empty(z.shape, z.dtype, z.device) if dz is None else dz
    _check("singa_softmax_ce", _lib().singa_softmax_ce(_dt(z), B, classes, _ptr(z), _ptr(labels), _ptr(loss),
                                                       _ptr(dz), _stream()))
    return loss, dz


def sgd_momentum_update(w, g, v, w_bf16=None, lr=0.01, momentum=0.9, weight_decay=0.0):
    """Fused Updater step in place on fp32 w and v (and the bf16 shadow if given)."""
    _check("singa_sgd_momentum_update", _lib().singa_sgd_momentum_update(
        w.numel(), _ptr(w), _ptr(g), _ptr(v), _ptr(w_bf16), float(lr), float(momentum), float(weight_decay),
        _stream()))
    return w, v


def lrn_fwd(x, size=5, alpha=1e-4, beta=0.75, k=1.0, layout="NHWC", out=None):
    """Local response normalization across channels (Caffe's form)."""
    lay = _layout(layout)
    y = empty(x.shape, x.dtype, x.device) if out is None else out
    _check("singa_lrn_fwd", _lib().singa_lrn_fwd(
        _dt(x), lay, ctypes.byref(_act_shape4(x.shape, lay)), _ptr(x),
        ctypes.byref(LrnDesc(int(size), float(alpha), float(beta), float(k))), _ptr(y), _stream()))
    return y


def lrn_bwd(x, dy, size=5, alpha=1e-4, beta=0.75, k=1.0, layout="NHWC", out=None):
    """Gradient of sum(dy * lrn_fwd(x)) with respect to x."""
    lay = _layout(layout)
    dx = empty(x.shape, x.dtype, x.device) if out is None else out
    _check("singa_lrn_bwd", _lib().singa_lrn_bwd(
        _dt(x), lay, ctypes.byref(_act_shape4(x.shape, lay)), _ptr(x), _ptr(dy),
        ctypes.byref(LrnDesc(int(size), float(alpha), float(beta), float(k))), _ptr(dx), _stream()))
    return dx


def adagrad_update(w, g, h, w_bf16=None, lr=0.01, delta=1e-6, weight_decay=0.0):
    """AdaGrad Updater step in place on fp32 w and h (and the bf16 shadow if given)."""
    _check("singa_adagrad_update", _lib().singa_adagrad_update(
        w.numel(), _ptr(w), _ptr(g), _ptr(h), _ptr(w_bf16), float(lr), float(delta), float(weight_decay),
        _stream()))
    return w, h


def trace_enable(on: bool = True):
    """Start (clearing) or stop the library's per-kernel timing trace."""
    _lib().singa_trace_enable(int(bool(on)))


def trace_records():
    """[(kernel name, ms, work, unit)] of the recorded launches; synchronize first."""
    out = []
    name, ms, work, unit = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_double(), ctypes.c_int()
    for i in range(_lib().singa_trace_count()):
        rc = _lib().singa_trace_get(i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(work), ctypes.byref(unit))
        if rc != 0:
            raise RuntimeError("singa_trace_get(%d) failed: %d" % (i, rc))
        out.append((name.value.decode(), ms.value, work.value, "flop" if unit.value == 0 else "byte"))
    return out


# Import-time load: the product path fails loudly when the HIP library is missing.
_lib()
