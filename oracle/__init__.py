"""CPU oracle for the SINGA conv-training hot path (arXiv 1603.07846).

TEST INFRASTRUCTURE ONLY.  This package is the plain fp64 definition that the
GPU library is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does, and
it imports nothing from the product package.

The arithmetic lives in ``singa_oracle.c`` (plain C, fp64, OpenMP over output
elements).  This module only marshals numpy arrays into it.  Layouts are NCHW
for activations and KCRS for filters, as in Caffe's convolution and pooling
code that SINGA adopts (Sec. 6.2.1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "singa_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

_i64 = ctypes.c_int64
_dp = ctypes.POINTER(ctypes.c_double)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


# A checking build (sanitize=True: AddressSanitizer and UndefinedBehavior-
# Sanitizer, every report fatal) loads only in a process that preloads the
# ASan runtime; SINGA_ORACLE_LIB names the library to load instead of the
# default build.
SANITIZE_FLAGS = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                  "-fno-omit-frame-pointer"]


def build(path: str = None, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (always recompiles).  Returns the .so path."""
    path = _LIB_PATH if path is None else path
    tmp = path + ".tmp%d" % os.getpid()
    opt = SANITIZE_FLAGS if sanitize else ["-O2"]
    cmd = (["gcc"] + opt + ["-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC,
                            "-lm"])
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)
    return path


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        path = os.environ.get("SINGA_ORACLE_LIB") or _LIB_PATH
        if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(path)
        geo = [_i64] * 11
        lib.oracle_conv_out.argtypes = [_i64] * 4
        lib.oracle_conv_out.restype = _i64
        lib.oracle_pool_out.argtypes = [_i64] * 4 + [ctypes.c_int]
        lib.oracle_pool_out.restype = _i64
        lib.oracle_conv_fwd.argtypes = geo + [_dp, _dp, _dp, _dp]
        lib.oracle_conv_bwd_data.argtypes = geo + [_dp, _dp, _dp]
        lib.oracle_conv_bwd_filter.argtypes = geo + [_dp, _dp, _dp, _dp]
        lib.oracle_conv_fwd_points.argtypes = geo + [_dp, _dp, _dp, _i64, _i64p, _dp]
        lib.oracle_conv_bwd_data_points.argtypes = geo + [_dp, _dp, _i64, _i64p, _dp]
        lib.oracle_conv_bwd_filter_points.argtypes = geo + [_dp, _dp, _i64, _i64p, _dp]
        lib.oracle_fc_fwd.argtypes = [_i64] * 3 + [_dp, _dp, _dp, _dp]
        lib.oracle_fc_bwd.argtypes = [_i64] * 3 + [_dp, _dp, _dp, _dp, _dp, _dp]
        pool = [ctypes.c_int] + [_i64] * 10 + [ctypes.c_int]
        lib.oracle_pool_fwd.argtypes = pool + [_dp, _dp, _u8p]
        lib.oracle_pool_bwd.argtypes = pool + [_dp, _u8p, _dp]
        lib.oracle_relu_fwd.argtypes = [_i64, _dp, _dp]
        lib.oracle_relu_bwd.argtypes = [_i64, _dp, _dp, _dp]
        _d = ctypes.c_double
        lib.oracle_lrn_fwd.argtypes = [_i64, _i64, _i64, _i64, _dp, _i64, _d, _d, _d, _dp]
        lib.oracle_lrn_bwd.argtypes = [_i64, _i64, _i64, _i64, _dp, _dp, _i64, _d, _d, _d, _dp]
        lib.oracle_softmax_ce.argtypes = [_i64, _i64, _dp, _i32p, _dp]
        lib.oracle_softmax_ce.restype = ctypes.c_double
        lib.oracle_round_bf16.argtypes = [_i64, _dp]
        lib.oracle_sgd_momentum.argtypes = [_i64, _dp, _dp, _dp,
                                            ctypes.c_double, ctypes.c_double, ctypes.c_double]
        lib.oracle_adagrad.argtypes = [_i64, _dp, _dp, _dp, ctypes.c_double, ctypes.c_double, ctypes.c_double]
        _lib = lib
        return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray, typ=_dp):
    return a.ctypes.data_as(typ)


def _optr(a):
    return None if a is None else _ptr(a)


def conv_out(n: int, k: int, pad: int, stride: int) -> int:
    return int(_load().oracle_conv_out(n, k, pad, stride))


def pool_out(n: int, k: int, pad: int, stride: int, ceil_mode: bool = True) -> int:
    return int(_load().oracle_pool_out(n, k, pad, stride, int(bool(ceil_mode))))


def _geo(x_shape, w_shape, pad, stride):
    N, C, H, W = x_shape
    K, C2, R, S = w_shape
    if C != C2:
        raise ValueError("channel mismatch between input and filter")
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    return (N, C, H, W, K, R, S, ph, pw, sh, sw)


def conv_fwd(x, w, b=None, pad=0, stride=1) -> np.ndarray:
    """y = conv(x; w) + b, NCHW / KCRS, cross-correlation (Sec. 4.1.2 ComputeFeature)."""
    x, w = _f64(x), _f64(w)
    b = None if b is None else _f64(b)
    g = _geo(x.shape, w.shape, pad, stride)
    N, K = g[0], g[4]
    P = conv_out(g[2], g[5], g[7], g[9])
    Q = conv_out(g[3], g[6], g[8], g[10])
    y = np.empty((N, K, P, Q), np.float64)
    _load().oracle_conv_fwd(*g, _ptr(x), _ptr(w), _optr(b), _ptr(y))
    return y


def conv_bwd_data(dy, w, x_shape, pad=0, stride=1) -> np.ndarray:
    """Gradient w.r.t. the conv input (Sec. 4.1.2 ComputeGradient, source gradient)."""
    dy, w = _f64(dy), _f64(w)
    g = _geo(x_shape, w.shape, pad, stride)
    dx = np.empty(tuple(x_shape), np.float64)
    _load().oracle_conv_bwd_data(*g, _ptr(dy), _ptr(w), _ptr(dx))
    return dx


def conv_bwd_filter(x, dy, w_shape, pad=0, stride=1, with_bias=True):
    """Gradients w.r.t. the filter and bias (Sec. 4.1.2 ComputeGradient, Param gradients)."""
    x, dy = _f64(x), _f64(dy)
    g = _geo(x.shape, w_shape, pad, stride)
    dw = np.empty(tuple(w_shape), np.float64)
    db = np.empty((w_shape[0],), np.float64) if with_bias else None
    _load().oracle_conv_bwd_filter(*g, _ptr(x), _ptr(dy), _ptr(dw), _optr(db))
    return (dw, db) if with_bias else dw


def conv_fwd_points(x, w, b, idx, pad=0, stride=1) -> np.ndarray:
    x, w = _f64(x), _f64(w)
    b = None if b is None else _f64(b)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape, np.float64)
    g = _geo(x.shape, w.shape, pad, stride)
    _load().oracle_conv_fwd_points(*g, _ptr(x), _ptr(w), _optr(b), idx.size, _ptr(idx, _i64p), _ptr(out))
    return out


def conv_bwd_data_points(dy, w, x_shape, idx, pad=0, stride=1) -> np.ndarray:
    dy, w = _f64(dy), _f64(w)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape, np.float64)
    g = _geo(x_shape, w.shape, pad, stride)
    _load().oracle_conv_bwd_data_points(*g, _ptr(dy), _ptr(w), idx.size, _ptr(idx, _i64p), _ptr(out))
    return out


def conv_bwd_filter_points(x, dy, w_shape, idx, pad=0, stride=1) -> np.ndarray:
    x, dy = _f64(x), _f64(dy)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape, np.float64)
    g = _geo(x.shape, w_shape, pad, stride)
    _load().oracle_conv_bwd_filter_points(*g, _ptr(x), _ptr(dy), idx.size, _ptr(idx, _i64p), _ptr(out))
    return out


def fc_fwd(x, w, b=None) -> np.ndarray:
    x, w = _f64(x), _f64(w)
    b = None if b is None else _f64(b)
    N, I = x.shape
    J = w.shape[0]
    y = np.empty((N, J), np.float64)
    _load().oracle_fc_fwd(N, I, J, _ptr(x), _ptr(w), _optr(b), _ptr(y))
    return y


def fc_bwd(x, w, dy, with_bias=True):
    x, w, dy = _f64(x), _f64(w), _f64(dy)
    N, I = x.shape
    J = w.shape[0]
    dx = np.empty((N, I), np.float64)
    dw = np.empty((J, I), np.float64)
    db = np.empty((J,), np.float64) if with_bias else None
    _load().oracle_fc_bwd(N, I, J, _ptr(x), _ptr(w), _ptr(dy), _ptr(dx), _ptr(dw), _optr(db))
    return dx, dw, db


MAX, AVG = 0, 1


def pool_fwd(x, mode, k=3, stride=2, pad=0, ceil_mode=True):
    """Pooling ComputeFeature; returns (y, argmax) with argmax None for AVG."""
    x = _f64(x)
    N, C, H, W = x.shape
    kh, kw = (k, k) if np.isscalar(k) else k
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    P = pool_out(H, kh, ph, sh, ceil_mode)
    Q = pool_out(W, kw, pw, sw, ceil_mode)
    y = np.empty((N, C, P, Q), np.float64)
    am = np.empty((N, C, P, Q), np.uint8) if mode == MAX else None
    _load().oracle_pool_fwd(mode, N, C, H, W, kh, kw, sh, sw, ph, pw, int(bool(ceil_mode)),
                            _ptr(x), _ptr(y), None if am is None else _ptr(am, _u8p))
    return y, am


def pool_bwd(dy, argmax, x_shape, mode, k=3, stride=2, pad=0, ceil_mode=True):
    dy = _f64(dy)
    N, C, H, W = x_shape
    kh, kw = (k, k) if np.isscalar(k) else k
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    dx = np.empty(tuple(x_shape), np.float64)
    am = None
    if mode == MAX:
        am = np.ascontiguousarray(argmax, dtype=np.uint8)
    _load().oracle_pool_bwd(mode, N, C, H, W, kh, kw, sh, sw, ph, pw, int(bool(ceil_mode)),
                            _ptr(dy), None if am is None else _ptr(am, _u8p), _ptr(dx))
    return dx


def relu_fwd(x) -> np.ndarray:
    x = _f64(x)
    y = np.empty_like(x)
    _load().oracle_relu_fwd(x.size, _ptr(x), _ptr(y))
    return y


def lrn_fwd(x, size=5, alpha=1e-4, beta=0.75, k=1.0) -> np.ndarray:
    """Local response normalization across channels (NCHW), Caffe's form:
    y = x * (k + alpha/size * sum of x^2 over the channel window)^-beta."""
    x = _f64(x)
    y = np.empty_like(x)
    N, C, H, W = x.shape
    _load().oracle_lrn_fwd(N, C, H, W, _ptr(x), int(size), float(alpha), float(beta), float(k), _ptr(y))
    return y


def lrn_bwd(x, dy, size=5, alpha=1e-4, beta=0.75, k=1.0) -> np.ndarray:
    """Gradient of sum(dy * lrn_fwd(x)) with respect to x."""
    x, dy = _f64(x), _f64(dy)
    dx = np.empty_like(x)
    N, C, H, W = x.shape
    _load().oracle_lrn_bwd(N, C, H, W, _ptr(x), _ptr(dy), int(size), float(alpha), float(beta), float(k),
                           _ptr(dx))
    return dx


def relu_bwd(y, dy) -> np.ndarray:
    y, dy = _f64(y), _f64(dy)
    dx = np.empty_like(dy)
    _load().oracle_relu_bwd(dy.size, _ptr(y), _ptr(dy), _ptr(dx))
    return dx


def softmax_ce(z, labels):
    """Returns (mean loss, dz) for logits z (B x classes) and int labels."""
    z = _f64(z)
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    B, classes = z.shape
    dz = np.empty_like(z)
    loss = _load().oracle_softmax_ce(B, classes, _ptr(z), _ptr(lab, _i32p), _ptr(dz))
    return float(loss), dz


def round_bf16(x) -> np.ndarray:
    """Values a bf16 tensor holds after an fp32 computation produced x (returns a copy)."""
    y = _f64(x).copy()
    _load().oracle_round_bf16(y.size, _ptr(y))
    return y


def adagrad(w, g, h, lr, delta, wd=0.0):
    """One AdaGrad Updater step (Sec. 4.1.4; Duchi et al. 2011, diagonal form);
    returns new (w, h) and leaves inputs alone."""
    w = _f64(w).copy()
    h = _f64(h).copy()
    g = _f64(g)
    _load().oracle_adagrad(w.size, _ptr(w), _ptr(g), _ptr(h), float(lr), float(delta), float(wd))
    return w, h


def sgd_momentum(w, g, v, lr, momentum, wd=0.0):
    """One Updater step (Sec. 4.1.4); returns new (w, v) and leaves inputs alone."""
    w = _f64(w).copy()
    v = _f64(v).copy()
    g = _f64(g)
    _load().oracle_sgd_momentum(w.size, _ptr(w), _ptr(g), _ptr(v),
                                float(lr), float(momentum), float(wd))
    return w, v
