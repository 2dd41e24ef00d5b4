"""Oracle network driver: BPTrainOneBatch (Sec. 4.1.3, Alg. 1) over the fp64 oracle.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The forward loop visits the layers in order and calls each layer's
ComputeFeature; the backward loop visits them in reverse and calls
ComputeGradient, which yields the parameter gradients and the source layer's
gradient (Sec. 4.1.2); the Updater (Sec. 4.1.4) then applies SGD with
momentum to every parameter.  All arithmetic is the oracle's (fp64).

Layer records are duck-typed by class name ("Conv", "Pool", "Relu", "FC",
"SoftmaxCE") and read only through their attributes, so this module needs
no import from outside the oracle.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from . import (AVG, MAX, adagrad, conv_bwd_data, conv_bwd_filter, conv_fwd, fc_bwd, fc_fwd, lrn_bwd, lrn_fwd,
               pool_bwd, pool_fwd, relu_bwd, relu_fwd, sgd_momentum, softmax_ce)


def _kind(layer) -> str:
    return type(layer).__name__


def forward(layers, x, params: List, labels=None, store=None) -> Dict:
    """Forward pass.  ``params`` is a list of (w, b) in forward order of the
    parametrised layers (conv KCRS, FC (J, I) with I flattened as (c, h, w)).
    Returns a dict with per-layer outputs ``out[name]``, pooling argmax
    ``argmax[name]``, and, for a stack ending in a softmax loss, ``loss`` and
    ``dlogits``.  ``store`` (optional) is applied to every layer output, as
    the storage rounding of a reduced-precision pipeline."""
    keep = (lambda a: a) if store is None else store
    acts = {"out": {}, "argmax": {}, "in": {}}
    h = np.asarray(x, dtype=np.float64)
    pi = 0
    for l in layers:
        k = _kind(l)
        acts["in"][l.name] = h
        if k == "Conv":
            w, b = params[pi]
            pi += 1
            h = conv_fwd(h, w, b, pad=l.pad, stride=l.stride)
        elif k == "Pool":
            mode = MAX if l.mode == "max" else AVG
            h, am = pool_fwd(h, mode, k=l.kernel, stride=l.stride, pad=l.pad, ceil_mode=l.ceil_mode)
            acts["argmax"][l.name] = am
        elif k == "Relu":
            h = relu_fwd(h)
        elif k == "Lrn":
            h = lrn_fwd(h, l.size, l.alpha, l.beta, l.k)
        elif k == "FC":
            w, b = params[pi]
            pi += 1
            B = h.shape[0]
            h = fc_fwd(h.reshape(B, -1), w, b).reshape(B, -1, 1, 1)
        elif k == "SoftmaxCE":
            B = h.shape[0]
            loss, dz = softmax_ce(h.reshape(B, -1), labels)
            acts["loss"] = loss
            acts["dlogits"] = keep(dz.reshape(h.shape))
        else:
            raise ValueError("unknown layer kind %s" % k)
        if k != "SoftmaxCE":
            h = keep(h)
        acts["out"][l.name] = h
    return acts


def backward(layers, params: List, acts: Dict, dy_top=None, need_input_grad: bool = False, store=None) -> Dict:
    """Backward pass in reverse layer order.  Returns ``grad_in[name]`` (the
    gradient w.r.t. each layer's input), and ``dw[name]``/``db[name]`` for
    parametrised layers.  The first layer's input gradient is only computed
    when ``need_input_grad`` is set (training never needs it).  ``store`` is
    applied to every activation gradient, as in ``forward``."""
    keep = (lambda a: a) if store is None else store
    res = {"grad_in": {}, "dw": {}, "db": {}}
    pidx = {}
    pi = 0
    for l in layers:
        if _kind(l) in ("Conv", "FC"):
            pidx[l.name] = pi
            pi += 1
    g = None if dy_top is None else np.asarray(dy_top, dtype=np.float64)
    for li in range(len(layers) - 1, -1, -1):
        l = layers[li]
        k = _kind(l)
        xin = acts["in"][l.name]
        first = li == 0
        if k == "SoftmaxCE":
            g = acts["dlogits"]
        elif k == "Relu":
            g = relu_bwd(acts["out"][l.name], g)
        elif k == "Lrn":
            g = lrn_bwd(xin, g, l.size, l.alpha, l.beta, l.k)
        elif k == "Pool":
            mode = MAX if l.mode == "max" else AVG
            g = pool_bwd(g, acts["argmax"].get(l.name), xin.shape, mode, k=l.kernel,
                         stride=l.stride, pad=l.pad, ceil_mode=l.ceil_mode)
        elif k == "Conv":
            w, b = params[pidx[l.name]]
            if b is not None:
                dw, db = conv_bwd_filter(xin, g, w.shape, pad=l.pad, stride=l.stride, with_bias=True)
            else:
                dw, db = conv_bwd_filter(xin, g, w.shape, pad=l.pad, stride=l.stride, with_bias=False), None
            res["dw"][l.name], res["db"][l.name] = dw, db
            g = conv_bwd_data(g, w, xin.shape, pad=l.pad, stride=l.stride) if (not first or need_input_grad) else None
        elif k == "FC":
            w, b = params[pidx[l.name]]
            B = xin.shape[0]
            dx, dw, db = fc_bwd(xin.reshape(B, -1), w, g.reshape(B, -1), with_bias=b is not None)
            res["dw"][l.name], res["db"][l.name] = dw, db
            g = dx.reshape(xin.shape)
        else:
            raise ValueError("unknown layer kind %s" % k)
        if g is not None:
            g = keep(g)
        res["grad_in"][l.name] = g
    return res


def train_one_batch(layers, x, params: List, master: Optional[List] = None, labels=None, dy_top=None,
                    lr: float = 0.0, momentum: float = 0.0, wd: float = 0.0, velocity: Optional[List] = None,
                    need_input_grad: bool = False, store=None, adagrad_delta: Optional[float] = None) -> Dict:
    """Alg. 1 followed by the Updater.  ``params`` are the values the layers
    compute with; ``master`` (default: ``params``) are the values the Updater
    steps (for bf16 compute these are the fp32 master weights).  Returns the
    forward dict, the backward dict and the updated (w, b) and momentum.
    ``store`` rounds stored activations and activation gradients (see
    ``forward``); parameter gradients and the update stay in fp64.  With
    ``adagrad_delta`` the Updater is AdaGrad (``momentum`` unused) and
    ``velocity`` holds its sums of squared gradients."""
    acts = forward(layers, x, params, labels=labels, store=store)
    grads = backward(layers, params, acts, dy_top=dy_top, need_input_grad=need_input_grad, store=store)
    master = params if master is None else master
    names = [l.name for l in layers if _kind(l) in ("Conv", "FC")]
    new_params, new_vel = [], []
    for i, name in enumerate(names):
        w, b = master[i]
        vw, vb = (None, None) if velocity is None else velocity[i]
        vw = np.zeros(np.shape(w)) if vw is None else vw
        def step(p, g, state):
            if adagrad_delta is not None:
                return adagrad(p, g, state, lr, adagrad_delta, wd)
            return sgd_momentum(p, g, state, lr, momentum, wd)
        w2, vw2 = step(w, grads["dw"][name], vw)
        if b is not None:
            vb = np.zeros(np.shape(b)) if vb is None else vb
            b2, vb2 = step(b, grads["db"][name], vb)
        else:
            b2 = vb2 = None
        new_params.append((w2, b2))
        new_vel.append((vw2, vb2))
    return {"acts": acts, "grads": grads, "params": new_params, "velocity": new_vel}
