"""BPTrainOneBatch (Sec. 4.1.3, Alg. 1) over the C-ABI library, one GPU.

Layers mirror the paper's Layer abstraction (Sec. 4.1.2): ``compute_feature``
maps the source layer's blob to this layer's blob, ``compute_gradient``
produces the Param gradients and the source layer's gradient.  The whole
step runs in the library's HIP kernels on torch's current stream; this module
only wires buffers together.

Data layout in HBM (chosen for the gfx950 kernels, not the paper's CPUs):
  * activations and their gradients are NHWC, in the workload's dtype
    (fp32, or bf16 with fp32 accumulation inside the kernels);
  * filters are KRSC; a fully connected layer is a convolution whose filter
    covers the whole input (R = H, S = W, no padding), so its weight matrix
    is KRSC too, i.e. its input is flattened in (h, w, c) order;
  * all parameters live in one flat fp32 master buffer (weights then bias per
    layer, each padded to 64 elements), with a flat fp32 gradient buffer, a
    flat fp32 momentum buffer and, for bf16 workloads, a flat bf16 shadow
    that the fused Updater writes; per-layer tensors are views into these.
Every buffer is allocated once, when the net is built; a step allocates
nothing.

Alg. 1 calls Update(layer.params()) inside the backward loop, right after the
layer's ComputeGradient.  Layers whose filter gradient is one pass of the
large gradient kernel (the fully connected layers, which hold almost all of
the parameters) do exactly that: the update is fused into the gradient
kernel, so their gradient never goes through memory, and their backward-data
runs first because it still needs the old bf16 weights.  The other layers'
gradients go to the flat gradient buffer and one fused update over their
(contiguous) part of the flat buffers follows the backward loop; the fresh
values only reach any layer at the next iteration's forward, so this is the
same computation, element for element.

With ``concurrent_wgrad`` (the default on a GPU) the filter gradients, and
the fused gradient + update of the fully connected layers, run on a second
stream as soon as their inputs exist, beside the backward-data passes of the
layers below; the backward loop ends by joining the two streams.
"""
from __future__ import annotations

import contextlib
from typing import Dict, List, Optional

import numpy as np
import torch

from . import singa
from . import workloads as wl

PAD = 64  # elements; keeps every parameter view 256-byte aligned


def _pad(n: int) -> int:
    return (n + PAD - 1) // PAD * PAD


class Layer:
    name = ""
    params: List = []

    def compute_feature(self, x):
        raise NotImplementedError

    def compute_gradient(self, dy, need_dx=True):
        raise NotImplementedError


class ConvLayer(Layer):
    """Convolution (or fully connected, as a whole-input convolution)."""

    def __init__(self, net, spec, in_shape, fc=False):
        self.name = spec.name
        self.net = net
        N, H, W, C = in_shape
        if fc:
            self.K, self.R, self.S, self.pad, self.stride = spec.out_features, H, W, 0, 1
        else:
            self.K, self.R, self.S, self.pad, self.stride = (spec.out_channels, spec.kernel, spec.kernel, spec.pad,
                                                             spec.stride)
        self.fc = fc
        self.has_bias = spec.bias
        self.in_shape = (N, H, W, C)
        self.w_shape = (self.K, self.R, self.S, C)
        self.out_shape = singa.conv_out_shape(self.in_shape, self.w_shape, self.pad, self.stride)
        self.relu = False  # set when a ReLU layer directly follows and is fused
        self.relu_src = None  # the ReLU layer feeding this one, whose backward bwd-data folds in
        dev, dt = net.device, net.dtype
        # update fused into the filter-gradient kernel (no workspace needed exactly then)
        self.fused_update = bool(net.fuse_update and net.wl.update and net.updater == "sgd" and singa.conv_workspace_bytes(
            singa.OP_BWD_FILTER_SGD, dt, self.in_shape, self.w_shape, self.pad, self.stride) == 0)
        # update applied by the filter gradient's split-K reduction (convolutions
        # whose input the library takes as it is)
        self.reduce_update = bool(net.fuse_update and net.reduce_update and net.wl.update and net.updater == "sgd"
                                  and not self.fused_update and not fc
                                  and singa.space_to_depth_bytes(dt, self.in_shape, self.w_shape, self.pad,
                                                                 self.stride) == 0)
        self.y = singa.empty(self.out_shape, dt, dev)
        self.dx = singa.empty(self.in_shape, dt, dev)
        self.x = None
        # a strided layer that the library runs on the space-to-depth form of
        # its input (the first layer): that form is built once per step and
        # read by both the forward pass and the filter gradient
        self.xs = None
        if not fc and singa.space_to_depth_bytes(dt, self.in_shape, self.w_shape, self.pad, self.stride) > 0:
            self.xs = singa.empty(singa.space_to_depth_shape(self.in_shape, self.w_shape, self.pad, self.stride),
                                  dt, dev)
        self.x_layout = "NHWC_S2D" if self.xs is not None else "NHWC"
        for op in (singa.OP_FWD, singa.OP_BWD_DATA, singa.OP_BWD_FILTER):
            net.need_workspace(singa.conv_workspace_bytes(op, dt, self.in_shape, self.w_shape, self.pad,
                                                          self.stride,
                                                          self.x_layout if op != singa.OP_BWD_DATA else "NHWC"))
        wop = singa.OP_BWD_FILTER_SGD if self.reduce_update else singa.OP_BWD_FILTER
        net.ws_wgrad_bytes = max(net.ws_wgrad_bytes, singa.conv_workspace_bytes(
            wop, dt, self.in_shape, self.w_shape, self.pad, self.stride, self.x_layout))
        if self.reduce_update:
            net.need_workspace(net.ws_wgrad_bytes)

    def bind(self, w, b, w_compute, dw, db, v, vb, b_compute):
        self.w, self.b, self.w_compute, self.dw, self.db = w, b, w_compute, dw, db
        self.v, self.vb, self.b_compute = v, vb, b_compute

    def compute_feature(self, x):
        if self.xs is not None:
            singa.space_to_depth(x, self.w_shape, self.pad, self.stride, out=self.xs)
            x = self.xs
        self.x = x
        singa.conv_fwd(x, self.w_compute, self.b, self.pad, self.stride, relu=self.relu, out=self.y,
                       workspace=self.net.workspace, layout=self.x_layout, x_shape=self.in_shape)
        return self.y

    def compute_gradient(self, dy, need_dx=True):
        if self.fused_update or self.reduce_update:
            # backward-data first: it reads the bf16 weights the update rewrites
            # (fused into the gradient kernel, or applied by its split-K
            # reduction)
            self._bwd_data(dy, need_dx)
            net, wl_ = self.net, self.net.wl
            keep = net.keep_grads
            side = net.wgrad_stream
            # with a second stream, gradient + update run there, beside the
            # backward passes of the layers below (which read neither this
            # layer's weights nor write its x or dy)
            if side is not None:
                side.wait_stream(torch.cuda.current_stream(net.device))
            with torch.cuda.stream(side) if side is not None else contextlib.nullcontext():
                singa.conv_bwd_filter_sgd(
                    self.x, dy, self.w_shape, self.w, self.v, self.w_compute if net.wb_flat is not None else None,
                    b=self.b, vb=self.vb, b_bf16=self.b_compute, lr=wl_.lr, momentum=wl_.momentum,
                    weight_decay=wl_.weight_decay, pad=self.pad, stride=self.stride,
                    dw=self.dw if keep else None,
                    db=self.db if keep else None, workspace=net.workspace if side is None else net.workspace_wgrad)
            return self.dx if need_dx else None
        side = self.net.wgrad_stream
        if side is None or (not need_dx and self.net.last_wgrad_on_main):
            # one stream; or the first layer of a training step, whose input
            # gradient is not needed: the main stream has nothing left to do,
            # while the second one is still busy with the layers above
            singa.conv_bwd_filter(self.x, dy, self.w_shape, self.pad, self.stride, with_bias=self.has_bias,
                                  dw=self.dw, db=self.db, workspace=self.net.workspace, layout=self.x_layout,
                                  x_shape=self.in_shape)
        else:
            # the filter gradient on the second stream, beside this layer's
            # backward-data and the layers below (both only read dy and x)
            side.wait_stream(torch.cuda.current_stream(self.net.device))
            with torch.cuda.stream(side):
                singa.conv_bwd_filter(self.x, dy, self.w_shape, self.pad, self.stride, with_bias=self.has_bias,
                                      dw=self.dw, db=self.db, workspace=self.net.workspace_wgrad,
                                      layout=self.x_layout, x_shape=self.in_shape)
        return self._bwd_data(dy, need_dx)

    def _bwd_data(self, dy, need_dx):
        if not need_dx:
            return None
        singa.conv_bwd_data(dy, self.w_compute, self.in_shape, self.pad, self.stride, out=self.dx,
                            workspace=self.net.workspace,
                            relu_y=None if self.relu_src is None else self.relu_src.y)
        return self.dx


class PoolLayer(Layer):
    def __init__(self, net, spec, in_shape):
        self.name = spec.name
        self.mode = spec.mode
        self.k, self.stride, self.pad, self.ceil = spec.kernel, spec.stride, spec.pad, spec.ceil_mode
        self.in_shape = tuple(in_shape)
        self.out_shape = singa.pool_out_shape(self.in_shape, self.mode, self.k, self.stride, self.pad, self.ceil)
        dev, dt = net.device, net.dtype
        self.y = singa.empty(self.out_shape, dt, dev)
        self.argmax = singa.empty(self.out_shape, torch.uint8, dev) if self.mode == "max" else None
        self.dx = singa.empty(self.in_shape, dt, dev)
        self.relu_src = None  # the ReLU layer feeding this max pooling, whose backward folds in

    def compute_feature(self, x):
        singa.pool_fwd(x, self.mode, self.k, self.stride, self.pad, self.ceil, out=self.y, argmax=self.argmax)
        return self.y

    def compute_gradient(self, dy, need_dx=True):
        singa.pool_bwd(dy, self.argmax, self.in_shape, self.mode, self.k, self.stride, self.pad, self.ceil,
                       out=self.dx, relu_y=None if self.relu_src is None else self.y)
        return self.dx


class ReluLayer(Layer):
    def __init__(self, net, spec, in_shape, fused_into: Optional[ConvLayer]):
        self.name = spec.name
        self.fused = fused_into
        self.folded = False  # backward done by the consuming layer (set by Net)
        self.out_shape = tuple(in_shape)
        self.y = None
        if fused_into is None:
            self.y = singa.empty(self.out_shape, net.dtype, net.device)

    def compute_feature(self, x):
        if self.fused is not None:
            self.y = x  # the producing convolution already applied max(., 0)
            return x
        singa.relu_fwd(x, out=self.y)
        return self.y

    def compute_gradient(self, dy, need_dx=True):
        if self.folded:
            return dy  # the consuming layer already produced the gradient at this ReLU's input
        # in place on the incoming gradient buffer
        return singa.relu_bwd(self.y, dy, out=dy)


class LrnLayer(Layer):
    """Local response normalization across channels (the layer Sec. 5.4.1
    names beside pooling)."""

    def __init__(self, net, spec, in_shape):
        self.name = spec.name
        self.args = (spec.size, spec.alpha, spec.beta, spec.k)
        self.in_shape = self.out_shape = tuple(in_shape)
        self.y = singa.empty(self.out_shape, net.dtype, net.device)
        self.dx = singa.empty(self.in_shape, net.dtype, net.device)
        self.x = None

    def compute_feature(self, x):
        self.x = x
        return singa.lrn_fwd(x, *self.args, out=self.y)

    def compute_gradient(self, dy, need_dx=True):
        if not need_dx:
            return None
        return singa.lrn_bwd(self.x, dy, *self.args, out=self.dx)


class SoftmaxCELayer(Layer):
    def __init__(self, net, spec, in_shape):
        self.name = spec.name
        self.in_shape = tuple(in_shape)
        self.loss = singa.empty((in_shape[0] + 1,), torch.float32, net.device)  # mean, then rows
        self.dz = singa.empty(self.in_shape, net.dtype, net.device)
        self.labels = None
        self.out_shape = (1,)

    def compute_feature(self, z):
        B = z.shape[0]
        singa.softmax_ce(z.reshape(B, -1), self.labels, loss=self.loss, dz=self.dz.reshape(B, -1))
        return self.loss

    def compute_gradient(self, dy=None, need_dx=True):
        return self.dz


class Net:
    """A workload's layer stack on one GPU, with flat parameter buffers."""

    def __init__(self, workload: wl.Workload, batch: Optional[int] = None, device="cuda", fuse_update: bool = True,
                 keep_grads: bool = False, concurrent_wgrad: bool = True, updater: str = "sgd",
                 adagrad_delta: float = 1e-6, reduce_update: bool = False, last_wgrad_on_main: bool = True,
                 side_update: bool = True):
        """fuse_update: apply the update inside the filter-gradient kernel
        where it can be fused; keep_grads: those layers also store their
        gradients in the flat gradient buffer (for inspection);
        concurrent_wgrad: the filter gradients (with the fused update where
        there is one) run on a second stream, concurrently with the
        backward-data passes, except the first layer's when its input
        gradient is not needed (last_wgrad_on_main: that one runs on the
        main stream, idle by then); updater: "sgd"
        (momentum, the workloads' Updater) or "adagrad" (Sec. 4.1.4's named
        protocol, with the workload's learning rate and weight decay; the
        momentum buffer holds its sums of squared gradients); side_update:
        with a second stream, the update of every layer whose filter gradient
        ran there (all but the first) also runs there, once the main stream
        has issued the last backward-data pass that reads those weights,
        beside the first layer's filter gradient on the main stream (0.4-0.6 %
        faster on the AlexNet-shaped step than the whole update after it)."""
        if updater not in ("sgd", "adagrad"):
            raise ValueError(updater)
        self.updater = updater
        self.adagrad_delta = adagrad_delta
        self.reduce_update = reduce_update
        self.last_wgrad_on_main = last_wgrad_on_main
        self.side_update = side_update
        self.wl = workload
        self.fuse_update = fuse_update
        self.keep_grads = keep_grads
        self.ws_wgrad_bytes = 0
        self.batch = workload.batch if batch is None else batch
        self.device = torch.device(device)
        self.dtype = torch.bfloat16 if workload.dtype == "bf16" else torch.float32
        self.ws_bytes = 0
        self.layers: List[Layer] = []
        C, H, W = workload.in_shape
        shape = (self.batch, H, W, C)
        prev = None
        for spec in workload.layers:
            if isinstance(spec, wl.Conv):
                layer = ConvLayer(self, spec, shape)
            elif isinstance(spec, wl.FC):
                layer = ConvLayer(self, spec, shape, fc=True)
            elif isinstance(spec, wl.Pool):
                layer = PoolLayer(self, spec, shape)
            elif isinstance(spec, wl.Relu):
                fuse = prev if isinstance(prev, ConvLayer) else None
                if fuse is not None:
                    fuse.relu = True
                layer = ReluLayer(self, spec, shape, fuse)
            elif isinstance(spec, wl.Lrn):
                layer = LrnLayer(self, spec, shape)
            elif isinstance(spec, wl.SoftmaxCE):
                layer = SoftmaxCELayer(self, spec, shape)
            else:
                raise TypeError(spec)
            # a convolution's backward-data or a max pooling's backward can
            # also apply the backward of the ReLU that feeds it
            if isinstance(prev, ReluLayer) and (isinstance(layer, ConvLayer) or
                                               (isinstance(layer, PoolLayer) and layer.mode == "max")):
                layer.relu_src = prev
                prev.folded = True
            self.layers.append(layer)
            shape = layer.out_shape
            prev = layer
        self.out_shape = shape
        self.workspace = singa.empty((max(self.ws_bytes, 256),), torch.uint8, self.device)
        # default priority, like every stream the library runs on
        self.wgrad_stream = None
        if concurrent_wgrad and self.device.type == "cuda" and any(isinstance(l, ConvLayer) for l in self.layers):
            self.wgrad_stream = torch.cuda.Stream(device=self.device)
            self.workspace_wgrad = singa.empty((max(self.ws_wgrad_bytes, 256),), torch.uint8, self.device)
        self._build_params()

    def need_workspace(self, nbytes: int):
        self.ws_bytes = max(self.ws_bytes, int(nbytes))

    def param_layers(self) -> List[ConvLayer]:
        return [l for l in self.layers if isinstance(l, ConvLayer)]

    def _build_params(self):
        offs = []
        total = 0
        for l in self.param_layers():
            nw = int(np.prod(l.w_shape))
            nb = l.K if l.has_bias else 0
            offs.append((total, nw, total + _pad(nw), nb))
            total += _pad(nw) + _pad(nb)
        self.n_params_padded = total
        self.n_params = sum(o[1] + o[3] for o in offs)
        dev = self.device
        self.w_flat = singa.empty((total,), torch.float32, dev).zero_()
        self.g_flat = singa.empty((total,), torch.float32, dev).zero_()
        self.v_flat = singa.empty((total,), torch.float32, dev).zero_()
        self.wb_flat = singa.empty((total,), torch.bfloat16, dev).zero_() if self.dtype == torch.bfloat16 else None
        self.offsets = offs
        for l, (ow, nw, ob, nb) in zip(self.param_layers(), offs):
            l.flat_range = (ow, ob + _pad(nb))  # the layer's weights and bias, padding included
            w = self.w_flat[ow:ow + nw].view(l.w_shape)
            dw = self.g_flat[ow:ow + nw].view(l.w_shape)
            v = self.v_flat[ow:ow + nw].view(l.w_shape)
            b = self.w_flat[ob:ob + nb] if nb else None
            db = self.g_flat[ob:ob + nb] if nb else None
            vb = self.v_flat[ob:ob + nb] if nb else None
            wc = self.wb_flat[ow:ow + nw].view(l.w_shape) if self.wb_flat is not None else w
            bc = self.wb_flat[ob:ob + nb] if (nb and self.wb_flat is not None) else None
            l.bind(w, b, wc, dw, db, v, vb, bc)
        # contiguous runs of the flat buffers that the update after the backward
        # loop covers (with side_update: the first parameter layer's alone on
        # the main stream, the others' on the second stream)
        plain = [l for l in self.param_layers() if not (l.fused_update or l.reduce_update)]
        on_side = self.side_update and self.wgrad_stream is not None and len(plain) > 1
        self.side_update_layers = plain[1:] if on_side else []
        self.side_update_ranges = self._runs(self.side_update_layers)
        self.main_update_ranges = self._runs(plain[:1] if on_side else plain)
        self.update_ranges = self._runs(plain)
        self._issued = None

    @staticmethod
    def _runs(layers):
        runs = []
        for l in layers:
            a, e = l.flat_range
            if runs and runs[-1][1] == a:
                runs[-1] = (runs[-1][0], e)
            else:
                runs.append((a, e))
        return runs

    # ------------------------------------------------------------ marshalling
    def load_params(self, params: List[wl.LayerParams]):
        """Copy fp32 master parameters (KCRS / (J, I) with I in (c, h, w) order)
        into the flat buffers, permuted to KRSC; fill the bf16 shadow with the
        round-to-nearest-even bf16 copy."""
        flat = np.zeros(self.n_params_padded, np.float32)
        for l, p, (ow, nw, ob, nb) in zip(self.param_layers(), params, self.offsets):
            K, R, S, C = l.w_shape
            w = np.asarray(p.w, np.float32).reshape(K, C, R, S).transpose(0, 2, 3, 1)
            flat[ow:ow + nw] = w.ravel()
            if nb:
                flat[ob:ob + nb] = np.asarray(p.b, np.float32)
        self.w_flat.copy_(torch.from_numpy(flat))
        self.v_flat.zero_()
        if self.wb_flat is not None:
            bits = wl.bf16_bits(flat).view(np.int16)
            self.wb_flat.view(torch.int16).copy_(torch.from_numpy(bits))

    def to_device_input(self, x_nchw: np.ndarray) -> torch.Tensor:
        t = torch.from_numpy(np.ascontiguousarray(np.asarray(x_nchw, np.float32).transpose(0, 2, 3, 1)))
        return t.to(self.device).to(self.dtype)

    # --------------------------------------------------------------- Alg. 1
    def forward(self, x, labels=None):
        h = x
        for l in self.layers:
            if isinstance(l, SoftmaxCELayer):
                l.labels = labels
            h = l.compute_feature(h)
        return h

    def backward(self, dy_top=None, need_input_grad=False, defer_join=False):
        """Alg. 1's backward loop.  The second stream is joined at the end,
        unless defer_join (train_one_batch with side_update): then update()
        issues the second-stream update and joins."""
        g = dy_top
        side_after = (self.side_update_layers[0]
                      if defer_join and self.side_update_layers and self.wgrad_stream is not None else None)
        self._issued = None
        for i in range(len(self.layers) - 1, -1, -1):
            g = self.layers[i].compute_gradient(g, need_dx=(i > 0 or need_input_grad))
            if self.layers[i] is side_after:
                # every backward-data pass that reads those layers' weights is issued
                self._issued = torch.cuda.Event()
                self._issued.record(torch.cuda.current_stream(self.device))
        if self.wgrad_stream is not None and self._issued is None:
            torch.cuda.current_stream(self.device).wait_stream(self.wgrad_stream)
        return g

    def update(self):
        """The update of every layer whose update is not fused into its
        filter-gradient kernel, over their parts of the flat buffers; after a
        backward pass with a deferred join, the layers whose filter gradient
        ran on the second stream are updated there (once the main stream has
        issued their backward-data passes), then the streams join."""
        if self._issued is not None:
            self.wgrad_stream.wait_event(self._issued)
            with torch.cuda.stream(self.wgrad_stream):
                self._update_ranges(self.side_update_ranges)
            torch.cuda.current_stream(self.device).wait_stream(self.wgrad_stream)
            self._issued = None
            self._update_ranges(self.main_update_ranges)
        else:
            self._update_ranges(self.update_ranges)

    def _update_ranges(self, ranges):
        for a, e in ranges:
            wb = self.wb_flat[a:e] if self.wb_flat is not None else None
            if self.updater == "adagrad":
                singa.adagrad_update(self.w_flat[a:e], self.g_flat[a:e], self.v_flat[a:e], wb, self.wl.lr,
                                     self.adagrad_delta, self.wl.weight_decay)
            else:
                singa.sgd_momentum_update(self.w_flat[a:e], self.g_flat[a:e], self.v_flat[a:e], wb, self.wl.lr,
                                          self.wl.momentum, self.wl.weight_decay)

    def train_one_batch(self, x, labels=None, dy_top=None, need_input_grad=False):
        self.forward(x, labels)
        gx = self.backward(dy_top, need_input_grad, defer_join=self.wl.update)
        if self.wl.update:
            self.update()
        return gx

    def capture(self, x, labels=None, dy_top=None, need_input_grad=False) -> torch.cuda.CUDAGraph:
        """Record one train_one_batch on (x, labels, dy_top) into a HIP graph.

        A step launches some 75 kernels whose host-side launch cost is
        comparable to the shorter ones; replaying the graph issues them all at
        once.  Every buffer a step touches was allocated when the net was
        built and the library allocates nothing and records no memset, so the
        graph holds exactly the step's kernels.  Capturing runs nothing;
        each ``replay()`` performs one full step (forward, backward, update)
        on whatever the captured input, label and gradient tensors hold then.
        """
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.train_one_batch(x, labels, dy_top, need_input_grad)
        return g

    def layer(self, name: str) -> Layer:
        for l in self.layers:
            if l.name == name:
                return l
        raise KeyError(name)
