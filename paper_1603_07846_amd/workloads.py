"""Seeded synthetic workloads for the SINGA conv-training hot path.

This module holds only workload *data*: the five layer stacks as plain
records and the seeded input generators that feed both the GPU library and
the CPU oracle.  It contains none of the method's arithmetic (no convolution,
pooling or loss math); every expected output shape is listed here as data so
that each side can check its own shape arithmetic against it.

Inputs stand in for the paper's workloads (Sec. 6.2.1 trains the cuda-convnet
CIFAR-10 DCNN; Sec. 6.3.1 trains an AlexNet variant on ImageNet-sized images):
uniform images with random labels replace CIFAR-10, standard-normal
227x227 images with random 1000-way labels replace ImageNet.  No dataset is
read.

Draw order (one ``numpy.random.default_rng(1603078460 + cfg)`` stream per
workload): the input batch; then, per parametrised layer in forward order,
its weights (normal, std 0.01) followed by a zero bias; then either the class
labels or the upstream gradient.  Values are drawn in float64 and rounded to
fp32 (round to nearest even); for bf16 workloads the compute copies are
rounded again to bf16 (round to nearest even) by ``bf16_bits``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

SEED_BASE = 1603078460


@dataclass(frozen=True)
class Conv:
    name: str
    out_channels: int
    kernel: int
    stride: int = 1
    pad: int = 0
    bias: bool = True
    out_shape: Tuple[int, int, int] = (0, 0, 0)  # (C, H, W) per image, as data


@dataclass(frozen=True)
class Pool:
    name: str
    mode: str  # "max" or "avg"
    kernel: int = 3
    stride: int = 2
    pad: int = 0
    ceil_mode: bool = True
    out_shape: Tuple[int, int, int] = (0, 0, 0)


@dataclass(frozen=True)
class Relu:
    name: str


@dataclass(frozen=True)
class Lrn:
    """Local response normalization across channels (Caffe's form):
    y = x * (k + alpha/size * sum of x^2 over `size` channels)^-beta."""
    name: str
    size: int = 5
    alpha: float = 1e-4
    beta: float = 0.75
    k: float = 1.0


@dataclass(frozen=True)
class FC:
    name: str
    out_features: int
    bias: bool = True
    out_shape: Tuple[int, int, int] = (0, 1, 1)


@dataclass(frozen=True)
class SoftmaxCE:
    name: str = "loss"


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    dtype: str  # "f32" or "bf16"
    batch: int
    in_shape: Tuple[int, int, int]  # (C, H, W)
    input_dist: str  # "uniform01", "uniform11" or "normal"
    layers: Tuple
    classes: int = 0  # > 0 when the stack ends in a softmax loss
    lr: float = 0.0
    momentum: float = 0.0
    weight_decay: float = 0.0
    update: bool = False
    description: str = ""

    def param_layers(self):
        return [l for l in self.layers if isinstance(l, (Conv, FC))]


def _conv(name, k, r, s=1, p=0, bias=True, out=(0, 0, 0)):
    return Conv(name, k, r, s, p, bias, out)


CFG1 = Workload(
    1, "single conv layer, 16x3x32x32, 32 filters 5x5 p2, fp32", "f32", 16, (3, 32, 32), "uniform11",
    (_conv("conv1", 32, 5, 1, 2, bias=False, out=(32, 32, 32)),),
    lr=0.01, momentum=0.9, weight_decay=0.0, update=True,
    description="conv fwd + bwd-data + bwd-filter, then SGD-momentum on the filter")

CFG2 = Workload(
    2, "CIFAR-10-shaped convnet training step, batch 100, fp32", "f32", 100, (3, 32, 32), "uniform01",
    (
        _conv("conv1", 32, 5, 1, 2, out=(32, 32, 32)),
        Pool("pool1", "max", 3, 2, 0, True, (32, 16, 16)),
        Relu("relu1"),
        _conv("conv2", 32, 5, 1, 2, out=(32, 16, 16)),
        Relu("relu2"),
        Pool("pool2", "avg", 3, 2, 0, True, (32, 8, 8)),
        _conv("conv3", 64, 5, 1, 2, out=(64, 8, 8)),
        Relu("relu3"),
        Pool("pool3", "avg", 3, 2, 0, True, (64, 4, 4)),
        FC("fc", 10, out_shape=(10, 1, 1)),
        SoftmaxCE(),
    ),
    classes=10, lr=0.01, momentum=0.9, weight_decay=0.0, update=True,
    description="conv-maxpool-relu, conv-relu-avgpool, conv-relu-avgpool, FC 1024->10, softmax-CE, SGD")

_ALEX_STACK = (
    _conv("conv1", 96, 11, 4, 0, out=(96, 55, 55)),
    Relu("relu1"),
    Pool("pool1", "max", 3, 2, 0, True, (96, 27, 27)),
    _conv("conv2", 256, 5, 1, 2, out=(256, 27, 27)),
    Relu("relu2"),
    Pool("pool2", "max", 3, 2, 0, True, (256, 13, 13)),
    _conv("conv3", 384, 3, 1, 1, out=(384, 13, 13)),
    Relu("relu3"),
    _conv("conv4", 384, 3, 1, 1, out=(384, 13, 13)),
    Relu("relu4"),
    _conv("conv5", 256, 3, 1, 1, out=(256, 13, 13)),
    Relu("relu5"),
)

CFG3 = Workload(
    3, "AlexNet-shaped conv stack fwd+bwd, batch 128, fp32", "f32", 128, (3, 227, 227), "normal",
    _ALEX_STACK, description="conv stack forward and backward, upstream gradient N(0,1) at relu5")

CFG4 = Workload(
    4, "AlexNet-shaped conv stack fwd+bwd, batch 256, bf16 (fp32 accumulate)", "bf16", 256, (3, 227, 227),
    "normal", _ALEX_STACK, description="as workload 3 in bf16")

CFG5 = Workload(
    5, "AlexNet-shaped training step, batch 256, bf16 compute, fp32 master weights", "bf16", 256,
    (3, 227, 227), "normal",
    _ALEX_STACK + (
        Pool("pool5", "max", 3, 2, 0, True, (256, 6, 6)),
        FC("fc6", 4096, out_shape=(4096, 1, 1)),
        Relu("relu6"),
        FC("fc7", 4096, out_shape=(4096, 1, 1)),
        Relu("relu7"),
        FC("fc8", 1000, out_shape=(1000, 1, 1)),
        SoftmaxCE(),
    ),
    classes=1000, lr=0.01, momentum=0.9, weight_decay=5e-4, update=True,
    description="full step: conv stack + FC 9216-4096-4096-1000 + softmax-CE + fused SGD on all params")

# The paper's full AlexNet: workload 5 with the local response normalization
# layers its GPU runs left out (Sec. 5.4.1 names them beside pooling), after
# the first two ReLUs, with AlexNet's constants in Caffe's form.
_ALEX_LRN_STACK = (_ALEX_STACK[:2] + (Lrn("norm1"),) + _ALEX_STACK[2:5] + (Lrn("norm2"),) + _ALEX_STACK[5:])

CFG6 = Workload(
    6, "AlexNet-shaped training step with LRN, batch 256, bf16 compute, fp32 master weights", "bf16", 256,
    (3, 227, 227), "normal", _ALEX_LRN_STACK + CFG5.layers[len(_ALEX_STACK):],
    classes=1000, lr=0.01, momentum=0.9, weight_decay=5e-4, update=True,
    description="workload 5 with LRN (size 5, alpha 1e-4, beta 0.75, k 1) after relu1 and relu2")

WORKLOADS = {1: CFG1, 2: CFG2, 3: CFG3, 4: CFG4, 5: CFG5, 6: CFG6}


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even (finite inputs)."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> the fp32 values they encode (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16, returned as fp32."""
    return bf16_to_f32(bf16_bits(a))


@dataclass
class LayerParams:
    name: str
    w: np.ndarray  # fp32 master, KCRS (conv) or (J, I) (FC)
    b: Optional[np.ndarray]  # fp32 or None


@dataclass
class Inputs:
    workload: Workload
    batch: int
    x: np.ndarray  # fp32 NCHW (already bf16-representable for bf16 workloads)
    params: List[LayerParams]
    labels: Optional[np.ndarray] = None  # int32 (B,)
    dy: Optional[np.ndarray] = None  # fp32 NCHW upstream gradient at the stack's output


def _draw_input(rng, dist, shape):
    if dist == "uniform01":
        return rng.uniform(0.0, 1.0, size=shape)
    if dist == "uniform11":
        return rng.uniform(-1.0, 1.0, size=shape)
    if dist == "normal":
        return rng.standard_normal(size=shape)
    raise ValueError(dist)


def stack_out_shape(wl: Workload) -> Tuple[int, int, int]:
    """Per-image (C, H, W) at the end of the stack, from the listed shapes."""
    shape = wl.in_shape
    for l in wl.layers:
        if isinstance(l, (Conv, Pool, FC)):
            shape = l.out_shape
    return shape


def make_inputs(wl: Workload, batch: Optional[int] = None, seed_offset: int = 0) -> Inputs:
    """Draw the seeded inputs of a workload (optionally at a smaller batch).

    The stream is ``default_rng(SEED_BASE + index + seed_offset)``.  With a
    batch other than the workload's, the draws differ from the full-size ones
    (the input block is smaller) but stay deterministic.
    """
    B = wl.batch if batch is None else int(batch)
    rng = np.random.default_rng(SEED_BASE + wl.index + seed_offset)
    x = _draw_input(rng, wl.input_dist, (B,) + tuple(wl.in_shape)).astype(np.float32)
    if wl.dtype == "bf16":
        x = round_bf16(x)
    params = []
    c_in, h_in, w_in = wl.in_shape
    for l in wl.layers:
        if isinstance(l, Conv):
            w = (rng.standard_normal((l.out_channels, c_in, l.kernel, l.kernel)) * 0.01).astype(np.float32)
            b = np.zeros((l.out_channels,), np.float32) if l.bias else None
            params.append(LayerParams(l.name, w, b))
        elif isinstance(l, FC):
            w = (rng.standard_normal((l.out_features, c_in * h_in * w_in)) * 0.01).astype(np.float32)
            b = np.zeros((l.out_features,), np.float32) if l.bias else None
            params.append(LayerParams(l.name, w, b))
        if isinstance(l, (Conv, Pool, FC)):
            c_in, h_in, w_in = l.out_shape
    inp = Inputs(wl, B, x, params)
    if wl.classes:
        inp.labels = rng.integers(0, wl.classes, size=(B,)).astype(np.int32)
    else:
        inp.dy = rng.standard_normal((B,) + tuple(stack_out_shape(wl))).astype(np.float32)
        if wl.dtype == "bf16":
            inp.dy = round_bf16(inp.dy)
    return inp


def random_array(shape: Sequence[int], seed: int, dist: str = "normal", scale: float = 1.0,
                 dtype: str = "f32") -> np.ndarray:
    """A seeded fp32 array for per-operator tests (bf16-representable if dtype == 'bf16')."""
    rng = np.random.default_rng(SEED_BASE + 1000 + int(seed))
    a = (_draw_input(rng, dist, tuple(shape)) * scale).astype(np.float32)
    if dtype == "bf16":
        a = round_bf16(a)
    return a
