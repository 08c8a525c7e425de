"""Seeded synthetic workloads: model specs, initial parameters and batches.

This module only *generates inputs*. It holds none of the training method's
arithmetic (no forward, loss, gradient or update), so both the GPU path and the
CPU oracle can draw their inputs from it without sharing any computation.

Random streams (numpy PCG64, one stream per purpose so that changing one
workload knob never shifts another's numbers):

* architecture draws  ``default_rng([seed, 0])``
* initial parameters  ``default_rng([seed, 1, i])`` for model ``i``
* data of step ``s``  ``default_rng([seed, 2, s])``

Inputs are x ~ N(0, 1) and labels uniform over the classes. They stand in for
the MNIST-shaped (1x28x28, 10 classes) and CIFAR-shaped (3x32x32) datasets of
the paper's evaluation (Evaluation setup, Table 2), which are not available.

A model spec is a plain dict: ``{"layers": [...], "num_classes": C}``. Each
layer is a tuple whose first item is the op name, mirroring a PyTorch
``nn.Sequential`` (the paper defines every sub-model as a sequential module,
Design overview):

* ``("linear", out)``
* ``("conv", out, kernel, pad)``   stride 1, square kernel
* ``("relu",)``
* ``("pool",)``                    2x2 max-pool, stride 2, floor mode
* ``("flatten",)``                 NCHW flatten order
* ``("res_begin",)`` ... ``("res_end",)``  a residual block: the enclosed
  layers' result plus the block's input (a module returning
  ``inner(x) + x``); a ReLU after ``res_end`` applies to the sum
* ``("unflatten", T)``             flat features as T tokens (a sequence); a
  following ``linear`` acts on every token
* ``("attention",)``               single-head self-attention on a sequence
"""
from __future__ import annotations

import json
import math
from dataclasses import dataclass, field

import numpy as np

OP_CODES = {"linear": 0, "conv": 1, "relu": 2, "pool": 3, "flatten": 4, "res_begin": 5, "res_end": 6,
            "unflatten": 7, "attention": 8}


@dataclass
class Workload:
    name: str
    n_models: int
    batch: int
    in_shape: tuple          # (F,) for an MLP input, (C, H, W) for an image input
    precision: str           # "f32" or "bf16" (bf16 storage, fp32 master weights)
    specs: list              # one spec dict per model
    lr: float
    steps: int               # steps the parity run takes
    seed: int = 0
    description: str = ""
    extra: dict = field(default_factory=dict)
    init: str = "kaiming"    # weight init rule of init_params

    @property
    def num_classes(self):
        return self.specs[0]["num_classes"]

    def to_json(self):
        d = dict(name=self.name, n_models=self.n_models, batch=self.batch,
                 in_shape=list(self.in_shape), precision=self.precision,
                 lr=self.lr, steps=self.steps, seed=self.seed,
                 specs=[{"layers": [list(l) for l in s["layers"]],
                         "num_classes": s["num_classes"]} for s in self.specs])
        return json.dumps(d)


# ---------------------------------------------------------------------------
# Parameter shapes. This is an input-side shape walk used only to size the
# initial parameters (fan-in for the init bounds); the oracle and the library
# each have their own.
# ---------------------------------------------------------------------------
def param_shapes(spec, in_shape):
    """Return [(shape, fan_in), ...] in state-dict order (weight then bias)."""
    shape = tuple(in_shape)
    out = []
    for layer in spec["layers"]:
        op = layer[0]
        if op == "linear":
            seq = len(shape) == 2          # a sequence [T, d]: the layer acts on every token
            f_in = shape[-1] if seq else int(np.prod(shape))
            out.append(((layer[1], f_in), f_in))
            out.append(((layer[1],), f_in))
            shape = (shape[0], layer[1]) if seq else (layer[1],)
        elif op == "conv":
            c, h, w = shape
            o, k, pad = layer[1], layer[2], layer[3]
            f_in = c * k * k
            out.append(((o, c, k, k), f_in))
            out.append(((o,), f_in))
            shape = (o, h + 2 * pad - k + 1, w + 2 * pad - k + 1)
        elif op == "pool":
            c, h, w = shape
            shape = (c, h // 2, w // 2)
        elif op == "flatten":
            shape = (int(np.prod(shape)),)
        elif op == "unflatten":
            shape = (layer[1], shape[0] // layer[1])
        elif op == "attention":
            d = shape[-1]
            out += [((3 * d, d), d), ((3 * d,), d), ((d, d), d), ((d,), d)]
    return out


def init_params(spec, in_shape, seed, model_index, rule="kaiming"):
    """Initial parameters, fp32: biases U(+-1/sqrt(fan_in)); weights
    U(+-sqrt(6/fan_in)) (Kaiming/He uniform, rule "kaiming") or U(+-1/sqrt(fan_in))
    (rule "torch", the bound of PyTorch's own Linear / Conv2d initialisation)."""
    if rule not in ("kaiming", "torch"):
        raise ValueError(f"unknown init rule {rule!r}")
    rng = np.random.default_rng([seed, 1, model_index])
    params = []
    for shape, fan_in in param_shapes(spec, in_shape):
        wbound = math.sqrt(6.0 / fan_in) if rule == "kaiming" else 1.0 / math.sqrt(fan_in)
        bound = wbound if len(shape) > 1 else 1.0 / math.sqrt(fan_in)
        params.append(rng.uniform(-bound, bound, size=shape).astype(np.float32))
    return params


def make_batch(wl: Workload, step: int):
    """The shared batch of one step: x fp32 [B, *in_shape], y int32 [B]."""
    rng = np.random.default_rng([wl.seed, 2, step])
    x = rng.standard_normal((wl.batch,) + tuple(wl.in_shape), dtype=np.float32)
    y = rng.integers(0, wl.num_classes, size=wl.batch).astype(np.int32)
    return x, y


# ---------------------------------------------------------------------------
# The workloads.
# ---------------------------------------------------------------------------
def _mlp(widths, classes):
    layers = []
    for w in widths:
        layers += [("linear", int(w)), ("relu",)]
    layers.append(("linear", int(classes)))
    return {"layers": layers, "num_classes": int(classes)}


def mlp2_tiny(seed=0):
    """N=2 MLPs 784-128-10 and 784-64-10, fp32, batch 64."""
    specs = [_mlp([128], 10), _mlp([64], 10)]
    return Workload("mlp2_b64_f32", 2, 64, (784,), "f32", specs, 0.01, 10, seed,
                    "2 MLPs 784-{128,64}-10 on a shared fp32 [64,784] input")


def mlp8_hetero(seed=0):
    """N=8 MLPs, 1-2 hidden layers with widths from {128,256,512}, fp32, batch 256."""
    rng = np.random.default_rng([seed, 0])
    specs = []
    for _ in range(8):
        depth = int(rng.integers(1, 3))
        widths = rng.choice([128, 256, 512], size=depth)
        specs.append(_mlp(widths, 10))
    return Workload("mlp8_b256_f32", 8, 256, (784,), "f32", specs, 0.01, 20, seed,
                    "8 heterogeneous MLPs (1-2 hidden, widths {128,256,512}) on [256,784] fp32")


def lenet4(seed=0):
    """N=4 LeNet-5-style CNNs on 1x28x28, first-conv channels from {6,8,12}, fp32, batch 128."""
    rng = np.random.default_rng([seed, 0])
    specs = []
    for _ in range(4):
        c1 = int(rng.choice([6, 8, 12]))
        layers = [("conv", c1, 5, 0), ("relu",), ("pool",),
                  ("conv", 16, 5, 0), ("relu",), ("pool",), ("flatten",),
                  ("linear", 120), ("relu",), ("linear", 84), ("relu",), ("linear", 10)]
        specs.append({"layers": layers, "num_classes": 10})
    return Workload("lenet4_b128_f32", 4, 128, (1, 28, 28), "f32", specs, 0.01, 10, seed,
                    "4 LeNet-5 CNNs (conv1 channels {6,8,12}) on [128,1,28,28] fp32")


def cifar16(seed=0):
    """N=16 CIFAR CNNs: 3 x (conv3x3 pad1 + ReLU + pool2), then fc-10; bf16 with fp32 master."""
    rng = np.random.default_rng([seed, 0])
    specs = []
    for _ in range(16):
        c1 = int(rng.choice([32, 48, 64]))
        c2 = int(rng.choice([64, 96, 128]))
        c3 = int(rng.choice([128, 192, 256]))
        layers = [("conv", c1, 3, 1), ("relu",), ("pool",),
                  ("conv", c2, 3, 1), ("relu",), ("pool",),
                  ("conv", c3, 3, 1), ("relu",), ("pool",), ("flatten",),
                  ("linear", 10)]
        specs.append({"layers": layers, "num_classes": 10})
    return Workload("cifar16_b256_bf16", 16, 256, (3, 32, 32), "bf16", specs, 0.01, 5, seed,
                    "16 CIFAR CNNs (3 conv blocks, widths {32,48,64}/{64,96,128}/{128,192,256}) "
                    "on [256,3,32,32], bf16 with fp32 master")


def mlp64_ragged(seed=0):
    """N=64 MLPs on [512,1024]: 2-6 Linear layers, widths log-uniform on [64, 2048], 100 classes."""
    rng = np.random.default_rng([seed, 0])
    specs = []
    lo, hi = math.log(64.0), math.log(2048.0)
    for _ in range(64):
        n_linear = int(rng.integers(2, 7))
        widths = [min(2048, max(64, int(math.floor(math.exp(rng.uniform(lo, hi))))))
                  for _ in range(n_linear - 1)]
        specs.append(_mlp(widths, 100))
    return Workload("mlp64_b512_bf16", 64, 512, (1024,), "bf16", specs, 0.01, 5, seed,
                    "64 ragged MLPs (2-6 Linear, widths log-U[64,2048], 100 classes) "
                    "on [512,1024], bf16 with fp32 master")


WORKLOADS = {
    "mlp2": mlp2_tiny,
    "mlp8": mlp8_hetero,
    "lenet4": lenet4,
    "cifar16": cifar16,
    "mlp64": mlp64_ragged,
}


def resnet8(seed=0):
    """N=8 small residual CNNs (ResNet-style: two-conv blocks with identity skips,
    and one residual Linear block in the head) on 3x32x32, base widths from
    {16, 32}, bf16, batch 64."""
    rng = np.random.default_rng([seed, 4])
    RB, RE, R = ("res_begin",), ("res_end",), ("relu",)
    specs = []
    for _ in range(8):
        c = int(rng.choice([16, 32]))
        h = int(rng.choice([64, 128]))
        layers = [("conv", c, 3, 1), R, ("pool",),
                  RB, ("conv", c, 3, 1), R, ("conv", c, 3, 1), RE, R,
                  ("conv", 2 * c, 3, 1), R, ("pool",),
                  RB, ("conv", 2 * c, 3, 1), R, ("conv", 2 * c, 3, 1), RE, R,
                  ("conv", 2 * c, 3, 1), R, ("pool",), ("flatten",),
                  ("linear", h), R, RB, ("linear", h), R, ("linear", h), RE, R, ("linear", 10)]
        specs.append({"layers": layers, "num_classes": 10})
    # PyTorch's default bound: with Kaiming-uniform weights these unnormalised
    # residual nets start at a loss of 11-34 (logits up to 55) and train
    # chaotically in bf16 (a 1-ulp change of the parameters moves the loss by
    # 2 % within four steps); with this bound they start near ln 10.
    return Workload("resnet8_b64_bf16", 8, 64, (3, 32, 32), "bf16", specs, 0.01, 10, seed,
                    "8 residual CNNs (two-conv identity blocks, widths {16,32}/{32,64}) on [64,3,32,32], bf16",
                    init="torch")


WORKLOADS["resnet8"] = resnet8


def attn8(seed=0):
    """N=8 transformer-style classifiers on synthetic token sequences: the
    input [128, 2048] is 32 tokens of 64 features; each model embeds the
    tokens (token-wise Linear to a width from {64, 128}), then 1-2 blocks of
    [residual self-attention, residual token-wise MLP of twice the width],
    then a token-wise Linear to 16, flatten and Linear-10. bf16 with fp32
    master weights. Stands in for the paper's Transformer / XLM-R models
    (Evaluation setup, Table 2), whose datasets are not available."""
    rng = np.random.default_rng([seed, 5])
    T, d0 = 32, 64
    RB, RE, R = ("res_begin",), ("res_end",), ("relu",)
    specs = []
    for _ in range(8):
        width = int(rng.choice([64, 128]))
        blocks = int(rng.integers(1, 3))
        layers = [("unflatten", T), ("linear", width), R]
        for _ in range(blocks):
            layers += [RB, ("attention",), RE, R, RB, ("linear", 2 * width), R, ("linear", width), RE, R]
        layers += [("linear", 16), R, ("flatten",), ("linear", 10)]
        specs.append({"layers": layers, "num_classes": 10})
    return Workload("attn8_b128_bf16", 8, 128, (T * d0,), "bf16", specs, 0.01, 5, seed,
                    "8 transformer-style classifiers (32 tokens x 64 features, 1-2 residual attention + MLP blocks, "
                    "widths {64,128}) on [128,2048], bf16 with fp32 master", init="torch")


WORKLOADS["attn8"] = attn8


def get(name, seed=0) -> Workload:
    return WORKLOADS[name](seed)


def shrink(wl: Workload, n_models=None, batch=None) -> Workload:
    """Same architecture draws on fewer models or a smaller batch (for quick parity cases)."""
    specs = wl.specs if n_models is None else wl.specs[:n_models]
    return Workload(wl.name + "_small", len(specs), batch or wl.batch, wl.in_shape,
                    wl.precision, specs, wl.lr, wl.steps, wl.seed, wl.description, init=wl.init)
