"""Per-model checkpoints of a fused hybrid.

The paper's Model Separator hands each trained sub-model back on its own
(Model Separator section); a checkpoint here is one sub-model's parameters,
its optimizer state and its update count, in one safetensors file, so that a
model can be resumed - in the same hybrid, in another hybrid with different
companions, or alone.

Tensor names follow the PyTorch ``nn.Sequential`` built from the model's spec:
``"<layer index>.weight"`` / ``"<layer index>.bias"`` (the file's parameters
load into that module with ``load_state_dict``). A residual block is one
child of that Sequential, a module with an ``inner`` Sequential of the
enclosed layers whose forward returns ``inner(x) + x``: its layers are named
``"<block index>.inner.<layer index in the block>.weight"``. The optimizer state is
stored as ``"momentum_buffer.<name>"`` (SGD with momentum) or
``"exp_avg.<name>"`` / ``"exp_avg_sq.<name>"`` (Adam). The metadata holds the
spec, the input shape, the precision, the optimizer and the update count.
"""
from __future__ import annotations

import json

import numpy as np
from safetensors.numpy import load_file, save_file
from safetensors import safe_open

from . import workloads as W
from .unifiednn import split_params

STATE_NAMES = {"sgd": [], "momentum": ["momentum_buffer"], "adam": ["exp_avg", "exp_avg_sq"]}


def param_names(spec):
    """state_dict names of the parameterised layers of ``spec``, in order: the
    index of the layer in the Sequential, where a residual block (its markers
    and the layers between them) is one child holding an ``inner`` Sequential."""
    names = []
    k, j, inside = 0, 0, False
    for layer in spec["layers"]:
        op = layer[0]
        if op == "res_begin":
            inside, j = True, 0
            continue
        if op == "res_end":
            inside = False
            k += 1
            continue
        prefix = f"{k}.inner.{j}" if inside else f"{k}"
        if op in ("linear", "conv"):
            names += [f"{prefix}.weight", f"{prefix}.bias"]
        if inside:
            j += 1
        else:
            k += 1
    return names


def _tensors(spec, in_shape, flat):
    shapes = [s for s, _ in W.param_shapes(spec, in_shape)]
    return dict(zip(param_names(spec), split_params(np.asarray(flat, dtype=np.float32), shapes)))


def model_state(hybrid, i):
    """Model i's checkpoint as (tensors, metadata)."""
    spec = hybrid.specs[i]
    opt = hybrid.optimizers[i]
    in_shape = hybrid.in_shape_of(i)
    tensors = _tensors(spec, in_shape, hybrid.get_params(i))
    state, step = hybrid.get_opt_state(i)
    names = STATE_NAMES[opt["kind"]]
    n = len(state) // len(names) if names else 0
    for k, sname in enumerate(names):
        for pname, t in _tensors(spec, in_shape, state[k * n:(k + 1) * n]).items():
            tensors[f"{sname}.{pname}"] = t
    meta = {"spec": json.dumps({"layers": [list(l) for l in spec["layers"]], "num_classes": spec["num_classes"]}),
            "in_shape": json.dumps(list(in_shape)), "precision": hybrid.precision,
            "optimizer": json.dumps(opt), "step": str(int(step))}
    return {k: np.ascontiguousarray(v) for k, v in tensors.items()}, meta


def save(hybrid, i, path):
    """Write model i's parameters, optimizer state and update count to ``path``."""
    tensors, meta = model_state(hybrid, i)
    save_file(tensors, path, metadata=meta)


def read(path):
    """(tensors, metadata) of a checkpoint file (metadata fields decoded)."""
    tensors = load_file(path)
    with safe_open(path, framework="numpy") as f:
        meta = dict(f.metadata())
    meta["spec"] = json.loads(meta["spec"])
    meta["spec"]["layers"] = [tuple(l) for l in meta["spec"]["layers"]]
    meta["in_shape"] = tuple(json.loads(meta["in_shape"]))
    meta["optimizer"] = json.loads(meta["optimizer"])
    meta["step"] = int(meta["step"])
    return tensors, meta


def load(hybrid, i, path):
    """Resume model i of ``hybrid`` from ``path``: same architecture and input
    shape required. Sets the saved optimizer (fresh), then the parameters,
    then the optimizer state and update count."""
    tensors, meta = read(path)
    spec = hybrid.specs[i]
    if [tuple(l) for l in spec["layers"]] != meta["spec"]["layers"] or spec["num_classes"] != meta["spec"]["num_classes"]:
        raise ValueError(f"checkpoint {path} holds a different architecture than model {i}")
    if tuple(hybrid.in_shape_of(i)) != meta["in_shape"]:
        raise ValueError(f"checkpoint {path} was trained on input shape {meta['in_shape']}")
    opt = meta["optimizer"]
    hybrid.set_optimizer(i, opt["kind"], opt["momentum"], tuple(opt["betas"]), opt["eps"])
    names = param_names(spec)
    hybrid.set_params(i, np.concatenate([tensors[n].ravel() for n in names]))
    state = [tensors[f"{s}.{n}"].ravel() for s in STATE_NAMES[opt["kind"]] for n in names]
    hybrid.set_opt_state(i, np.concatenate(state) if state else np.zeros(0, np.float32), meta["step"])
