"""Thin Python binding of libunifiednn.so (the C ABI in include/unifiednn.h).

Argument marshalling only: every step of the training path runs in the
library's HIP kernels. The functions keep the C names (un_create, un_load_batch,
un_step, un_get_params, ...); `Hybrid` wraps them in a small class.

Importing this module fails loudly if the library has not been built: there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libunifiednn.so")

UN_OK, UN_ERR_INVALID, UN_ERR_STATE, UN_ERR_OOM, UN_ERR_DEVICE, UN_ERR_RANGE, UN_ERR_BUFSIZE, UN_ERR_UNSUPPORTED = range(8)
STATUS_NAMES = ["UN_OK", "UN_ERR_INVALID", "UN_ERR_STATE", "UN_ERR_OOM", "UN_ERR_DEVICE", "UN_ERR_RANGE",
                "UN_ERR_BUFSIZE", "UN_ERR_UNSUPPORTED"]
UN_F32, UN_BF16_F32MASTER = 0, 1
UN_OPT_SGD, UN_OPT_MOMENTUM, UN_OPT_ADAM = 0, 1, 2
OPT_KINDS = {"sgd": UN_OPT_SGD, "momentum": UN_OPT_MOMENTUM, "adam": UN_OPT_ADAM}
OPS = {"linear": 0, "conv": 1, "relu": 2, "pool": 3, "flatten": 4, "res_begin": 5, "res_end": 6, "unflatten": 7,
       "attention": 8}
KERNEL_CLASSES = ["gemm_fwd", "gemm_bwd", "conv_fwd", "conv_dgrad", "conv_wgrad", "ce", "sgd", "other", "attn"]

# Every symbol the header declares.
EXPORTS = ["un_create", "un_create_grouped", "un_plan_bytes", "un_plan_bytes_grouped", "un_load_group_batch",
           "un_load_batch", "un_load_batch_device", "un_load_labels", "un_step", "un_step_lr",
           "un_set_active", "un_set_optimizer", "un_get_opt_state", "un_set_opt_state", "un_get_params",
           "un_set_params", "un_get_grads", "un_keep_grads", "un_param_count", "un_arena_bytes", "un_sync", "un_get_stream",
           "un_set_stream", "un_graph_capture", "un_graph_step", "un_step_scratch",
           "un_profile_enable", "un_profile_read", "un_destroy", "un_last_error"]


class un_layer(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("out", ctypes.c_int32), ("kernel", ctypes.c_int32), ("pad", ctypes.c_int32)]


class un_model_spec(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("layers", ctypes.POINTER(un_layer)),
                ("num_classes", ctypes.c_int32), ("init_seed", ctypes.c_uint64)]


class un_input_spec(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32),
                ("in_w", ctypes.c_int32), ("precision", ctypes.c_int32)]


class un_optimizer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("momentum", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps", ctypes.c_float)]


class UnError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES[status] if 0 <= status < 8 else status}: {msg}")
        self.status = status


_lib = None


def lib():
    """Load libunifiednn.so (raises if it is missing: build it first)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2408_01331_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, c_size_p = ctypes.c_void_p, ctypes.POINTER(ctypes.c_size_t)
        f = ctypes.POINTER(ctypes.c_float)
        i32 = ctypes.POINTER(ctypes.c_int32)
        sig = {
            "un_create": (ctypes.c_int, [ctypes.POINTER(un_model_spec), ctypes.c_int32, ctypes.POINTER(un_input_spec),
                                         ctypes.POINTER(P)]),
            "un_create_grouped": (ctypes.c_int, [ctypes.POINTER(un_model_spec), ctypes.c_int32,
                                                 ctypes.POINTER(un_input_spec), ctypes.c_int32, i32, ctypes.POINTER(P)]),
            "un_plan_bytes_grouped": (ctypes.c_int, [ctypes.POINTER(un_model_spec), ctypes.c_int32,
                                                     ctypes.POINTER(un_input_spec), ctypes.c_int32, i32, c_size_p,
                                                     c_size_p]),
            "un_load_group_batch": (ctypes.c_int, [P, ctypes.c_int32, f, i32]),
            "un_load_batch": (ctypes.c_int, [P, f, i32]),
            "un_load_batch_device": (ctypes.c_int, [P, P, P]),
            "un_step": (ctypes.c_int, [P, ctypes.c_float, f]),
            "un_step_lr": (ctypes.c_int, [P, f, f]),
            "un_plan_bytes": (ctypes.c_int, [ctypes.POINTER(un_model_spec), ctypes.c_int32,
                                             ctypes.POINTER(un_input_spec), c_size_p, c_size_p]),
            "un_set_optimizer": (ctypes.c_int, [P, ctypes.c_int32, ctypes.POINTER(un_optimizer)]),
            "un_get_opt_state": (ctypes.c_int, [P, ctypes.c_int32, f, ctypes.c_size_t, c_size_p,
                                                ctypes.POINTER(ctypes.c_int64)]),
            "un_set_opt_state": (ctypes.c_int, [P, ctypes.c_int32, f, ctypes.c_size_t, ctypes.c_int64]),
            "un_load_labels": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_int32)]),
            "un_set_active": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_uint8)]),
            "un_get_params": (ctypes.c_int, [P, ctypes.c_int32, f, ctypes.c_size_t, c_size_p]),
            "un_set_params": (ctypes.c_int, [P, ctypes.c_int32, f, ctypes.c_size_t]),
            "un_get_grads": (ctypes.c_int, [P, ctypes.c_int32, f, ctypes.c_size_t, c_size_p]),
            "un_keep_grads": (ctypes.c_int, [P, ctypes.c_int32]),
            "un_param_count": (ctypes.c_int, [P, ctypes.c_int32, c_size_p]),
            "un_arena_bytes": (ctypes.c_int, [P, c_size_p]),
            "un_sync": (ctypes.c_int, [P]),
            "un_get_stream": (ctypes.c_int, [P, ctypes.POINTER(P)]),
            "un_set_stream": (ctypes.c_int, [P, P]),
            "un_graph_capture": (ctypes.c_int, [P, ctypes.c_float]),
            "un_graph_step": (ctypes.c_int, [P, f]),
            "un_step_scratch": (ctypes.c_int, [P, ctypes.c_float, f]),
            "un_profile_enable": (ctypes.c_int, [P, ctypes.c_int32]),
            "un_profile_read": (ctypes.c_int, [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                               ctypes.POINTER(ctypes.c_int64)]),
            "un_destroy": (None, [P]),
            "un_last_error": (ctypes.c_char_p, [P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _fp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _check(status, ctx=None):
    if status != UN_OK:
        msg = lib().un_last_error(ctx)
        raise UnError(status, msg.decode() if msg else "")


# ---------------------------------------------------------------------------
# C-named functions
# ---------------------------------------------------------------------------
def make_specs(specs, seeds=None):
    """Python spec dicts -> (array of un_model_spec, keep-alive list)."""
    keep = []
    arr = (un_model_spec * len(specs))()
    for i, s in enumerate(specs):
        layers = (un_layer * len(s["layers"]))()
        for j, l in enumerate(s["layers"]):
            op = OPS[l[0]]
            out = l[1] if len(l) > 1 else 0
            k = l[2] if op == 1 else 0
            pad = l[3] if op == 1 else 0
            layers[j] = un_layer(op, out, k, pad)
        keep.append(layers)
        arr[i] = un_model_spec(len(s["layers"]), layers, s["num_classes"], 0 if seeds is None else seeds[i])
    return arr, keep


def _input_spec(batch, in_shape, precision):
    c, h, w = (tuple(in_shape) + (1, 1))[:3] if len(in_shape) != 3 else tuple(in_shape)
    return un_input_spec(batch, c, h, w, UN_BF16_F32MASTER if precision == "bf16" else UN_F32)


def _groups(specs, batch, in_shape, precision, inputs, group_of):
    """(input spec array, n_groups, group_of int32 array or None)."""
    if inputs is None:
        return (un_input_spec * 1)(_input_spec(batch, in_shape, precision)), 1, None
    arr = (un_input_spec * len(inputs))(*[_input_spec(b, sh, precision) for b, sh in inputs])
    go = np.ascontiguousarray(group_of, dtype=np.int32)
    if go.shape != (len(specs),):
        raise ValueError(f"group_of needs one entry per model ({len(specs)})")
    return arr, len(inputs), go


def un_create(specs, batch, in_shape, precision, seeds=None, inputs=None, group_of=None):
    """A context; with inputs = [(batch, in_shape) per input group] and
    group_of (a group per model) it is un_create_grouped."""
    arr, keep = make_specs(specs, seeds)
    ins, ng, go = _groups(specs, batch, in_shape, precision, inputs, group_of)
    ctx = ctypes.c_void_p()
    if go is None:
        _check(lib().un_create(arr, len(specs), ins, ctypes.byref(ctx)))
    else:
        _check(lib().un_create_grouped(arr, len(specs), ins, ng, go.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                       ctypes.byref(ctx)))
    return ctx


def un_plan_bytes(specs, batch, in_shape, precision, inputs=None, group_of=None):
    """(arena bytes, optimizer-state bytes) a context for these models would
    take; host only (no device needed)."""
    arr, keep = make_specs(specs, None)
    ins, ng, go = _groups(specs, batch, in_shape, precision, inputs, group_of)
    a, st = ctypes.c_size_t(), ctypes.c_size_t()
    if go is None:
        _check(lib().un_plan_bytes(arr, len(specs), ins, ctypes.byref(a), ctypes.byref(st)))
    else:
        _check(lib().un_plan_bytes_grouped(arr, len(specs), ins, ng, go.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                           ctypes.byref(a), ctypes.byref(st)))
    return a.value, st.value


def un_load_batch(ctx, x, y):
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    _check(lib().un_load_batch(ctx, _fp(x), y.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))), ctx)


def un_load_group_batch(ctx, g, x, y):
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    _check(lib().un_load_group_batch(ctx, g, _fp(x), y.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))), ctx)


def un_load_batch_device(ctx, x_ptr, y_ptr):
    _check(lib().un_load_batch_device(ctx, ctypes.c_void_p(x_ptr), ctypes.c_void_p(y_ptr)), ctx)


def un_load_labels(ctx, y, batches):
    """Per-model labels for the loaded batches: y[i] holds batches[i] labels
    of model i (a [N][B] array when every model has batch B)."""
    rows = [np.ascontiguousarray(r, dtype=np.int32).reshape(-1) for r in y]
    if [r.size for r in rows] != list(batches):
        raise ValueError(f"label rows must have lengths {list(batches)}, got {[r.size for r in rows]}")
    flat = np.ascontiguousarray(np.concatenate(rows), dtype=np.int32)
    _check(lib().un_load_labels(ctx, flat.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))), ctx)


def un_step_lr(ctx, lrs, n_models, losses=True):
    """One fused step with a learning rate per model; returns the losses unless losses=False."""
    lr = np.ascontiguousarray(lrs, dtype=np.float32)
    if lr.shape != (n_models,):
        raise ValueError(f"one learning rate per model ({n_models}) expected, got shape {lr.shape}")
    if not losses:
        _check(lib().un_step_lr(ctx, _fp(lr), None), ctx)
        return None
    out = np.zeros(n_models, dtype=np.float32)
    _check(lib().un_step_lr(ctx, _fp(lr), _fp(out)), ctx)
    return out


def un_step(ctx, lr, n_models=None):
    """One fused step; returns the per-model losses if n_models is given, else enqueues only."""
    if n_models is None:
        _check(lib().un_step(ctx, ctypes.c_float(lr), None), ctx)
        return None
    out = np.zeros(n_models, dtype=np.float32)
    _check(lib().un_step(ctx, ctypes.c_float(lr), _fp(out)), ctx)
    return out


def un_set_active(ctx, mask, n_models):
    m = np.ascontiguousarray(np.asarray(mask, dtype=bool), dtype=np.uint8)
    if m.shape != (n_models,):
        raise ValueError(f"mask must have one entry per model ({n_models}), got shape {m.shape}")
    _check(lib().un_set_active(ctx, m.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))), ctx)


def un_param_count(ctx, i):
    n = ctypes.c_size_t()
    _check(lib().un_param_count(ctx, i, ctypes.byref(n)), ctx)
    return n.value


def un_get_params(ctx, i):
    n = un_param_count(ctx, i)
    out = np.empty(n, dtype=np.float32)
    got = ctypes.c_size_t()
    _check(lib().un_get_params(ctx, i, _fp(out), n, ctypes.byref(got)), ctx)
    return out


def un_get_grads(ctx, i):
    n = un_param_count(ctx, i)
    out = np.empty(n, dtype=np.float32)
    got = ctypes.c_size_t()
    _check(lib().un_get_grads(ctx, i, _fp(out), n, ctypes.byref(got)), ctx)
    return out


def un_set_optimizer(ctx, i, kind="sgd", momentum=0.0, betas=(0.9, 0.999), eps=1e-8):
    if kind not in OPT_KINDS:
        raise ValueError(f"optimizer kind must be one of {sorted(OPT_KINDS)}")
    o = un_optimizer(OPT_KINDS[kind], float(momentum), float(betas[0]), float(betas[1]), float(eps))
    _check(lib().un_set_optimizer(ctx, i, ctypes.byref(o)), ctx)


def un_get_opt_state(ctx, i):
    """(flat fp32 state [k * n_params], update count) of model i's optimizer."""
    n = ctypes.c_size_t()
    step = ctypes.c_int64()
    _check(lib().un_get_opt_state(ctx, i, None, 0, ctypes.byref(n), ctypes.byref(step)), ctx)
    out = np.empty(n.value, dtype=np.float32)
    if n.value:
        _check(lib().un_get_opt_state(ctx, i, _fp(out), n.value, ctypes.byref(n), ctypes.byref(step)), ctx)
    return out, int(step.value)


def un_set_opt_state(ctx, i, state, step):
    state = np.ascontiguousarray(state, dtype=np.float32).reshape(-1)
    _check(lib().un_set_opt_state(ctx, i, _fp(state) if state.size else None, state.size, int(step)), ctx)


def un_keep_grads(ctx, on):
    _check(lib().un_keep_grads(ctx, 1 if on else 0), ctx)


def un_set_params(ctx, i, flat):
    flat = np.ascontiguousarray(flat, dtype=np.float32)
    _check(lib().un_set_params(ctx, i, _fp(flat), flat.size), ctx)


def un_sync(ctx):
    _check(lib().un_sync(ctx), ctx)


def un_get_stream(ctx):
    s = ctypes.c_void_p()
    _check(lib().un_get_stream(ctx, ctypes.byref(s)), ctx)
    return s.value


def un_step_scratch(ctx, lr, n_models=None):
    """un_step with the step's workspace in the library's static scratch
    array (no allocation); returns the losses if n_models is given."""
    if n_models is None:
        _check(lib().un_step_scratch(ctx, ctypes.c_float(lr), None), ctx)
        return None
    out = np.zeros(n_models, dtype=np.float32)
    _check(lib().un_step_scratch(ctx, ctypes.c_float(lr), _fp(out)), ctx)
    return out


def un_set_stream(ctx, stream):
    """Run the context's work on `stream` (a hipStream_t as an int, e.g.
    torch.cuda.Stream().cuda_stream); None returns to the context's own."""
    _check(lib().un_set_stream(ctx, ctypes.c_void_p(stream) if stream else None), ctx)


def un_graph_capture(ctx, lr):
    _check(lib().un_graph_capture(ctx, ctypes.c_float(lr)), ctx)


def un_graph_step(ctx, n_models=None):
    """Replay the captured step; returns the losses if n_models is given."""
    if n_models is None:
        _check(lib().un_graph_step(ctx, None), ctx)
        return None
    out = np.zeros(n_models, dtype=np.float32)
    _check(lib().un_graph_step(ctx, _fp(out)), ctx)
    return out


def un_arena_bytes(ctx):
    n = ctypes.c_size_t()
    _check(lib().un_arena_bytes(ctx, ctypes.byref(n)), ctx)
    return n.value


def un_profile_enable(ctx, on):
    _check(lib().un_profile_enable(ctx, 1 if on else 0), ctx)


def un_profile_read(ctx, kclass):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().un_profile_read(ctx, kclass, ctypes.byref(ms), ctypes.byref(n)), ctx)
    return ms.value, n.value


def un_destroy(ctx):
    if ctx:
        lib().un_destroy(ctx)


# ---------------------------------------------------------------------------
# Convenience wrapper
# ---------------------------------------------------------------------------
def flatten_params(params):
    return np.concatenate([np.asarray(p, dtype=np.float32).ravel() for p in params])


def split_params(flat, shapes):
    out, o = [], 0
    for s in shapes:
        n = int(np.prod(s))
        out.append(flat[o:o + n].reshape(s))
        o += n
    return out


class Hybrid:
    """N models merged into one fused training step on the GPU."""

    def __init__(self, specs, batch, in_shape, precision="f32", seeds=None, inputs=None, group_of=None):
        """One shared input [batch, *in_shape], or input groups: inputs =
        [(batch, in_shape) per group] and group_of = the group of each model."""
        self.specs = list(specs)
        self.n = len(self.specs)
        self.precision = precision
        self.inputs = None if inputs is None else [(int(b), tuple(sh)) for b, sh in inputs]
        self.group_of = None if group_of is None else [int(g) for g in group_of]
        self.ctx = None
        self.ctx = un_create(self.specs, batch, in_shape, precision, seeds, self.inputs, self.group_of)
        if self.inputs is None:
            self.batch = int(batch)
            self.in_shape = tuple(in_shape)
            self.batches = [self.batch] * self.n
        else:
            self.batch, self.in_shape = None, None
            self.batches = [self.inputs[g][0] for g in self.group_of]
        self.optimizers = {i: dict(kind="sgd", momentum=0.0, betas=[0.9, 0.999], eps=1e-8) for i in range(self.n)}

    def close(self):
        if self.ctx:
            un_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load_batch(self, x, y, group=None):
        """The shared batch, or input group `group`'s batch."""
        if group is None:
            un_load_batch(self.ctx, x, y)
        else:
            un_load_group_batch(self.ctx, group, x, y)

    def step(self, lr, losses=True):
        """lr: one rate for every model, or a sequence of N per-model rates."""
        if np.ndim(lr) == 0:
            return un_step(self.ctx, lr, self.n if losses else None)
        return un_step_lr(self.ctx, lr, self.n, losses)

    def in_shape_of(self, i):
        """Model i's input sample shape (its input group's)."""
        return self.in_shape if self.inputs is None else self.inputs[self.group_of[i]][1]

    def load_labels(self, y):
        un_load_labels(self.ctx, y, self.batches)

    def set_active(self, mask):
        un_set_active(self.ctx, mask, self.n)

    def get_params(self, i):
        return un_get_params(self.ctx, i)

    def set_params(self, i, flat):
        un_set_params(self.ctx, i, flat)

    def get_grads(self, i):
        return un_get_grads(self.ctx, i)

    def set_optimizer(self, i, kind="sgd", momentum=0.0, betas=(0.9, 0.999), eps=1e-8):
        """Fresh optimizer for model i ("sgd", "momentum" or "adam")."""
        un_set_optimizer(self.ctx, i, kind, momentum, betas, eps)
        self.optimizers[i] = dict(kind=kind, momentum=float(momentum), betas=[float(b) for b in betas],
                                  eps=float(eps))

    def get_opt_state(self, i):
        return un_get_opt_state(self.ctx, i)

    def set_opt_state(self, i, state, step):
        un_set_opt_state(self.ctx, i, state, step)

    def keep_grads(self, on=True):
        un_keep_grads(self.ctx, on)

    def capture(self, lr):
        """Capture one step at rate lr as a HIP graph (un_graph_capture)."""
        un_graph_capture(self.ctx, lr)

    def replay(self, losses=True):
        """One step by replaying the captured graph (un_graph_step)."""
        return un_graph_step(self.ctx, self.n if losses else None)

    def set_stream(self, stream):
        un_set_stream(self.ctx, stream)

    def sync(self):
        un_sync(self.ctx)
