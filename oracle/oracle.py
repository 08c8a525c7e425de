"""CPU oracle for one UnifiedNN training step -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module. The library's compute path never reaches it.

What it computes (UnifiedNN, Trainer section, Algorithm 2): for every
sub-model m, the gradient of m's own loss on the batch, then the plain SGD
update theta^m <- theta^m - eta * g^m. Each sub-model has its own criterion and
optimizer and no sub-model interferes with another (Model Unifier section), so
the oracle trains every model ALONE: nothing here ever reads another model's
parameters, and the merged run must equal these separate runs (the paper's
claim that the hybrid trains each sub-model exactly as separate training would,
Design overview).

Every function below is the plain definition of its operation, written with
numpy in float64. Readings where the paper is silent (all taken to match the
paper's PyTorch prototype, whose defaults these are):

* loss: softmax cross-entropy, mean over the batch;
* optimizer: plain SGD, no momentum or weight decay, computed as the
  correctly rounded fp32 fma(-lr, g, theta); each sub-model may instead have
  SGD with momentum or Adam (its own optimizer, Model Unifier section), with
  torch.optim's definitions (momentum_update, adam_update);
* gradients are recomputed every step (nothing accumulates across steps);
* the loss a step reports is the forward loss at the pre-update parameters;
* convolution is cross-correlation, stride 1, zero padding;
* max-pool is 2x2 / stride 2 / floor mode, the first maximum in row-major
  window order wins ties; ReLU'(0) = 0;
* flatten is NCHW (c, h, w) order, and a sequence [T, d] flattens token by
  token (t, j); ``unflatten`` views the flat features as a sequence of T
  tokens of F / T features (PyTorch's Unflatten), on which a Linear layer
  acts token by token;
* ``attention`` is single-head self-attention on a sequence, PyTorch's
  MultiheadAttention with one head (no mask, no dropout): [Q K V] =
  x W_in^T + b_in (in-projection [3d, d]), A = softmax(Q K^T / sqrt(d)) V,
  y = A W_out^T + b_out; its parameters are in_proj_weight, in_proj_bias,
  out_proj.weight, out_proj.bias;
* a residual block (``res_begin`` ... ``res_end``) is a module returning
  inner(x) + x, the standard skip connection: the sum is formed before any
  ReLU that follows the block, and in backward the gradient at the sum flows
  both through the enclosed layers and unchanged to x, where the two add.

Precision modes:

* ``"f64"``  no rounding at all (used for finite-difference checks);
* ``"f32"``  every dot product accumulates in fp64 and is rounded to fp32 when
  stored;
* ``"bf16"`` as f32, and in addition the operands of every Linear/Conv layer
  (its input activation, its weights, and the gradient arriving at its output)
  are rounded to bf16 (round to nearest, ties to even) when read. Logits, the
  softmax-CE arithmetic, all accumulators, dW, db and the fp32 master weights
  stay fp32. Because ReLU, max-pool, flatten and their backward passes are
  exact, rounding at the reader equals rounding the stored tensor. In an
  attention layer the two projections are Linear layers; the core reads Q, K,
  V and the gradient dA at its output as bf16 operands, keeps the scores S and
  the probabilities P in fp32 (both modes), and stores A and dQKV (read as
  operands by the projections).

Accumulation (``acc``): ``"f64"`` (the default, the reference) sums every dot
product exactly enough to be rounded once; ``"f32"`` evaluates the same
products and the softmax cross-entropy in fp32 arithmetic (float32 BLAS, its
own summation order). Both are evaluation orders the reading allows, and
their difference measures how far two correct implementations of the same
step may legitimately lie apart.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64
F32 = np.float32


# ---------------------------------------------------------------------------
# Rounding
# ---------------------------------------------------------------------------
def to_f32(a):
    """Round to nearest fp32 (IEEE conversion)."""
    return np.asarray(a, dtype=F64).astype(F32)


def to_bf16(a):
    """Round an fp32 array to bf16 (nearest, ties to even), returned as fp32 values.

    bf16 keeps the top 16 bits of the fp32 pattern; adding 0x7FFF plus the lowest
    kept bit before truncation rounds to nearest with ties to the even pattern.
    NaNs stay NaN (quiet bit forced so truncation cannot turn them into inf).
    """
    a = np.ascontiguousarray(np.asarray(a, dtype=F32))
    u = a.view(np.uint32)
    r = u + np.uint32(0x7FFF)            # wraps only for NaN patterns, which are replaced below
    r += (u >> np.uint32(16)) & np.uint32(1)
    r &= np.uint32(0xFFFF0000)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = (u[nan] | np.uint32(0x00400000)) & np.uint32(0xFFFF0000)
    return r.view(F32).reshape(a.shape)


def fma32(a, b, c):
    """Correctly rounded fp32 a*b + c for fp32 arrays.

    a*b is exact in fp64 (24+24 bits). s = fl64(a*b + c) has exact error e
    (TwoSum). Rounding s to fp32 is then correct unless s lies exactly on an fp32
    midpoint, in which case the sign of e decides the direction.
    """
    a64 = np.asarray(a, dtype=F32).astype(F64)
    b64 = np.asarray(b, dtype=F32).astype(F64)
    c64 = np.asarray(c, dtype=F32).astype(F64)
    p = a64 * b64
    s = p + c64
    bb = s - p
    e = (p - (s - bb)) + (c64 - bb)
    r = s.astype(F32)
    d = s - r.astype(F64)
    toward = np.where(d > 0, np.inf, -np.inf).astype(F32)
    nb = np.nextafter(r, toward)
    midpoint = (d != 0) & (2.0 * d == nb.astype(F64) - r.astype(F64))
    go_nb = midpoint & (e != 0) & (np.sign(e) == np.sign(d))
    return np.where(go_nb, nb, r).astype(F32)


class _Mode:
    def __init__(self, mode, acc="f64"):
        if mode not in ("f64", "f32", "bf16"):
            raise ValueError(f"unknown precision mode {mode!r}")
        if acc not in ("f64", "f32"):
            raise ValueError(f"unknown accumulation {acc!r}")
        self.mode = mode
        self.acc = acc

    def run(self, fn, *arrays, **kw):
        """A layer function on fp64 arrays, or in fp32 arithmetic when acc is "f32"."""
        if self.acc == "f64":
            return fn(*arrays, **kw)
        out = fn(*[a.astype(F32) if isinstance(a, np.ndarray) else a for a in arrays], **kw)
        if isinstance(out, tuple):
            return tuple(None if o is None else np.asarray(o, dtype=F64) for o in out)
        return np.asarray(out, dtype=F64)

    def operand(self, a):
        """A tensor as a Linear/Conv layer reads it (activation, weight or gradient)."""
        if self.mode == "f64":
            return np.asarray(a, dtype=F64)
        a32 = to_f32(a)
        if self.mode == "bf16":
            a32 = to_bf16(a32)
        return a32.astype(F64)

    def store(self, a):
        """The result of an fp64 accumulation as it is stored."""
        if self.mode == "f64":
            return np.asarray(a, dtype=F64)
        return to_f32(a).astype(F64)


# ---------------------------------------------------------------------------
# Layers (definitions)
# ---------------------------------------------------------------------------
def linear_fwd(h, W, b):
    """z = h W^T + b  (PyTorch Linear; W is [out, in])."""
    return h @ W.T + b


def linear_bwd(dz, h, W, need_dh=True):
    """dW = dz^T h, db = sum_b dz, dh = dz W. On a sequence [B, T, d] the layer
    acts on every token (PyTorch's Linear on a 3-D input): dW and db sum over
    every sample and token."""
    d2, h2 = dz.reshape(-1, dz.shape[-1]), h.reshape(-1, h.shape[-1])
    dW = d2.T @ h2
    db = d2.sum(axis=0)
    dh = dz @ W if need_dh else None
    return dW, db, dh


def attention_core_fwd(q, k, v, rnd=lambda t: t):
    """Scaled dot-product attention of one head over a sequence, per sample:
    S = Q K^T / sqrt(d), P = softmax(S) over the keys, A = P V (q, k, v:
    [B, T, d]). `rnd` rounds S and P as they are stored. Returns (A, P)."""
    d = q.shape[-1]
    s = rnd((q @ np.swapaxes(k, -1, -2)) / np.sqrt(d))
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    p = rnd(e / e.sum(axis=-1, keepdims=True))
    return p @ v, p


def attention_core_bwd(da, q, k, v, p):
    """Gradients of A = softmax(Q K^T / sqrt(d)) V: dP = dA V^T, dV = P^T dA,
    dS = P * (dP - rowsum(P * dP)) (softmax's Jacobian), dQ = dS K / sqrt(d),
    dK = dS^T Q / sqrt(d). Returns (dQ, dK, dV)."""
    d = q.shape[-1]
    dp = da @ np.swapaxes(v, -1, -2)
    dv = np.swapaxes(p, -1, -2) @ da
    ds = p * (dp - (p * dp).sum(axis=-1, keepdims=True))
    dq = (ds @ k) / np.sqrt(d)
    dk = (np.swapaxes(ds, -1, -2) @ q) / np.sqrt(d)
    return dq, dk, dv


def conv2d_fwd(h, W, b, pad):
    """z[n,o,p,q] = b[o] + sum_{c,u,v} W[o,c,u,v] * h[n,c,p+u-pad,q+v-pad]; outside reads are 0.

    Written as the sum over the k*k kernel taps of a channel contraction.
    """
    n, c, H, Wd = h.shape
    o, c2, k, k2 = W.shape
    assert c == c2 and k == k2
    OH, OW = H + 2 * pad - k + 1, Wd + 2 * pad - k + 1
    hp = np.pad(h, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    z = np.zeros((n, OH, OW, o), dtype=F64)
    for u in range(k):
        for v in range(k):
            win = hp[:, :, u:u + OH, v:v + OW]                     # [n, c, OH, OW]
            z += np.tensordot(win, W[:, :, u, v], axes=([1], [1]))  # [n, OH, OW, o]
    return z.transpose(0, 3, 1, 2) + b[None, :, None, None]


def conv2d_bwd(dz, h, W, pad, need_dh=True):
    """dW[o,c,u,v] = sum_{n,p,q} dz[n,o,p,q] h[n,c,p+u-pad,q+v-pad];  db[o] = sum dz[n,o,:,:];
    dh[n,c,y,x] = sum_{o,u,v} dz[n,o,y-u+pad,x-v+pad] W[o,c,u,v]."""
    n, c, H, Wd = h.shape
    o, _, k, _ = W.shape
    OH, OW = dz.shape[2], dz.shape[3]
    hp = np.pad(h, ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    dW = np.zeros(W.shape, dtype=F64)
    dhp = np.zeros(hp.shape, dtype=F64) if need_dh else None
    for u in range(k):
        for v in range(k):
            win = hp[:, :, u:u + OH, v:v + OW]
            dW[:, :, u, v] = np.tensordot(dz, win, axes=([0, 2, 3], [0, 2, 3]))
            if need_dh:
                t = np.tensordot(dz, W[:, :, u, v], axes=([1], [0]))   # [n, OH, OW, c]
                dhp[:, :, u:u + OH, v:v + OW] += t.transpose(0, 3, 1, 2)
    db = dz.sum(axis=(0, 2, 3))
    dh = dhp[:, :, pad:pad + H, pad:pad + Wd] if need_dh else None
    return dW, db, dh


def relu_fwd(z):
    return np.maximum(z, 0.0)


def relu_bwd(dy, y):
    """ReLU' taken from the output: 1 where the output is > 0, else 0 (so ReLU'(0) = 0)."""
    return dy * (y > 0)


def maxpool2_fwd(h):
    """2x2 / stride 2 / floor max-pool. Returns (out, argmax in 0..3 = dy*2+dx).

    Ties go to the first maximum in row-major window order (numpy's argmax
    returns the first occurrence).
    """
    n, c, H, Wd = h.shape
    PH, PW = H // 2, Wd // 2
    win = h[:, :, :2 * PH, :2 * PW].reshape(n, c, PH, 2, PW, 2)
    win = win.transpose(0, 1, 2, 4, 3, 5).reshape(n, c, PH, PW, 4)
    am = np.argmax(win, axis=-1)
    out = np.take_along_axis(win, am[..., None], axis=-1)[..., 0]
    return out, am


def maxpool2_bwd(dout, am, in_shape):
    """Route each pooled gradient to its window's argmax; everything else gets 0."""
    n, c, H, Wd = in_shape
    PH, PW = dout.shape[2], dout.shape[3]
    win = np.zeros(dout.shape + (4,), dtype=F64)
    np.put_along_axis(win, am[..., None], np.asarray(dout, dtype=F64)[..., None], axis=-1)
    g = win.reshape(n, c, PH, PW, 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(n, c, 2 * PH, 2 * PW)
    dh = np.zeros(in_shape, dtype=F64)
    dh[:, :, :2 * PH, :2 * PW] = g
    return dh


def softmax_ce(z, y, dtype=F64):
    """Mean softmax cross-entropy and its gradient.

    L = (1/B) sum_b (lse(z_b) - z_{b,y_b}), lse(z) = m + log sum exp(z - m);
    dL/dz = (softmax(z) - onehot(y)) / B. `dtype` is the arithmetic (float64,
    or float32 for the fp32 evaluation order); the gradient is returned in
    float64 either way.
    """
    z = np.asarray(z, dtype=dtype)
    B = z.shape[0]
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(s[:, 0])
    rows = np.arange(B)
    loss = float(np.mean(lse - z[rows, y]))
    p = e / s
    p[rows, y] -= 1.0
    return loss, np.asarray(p / dtype(B), dtype=F64)


# ---------------------------------------------------------------------------
# One model, alone
# ---------------------------------------------------------------------------
def count_params(spec, in_shape):
    """Parameter count by walking the layer list (oracle's own shape inference)."""
    shape = tuple(in_shape)
    total = 0
    for layer in spec["layers"]:
        op = layer[0]
        if op == "linear":
            fin = shape[-1] if len(shape) == 2 else int(np.prod(shape))
            total += layer[1] * fin + layer[1]
            shape = (shape[0], layer[1]) if len(shape) == 2 else (layer[1],)
        elif op == "conv":
            c, H, W = shape
            o, k, pad = layer[1], layer[2], layer[3]
            total += o * c * k * k + o
            shape = (o, H + 2 * pad - k + 1, W + 2 * pad - k + 1)
        elif op == "pool":
            c, H, W = shape
            shape = (c, H // 2, W // 2)
        elif op == "flatten":
            shape = (int(np.prod(shape)),)
        elif op == "unflatten":
            shape = (layer[1], shape[0] // layer[1])
        elif op == "attention":
            d = shape[-1]
            total += 4 * d * d + 4 * d
        elif op not in ("relu", "res_begin", "res_end"):
            raise ValueError(f"unknown op {op!r}")
    return total


# Unit roundoff of fp32.
U32 = 2.0 ** -24


def forward(spec, params, x, mode="f32", flags=None, acc="f64"):
    """Forward pass. Returns (logits as stored, cache for backward).

    If `flags` (a dict) is given, it receives, per parameterised layer (keyed by
    the index of its weight in `params`), the set of output units (features or
    channels) for which a discrete decision of this pass is ill-conditioned in
    fp32: a ReLU input with |z| <= u * (sum_k |h_k w_k| + |b|), or a max-pool
    window whose two largest values differ by no more than that, u = 2^-24.
    Such a decision may legitimately come out either way in any fp32
    evaluation order; everything else is decided identically.
    """
    R = _Mode(mode, acc)
    h = np.asarray(x, dtype=F64)
    cache = []
    pi = 0
    mag, last_pi = None, None
    layers = spec["layers"]
    skip = None  # input of the open residual block
    for li, layer in enumerate(layers):
        op = layer[0]
        if op == "linear":
            W, b = params[pi], params[pi + 1]
            hin, Wq = R.operand(h), R.operand(W)
            if hin.ndim not in (2, 3):
                raise ValueError("linear layer needs flat features or a sequence (add a flatten)")
            z = R.run(linear_fwd, hin, Wq, np.asarray(b, dtype=F64))
            ends_block = li + 1 < len(layers) and layers[li + 1][0] == "res_end"
            if ends_block:
                # the residual sum is the stored tensor: x joins before rounding
                if skip is None or skip.shape != z.shape:
                    raise ValueError("residual block: missing begin or feature mismatch")
                z = z + R.operand(skip)
            h = R.store(z)
            if flags is not None:
                mag, last_pi = linear_fwd(np.abs(hin), np.abs(Wq), np.abs(np.asarray(b, dtype=F64))), pi
                if ends_block:
                    mag = mag + np.abs(R.operand(skip))
            cache.append(("linear", pi, hin, Wq))
            pi += 2
        elif op == "res_begin":
            if skip is not None:
                raise ValueError("nested residual blocks")
            skip = h
            cache.append(("res_begin",))
        elif op == "res_end":
            if skip is None or layers[li - 1][0] not in ("linear", "conv", "attention"):
                raise ValueError("residual end must directly follow the block's last linear, conv or attention")
            skip = None
            cache.append(("res_end",))
        elif op == "conv":
            W, b = params[pi], params[pi + 1]
            hin, Wq = R.operand(h), R.operand(W)
            z = R.run(conv2d_fwd, hin, Wq, np.asarray(b, dtype=F64), layer[3])
            ends_block = li + 1 < len(layers) and layers[li + 1][0] == "res_end"
            if ends_block:
                if skip is None or skip.shape != z.shape:
                    raise ValueError("residual block: missing begin or shape mismatch")
                z = z + R.operand(skip)
            h = R.store(z)
            if flags is not None:
                mag = conv2d_fwd(np.abs(hin), np.abs(Wq), np.abs(np.asarray(b, dtype=F64)), layer[3])
                if ends_block:
                    mag = mag + np.abs(R.operand(skip))
                last_pi = pi
            cache.append(("conv", pi, hin, Wq, layer[3]))
            pi += 2
        elif op == "relu":
            if flags is not None and mag is not None:
                bad = np.abs(h) <= U32 * mag
                axes = (0,) if h.ndim == 2 else (0, 1) if h.ndim == 3 else (0, 2, 3)
                flags.setdefault(last_pi, set()).update(np.nonzero(bad.any(axis=axes))[0].tolist())
            h = relu_fwd(h)
            cache.append(("relu", h))
        elif op == "pool":
            shp = h.shape
            if flags is not None and mag is not None:
                n, c, H, Wd = shp
                PH, PW = H // 2, Wd // 2
                win = h[:, :, :2 * PH, :2 * PW].reshape(n, c, PH, 2, PW, 2).transpose(0, 1, 2, 4, 3, 5)
                wm = mag[:, :, :2 * PH, :2 * PW].reshape(n, c, PH, 2, PW, 2).transpose(0, 1, 2, 4, 3, 5)
                win = win.reshape(n, c, PH, PW, 4)
                top2 = np.sort(win, axis=-1)[..., 2:]
                tol = U32 * wm.reshape(n, c, PH, PW, 4).max(axis=-1)
                # exact zero ties (ReLU outputs) are decided identically everywhere
                bad = (top2[..., 1] - top2[..., 0] <= tol) & ~((top2[..., 1] == 0) & (top2[..., 0] == 0))
                flags.setdefault(last_pi, set()).update(np.nonzero(bad.any(axis=(0, 2, 3)))[0].tolist())
            h, am = maxpool2_fwd(h)
            mag = None if mag is None else maxpool2_fwd(mag)[0]
            cache.append(("pool", am, shp))
        elif op == "flatten":
            cache.append(("flatten", h.shape))
            h = h.reshape(h.shape[0], -1)
        elif op == "unflatten":
            if h.ndim != 2 or h.shape[1] % layer[1]:
                raise ValueError("unflatten needs flat features divisible into the tokens")
            cache.append(("flatten", h.shape))
            h = h.reshape(h.shape[0], layer[1], -1)
        elif op == "attention":
            if h.ndim != 3:
                raise ValueError("attention needs a sequence (add an unflatten)")
            Wi, bi, Wo, bo = params[pi:pi + 4]
            hin, Wiq, Woq = R.operand(h), R.operand(Wi), R.operand(Wo)
            d = hin.shape[2]
            qkv = R.store(R.run(linear_fwd, hin, Wiq, np.asarray(bi, dtype=F64)))
            q, k, v = (R.operand(qkv[..., j * d:(j + 1) * d]) for j in range(3))
            a, p = R.run(attention_core_fwd, q, k, v, R.store)
            aq = R.operand(R.store(a))
            z = R.run(linear_fwd, aq, Woq, np.asarray(bo, dtype=F64))
            ends_block = li + 1 < len(layers) and layers[li + 1][0] == "res_end"
            if ends_block:
                if skip is None or skip.shape != z.shape:
                    raise ValueError("residual block: missing begin or shape mismatch")
                z = z + R.operand(skip)
            h = R.store(z)
            if flags is not None:
                mag, last_pi = linear_fwd(np.abs(aq), np.abs(Woq), np.abs(np.asarray(bo, dtype=F64))), pi + 2
                if ends_block:
                    mag = mag + np.abs(R.operand(skip))
            cache.append(("attention", pi, hin, Wiq, q, k, v, p, aq, Woq))
            pi += 4
        else:
            raise ValueError(f"unknown op {op!r}")
    return h, cache


def backward(spec, params, cache, dlogits, mode="f32", acc="f64"):
    """Backward pass from dL/dlogits. Returns the gradient list (state-dict order)."""
    R = _Mode(mode, acc)
    grads = [None] * len(params)
    g = np.asarray(dlogits, dtype=F64)
    first_param_layer = min(e[1] for e in cache if e[0] in ("linear", "conv", "attention"))
    gskip = None  # gradient at the sum of the open residual block
    for entry in reversed(cache):
        kind = entry[0]
        if kind == "res_end":
            gskip = g
            continue
        if kind == "res_begin":
            # both paths reach the block's input: the enclosed layers' and the
            # skip (a block opened at the network input needs no input gradient)
            g = None if g is None else R.store(g + R.operand(gskip))
            gskip = None
            continue
        if kind in ("linear", "conv"):
            pi, hin, Wq = entry[1], entry[2], entry[3]
            gq = R.operand(g)
            need_dh = pi != first_param_layer
            if kind == "linear":
                dW, db, dh = R.run(linear_bwd, gq, hin, Wq, need_dh)
            else:
                dW, db, dh = R.run(conv2d_bwd, gq, hin, Wq, entry[4], need_dh)
            grads[pi], grads[pi + 1] = R.store(dW), R.store(db)
            g = R.store(dh) if need_dh else None
        elif kind == "attention":
            pi, hin, Wiq, q, k, v, p, aq, Woq = entry[1:]
            gq = R.operand(g)
            dWo, dbo, da = R.run(linear_bwd, gq, aq, Woq, True)
            grads[pi + 2], grads[pi + 3] = R.store(dWo), R.store(dbo)
            dq, dk, dv = R.run(attention_core_bwd, R.operand(R.store(da)), q, k, v, p)
            gqi = R.operand(R.store(np.concatenate([dq, dk, dv], axis=-1)))
            need_dh = pi != first_param_layer
            dWi, dbi, dh = R.run(linear_bwd, gqi, hin, Wiq, need_dh)
            grads[pi], grads[pi + 1] = R.store(dWi), R.store(dbi)
            g = R.store(dh) if need_dh else None
        elif kind == "relu":
            if g is not None:
                g = relu_bwd(g, entry[1])
        elif kind == "pool":
            if g is not None:
                g = maxpool2_bwd(g, entry[1], entry[2])
        elif kind == "flatten":
            if g is not None:
                g = g.reshape(entry[1])
    return grads


def sgd_update(params, grads, lr, mode="f32"):
    """theta <- theta - lr * g  (Algorithm 2's update), as fp32 fma(-lr, g, theta)."""
    if mode == "f64":
        return [np.asarray(p, dtype=F64) - lr * np.asarray(g, dtype=F64) for p, g in zip(params, grads)]
    nlr = np.full((), -lr, dtype=F32)
    return [fma32(nlr, to_f32(g), p) for p, g in zip(params, grads)]


def momentum_update(params, grads, bufs, lr, momentum, mode="f32"):
    """SGD with momentum (the per-model optimizer option; torch.optim.SGD's
    definition without dampening, weight decay or Nesterov):
    b <- momentum * b + g,  theta <- theta - lr * b, with b = 0 before the first
    step. Returns (new params, new buffers). In the fp32 modes every stored
    value (b, theta) is the fp32 rounding of its exact value from fp32 inputs."""
    out_p, out_b = [], []
    for p, g, b in zip(params, grads, bufs):
        p64, g64, b64 = (np.asarray(a, dtype=F64) for a in (p, g, b))
        nb = momentum * b64 + g64
        if mode != "f64":
            nb = to_f32(nb).astype(F64)
        npar = p64 - lr * nb
        out_b.append(nb if mode == "f64" else to_f32(nb))
        out_p.append(npar if mode == "f64" else to_f32(npar))
    return out_p, out_b


def adam_update(params, grads, m, v, t, lr, beta1, beta2, eps, mode="f32"):
    """Adam (torch.optim.Adam's definition without weight decay or amsgrad),
    update number t >= 1:
    m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2;
    theta <- theta - (lr / (1 - beta1^t)) m / (sqrt(v) / sqrt(1 - beta2^t) + eps).
    Returns (new params, new m, new v); rounding as in momentum_update."""
    bc1 = 1.0 - beta1 ** t
    bc2 = 1.0 - beta2 ** t
    out_p, out_m, out_v = [], [], []
    for p, g, mm, vv in zip(params, grads, m, v):
        p64, g64, m64, v64 = (np.asarray(a, dtype=F64) for a in (p, g, mm, vv))
        nm = beta1 * m64 + (1.0 - beta1) * g64
        nv = beta2 * v64 + (1.0 - beta2) * g64 * g64
        if mode != "f64":
            nm = to_f32(nm).astype(F64)
            nv = to_f32(nv).astype(F64)
        npar = p64 - (lr / bc1) * nm / (np.sqrt(nv) / np.sqrt(bc2) + eps)
        out_m.append(nm if mode == "f64" else to_f32(nm))
        out_v.append(nv if mode == "f64" else to_f32(nv))
        out_p.append(npar if mode == "f64" else to_f32(npar))
    return out_p, out_m, out_v


def step_opt(spec, params, x, y, lr, opt, state, mode="f32", flags=None, acc="f64"):
    """One training step of one model under its optimizer.

    opt: {"kind": "sgd" | "momentum" | "adam", "momentum", "betas", "eps"};
    state: {"t": updates taken, "s1": [...], "s2": [...]} (zeros / absent at
    the start). Returns (loss, new params, grads, new state)."""
    logits, cache = forward(spec, params, x, mode, flags, acc)
    loss, dz = softmax_ce(logits, y, F64 if acc == "f64" else F32)
    dz = _Mode(mode).store(dz)
    grads = backward(spec, params, cache, dz, mode, acc)
    zeros = [np.zeros(np.shape(p), dtype=F64 if mode == "f64" else F32) for p in params]
    t = state.get("t", 0) + 1
    kind = opt["kind"]
    if kind == "sgd":
        return loss, sgd_update(params, grads, lr, mode), grads, {"t": t}
    if kind == "momentum":
        newp, b = momentum_update(params, grads, state.get("s1", zeros), lr, opt["momentum"], mode)
        return loss, newp, grads, {"t": t, "s1": b}
    b1, b2 = opt["betas"]
    newp, m, v = adam_update(params, grads, state.get("s1", zeros), state.get("s2", zeros), t, lr, b1, b2,
                             opt["eps"], mode)
    return loss, newp, grads, {"t": t, "s1": m, "s2": v}


def step(spec, params, x, y, lr, mode="f32", flags=None, acc="f64"):
    """One training step of one model. Returns (loss at pre-update params, new params, grads)."""
    logits, cache = forward(spec, params, x, mode, flags, acc)
    loss, dz = softmax_ce(logits, y, F64 if acc == "f64" else F32)
    dz = _Mode(mode).store(dz)
    grads = backward(spec, params, cache, dz, mode, acc)
    return loss, sgd_update(params, grads, lr, mode), grads


def loss_only(spec, params, x, y, mode="f64"):
    logits, _ = forward(spec, params, x, mode)
    return softmax_ce(logits, y)[0]


def train(spec, params, batches, lr, mode="f32", flags=None, acc="f64"):
    """Train one model alone over a sequence of (x, y) batches.

    Returns (losses per step, final params, grads of the last step). `flags`
    (optional dict) collects the ill-conditioned decisions of every step.
    """
    losses = []
    grads = None
    params = [np.array(p, dtype=F64 if mode == "f64" else F32) for p in params]
    for x, y in batches:
        loss, params, grads = step(spec, params, x, y, lr, mode, flags, acc)
        losses.append(loss)
    return np.array(losses), params, grads


def train_models(specs, theta0s, batches, lr, mode="f32", models=None, with_flags=False):
    """Train each listed model alone, one after another.

    Models are never run in concurrent Python threads: concurrent calls into
    the BLAS library from several threads gave run-to-run different results.

    Returns {model: (losses, params, grads)} or, with with_flags, (losses,
    params, grads, flags)."""
    idx = list(range(len(specs))) if models is None else list(models)
    batches = list(batches)
    out = {}
    for i in idx:
        if with_flags:
            fl = {}
            out[i] = train(specs[i], theta0s[i], batches, lr, mode, fl) + (fl,)
        else:
            out[i] = train(specs[i], theta0s[i], batches, lr, mode)
    return out
