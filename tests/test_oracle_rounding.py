"""Pins for the oracle's rounding points in the fp32 and bf16 modes, forward
AND backward, against an independent encoding of the same reading.

The reading (bf16 storage with fp32 master weights): every Linear / Conv2d
reads its input activation, its weights and the gradient arriving at its
output rounded to bf16; every tensor a pass stores (activations, activation
gradients, dW, db, the softmax-CE gradient) is fp32; accumulation is exact
(fp64 here); a residual sum adds the skip input as the layer reads it, and in
backward the gradient at the sum reaches the block input through the enclosed
layers and, rounded like any operand, through the skip, the two adding into
one stored tensor.

The reference below does not restate the oracle's backward. It builds the
forward graph in torch (float64) and places each rounding as a node:
``value_round`` rounds a value and passes gradients through unchanged (a
stored or read tensor), ``grad_round`` passes the value and rounds the
gradient flowing back through it (a gradient that is stored or read).
torch's autograd then derives the whole backward pass, and torch's own
float32 / bfloat16 conversions do the rounding (pinned separately against
hand-derived bit patterns). A slip in the oracle such as rounding dW instead
of the gradient operand, or adding the skip gradient unrounded, moves
elements by about 2^-9 relative; agreement here is to fp32 rounding of fp64
accumulation-order noise.
"""
import numpy as np
import pytest

import oracle
from paper_2408_01331_amd import workloads as W

torch = pytest.importorskip("torch")
F = torch.nn.functional
D = torch.float64


def _round(t, kind):
    if kind == "f64":
        return t
    t32 = t.to(torch.float32)
    if kind == "bf16":
        t32 = t32.to(torch.bfloat16).to(torch.float32)
    return t32.to(D)


class _ValueRound(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, kind):
        return _round(x, kind)

    @staticmethod
    def backward(ctx, g):
        return g, None


class _GradRound(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, kind):
        ctx.kind = kind
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return _round(g, ctx.kind), None


def value_round(x, kind):
    return _ValueRound.apply(x, kind)


def grad_round(x, kind):
    return _GradRound.apply(x, kind)


def reference_step(spec, params, x, y, mode):
    """Loss and gradients of one model under `mode`, by torch autograd over a
    graph with the reading's rounding nodes. Returns (loss, [grads])."""
    operand = {"f64": "f64", "f32": "f32", "bf16": "bf16"}[mode]
    store = "f64" if mode == "f64" else "f32"
    ps = [torch.tensor(np.asarray(p, dtype=np.float64), dtype=D, requires_grad=True) for p in params]
    h = torch.tensor(np.asarray(x, dtype=np.float64), dtype=D)
    layers = spec["layers"]
    pi, skip = 0, None
    for li, layer in enumerate(layers):
        op = layer[0]
        if op in ("linear", "conv"):
            W_, b_ = ps[pi], ps[pi + 1]
            hin = value_round(grad_round(h, store), operand)     # dh stored fp32; input read as operand
            Wq = value_round(W_, operand)
            z = F.linear(hin, Wq, b_) if op == "linear" else F.conv2d(hin, Wq, b_, padding=layer[3])
            z = grad_round(z, operand)                           # gradient at the output read as operand
            if li + 1 < len(layers) and layers[li + 1][0] == "res_end":
                z = z + grad_round(value_round(skip, operand), operand)
            h = value_round(z, store)                            # the stored output
            pi += 2
        elif op == "res_begin":
            h = grad_round(h, store)          # both branches' gradients sum into one stored tensor
            skip = h
        elif op == "res_end":
            skip = None
        elif op == "relu":
            h = F.relu(h)
        elif op == "pool":
            h = F.max_pool2d(h, 2, 2)
        elif op == "flatten":
            h = h.reshape(h.shape[0], -1)
    logits = grad_round(h, store)             # dL/dz stored fp32 before the last layer reads it
    loss = F.cross_entropy(logits, torch.tensor(np.asarray(y, dtype=np.int64)))
    loss.backward()
    return float(loss.detach()), [_round(p.grad, store).numpy() for p in ps]


def oracle_step(spec, params, x, y, mode):
    loss, _, grads = oracle.step(spec, params, x, y, 0.0, mode)
    return loss, grads


def _params(spec, in_shape, seed, bf16_exact=False):
    ps = W.init_params(spec, in_shape, seed, 0)
    if bf16_exact:
        ps = [oracle.to_bf16(p) for p in ps]
    return ps


def _batch(in_shape, B, C, seed):
    rng = np.random.default_rng([seed, 99])
    x = rng.standard_normal((B,) + tuple(in_shape)).astype(np.float32)
    y = rng.integers(0, C, size=B).astype(np.int32)
    return x, y


def _max_rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


L, RELU, RB, RE, POOL, FLAT = (lambda n: ("linear", n)), ("relu",), ("res_begin",), ("res_end",), ("pool",), \
    ("flatten",)
SPECS = {
    "one_layer": ({"layers": [L(7)], "num_classes": 7}, (24,)),
    "two_layers": ({"layers": [L(33), RELU, L(9)], "num_classes": 9}, (40,)),
    "deep": ({"layers": [L(48), RELU, L(31), L(20), RELU, L(6)], "num_classes": 6}, (56,)),
    "residual": ({"layers": [L(40), RELU, RB, L(25), RELU, L(40), RE, RELU, RB, L(40), RE, L(8)],
                  "num_classes": 8}, (32,)),
    "cnn": ({"layers": [("conv", 6, 3, 1), RELU, POOL, ("conv", 5, 3, 0), RELU, FLAT, L(7)],
             "num_classes": 7}, (3, 10, 10)),
    "residual_cnn": ({"layers": [("conv", 6, 3, 1), RELU, RB, ("conv", 6, 3, 1), RELU, ("conv", 6, 3, 1), RE,
                                 RELU, POOL, FLAT, L(5)], "num_classes": 5}, (2, 8, 8)),
}

# fp32 rounding of fp64 results that differ only in accumulation order: equal
# but for the rare element next to a rounding boundary
AGREE = 2.0 ** -20


@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("name", list(SPECS))
def test_oracle_backward_matches_autograd_with_rounding_nodes(name, mode):
    spec, in_shape = SPECS[name]
    params = _params(spec, in_shape, 11)
    x, y = _batch(in_shape, 13, spec["num_classes"], 5)
    lo, go = oracle_step(spec, params, x, y, mode)
    lr, gr = reference_step(spec, params, x, y, mode)
    assert abs(lo - lr) <= 1e-12 * abs(lr)
    for t, (a, b) in enumerate(zip(go, gr)):
        e = _max_rel(a, b)
        same = np.mean(np.asarray(a, np.float32).view(np.uint32) == np.asarray(b, np.float32).view(np.uint32))
        assert e <= AGREE, f"{name} {mode} tensor {t}: max rel diff {e:.3g}"
        assert same >= 0.999, f"{name} {mode} tensor {t}: only {same:.4f} of the elements bitwise equal"


@pytest.mark.parametrize("name", list(SPECS))
def test_bf16_rounding_is_visible_in_every_gradient(name):
    """The pin has teeth: the bf16 gradients differ from the f32 ones by far
    more than the agreement bound above (so a dropped or misplaced bf16 rounding
    cannot hide below it)."""
    spec, in_shape = SPECS[name]
    params = _params(spec, in_shape, 11)
    x, y = _batch(in_shape, 13, spec["num_classes"], 5)
    _, g16 = oracle_step(spec, params, x, y, "bf16")
    _, g32 = oracle_step(spec, params, x, y, "f32")
    for t, (a, b) in enumerate(zip(g16, g32)):
        assert _max_rel(a, b) > 64 * AGREE, f"{name} tensor {t}"


@pytest.mark.parametrize("name", ["one_layer", "cnn"])
def test_bf16_backward_equals_f32_on_prerounded_single_layer_operands(name):
    """With weights, input and the incoming gradient already bf16 values, the
    first layer's reads round nothing: its dW and db in bf16 mode equal the f32
    mode's bit for bit (dW itself is stored fp32, never rounded to bf16)."""
    spec, in_shape = SPECS[name]
    params = _params(spec, in_shape, 3, bf16_exact=True)
    x, _ = _batch(in_shape, 9, spec["num_classes"], 2)
    x = oracle.to_bf16(x)
    out = {}
    for mode in ("f32", "bf16"):
        logits, cache = oracle.forward(spec, params, x, mode)
        rng = np.random.default_rng(17)
        dz = oracle.to_bf16(rng.standard_normal(np.shape(logits)).astype(np.float32)).astype(np.float64)
        out[mode] = oracle.backward(spec, params, cache, dz, mode)
    if name == "one_layer":
        for a, b in zip(out["f32"], out["bf16"]):
            assert np.array_equal(np.asarray(a, np.float32).view(np.uint32), np.asarray(b, np.float32).view(np.uint32))
    else:
        # the last layer's operands are pre-rounded only where the forward
        # activations happen to be bf16 values; its bias gradient reads dz only
        assert np.array_equal(np.asarray(out["f32"][-1], np.float32), np.asarray(out["bf16"][-1], np.float32))
