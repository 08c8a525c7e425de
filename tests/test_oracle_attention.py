"""Pins for the oracle's sequence layers: ``unflatten``, token-wise Linear and
single-head self-attention (the attention family of the paper's transformer
models, Evaluation setup, Table 2).

* forward, float64, against torch: nn.Unflatten, nn.Linear on [B, T, d],
  nn.MultiheadAttention(d, 1 head, batch_first) called as attn(x, x, x),
  a residual wrapper x + attn(x), nn.Flatten;
* gradients against central finite differences of the float64 loss;
* the fp32 / bf16 rounding points, forward and backward, against torch
  autograd over a graph with rounding nodes (as test_oracle_rounding does for
  Linear and Conv2d);
* parameter counts against the torch modules.
"""
import numpy as np
import pytest

import oracle
from paper_2408_01331_amd import workloads as W
from test_oracle_rounding import _GradRound, _ValueRound, _round, grad_round, value_round

torch = pytest.importorskip("torch")
F = torch.nn.functional
D = torch.float64

U, A, L, RELU, FLAT, RB, RE = (lambda t: ("unflatten", t)), ("attention",), (lambda n: ("linear", n)), ("relu",), \
    ("flatten",), ("res_begin",), ("res_end",)
SPECS = {
    "attn": ({"layers": [U(6), A, FLAT, L(5)], "num_classes": 5}, (6 * 8,)),
    "embed_attn": ({"layers": [U(5), L(12), RELU, A, RELU, L(7), FLAT, L(4)], "num_classes": 4}, (5 * 6,)),
    "residual_attn": ({"layers": [U(4), L(8), RB, A, RE, RELU, RB, L(8), RELU, L(8), RE, FLAT, L(3)],
                       "num_classes": 3}, (4 * 5,)),
    "two_attn": ({"layers": [U(7), A, RB, A, RE, FLAT, L(6)], "num_classes": 6}, (7 * 4,)),
    # residual blocks opened at the network input (flat, and read as a sequence)
    "input_skip": ({"layers": [RB, L(6), RE, RELU, L(3)], "num_classes": 3}, (6,)),
    "input_skip_attn": ({"layers": [U(3), RB, A, RE, FLAT, L(3)], "num_classes": 3}, (3 * 4,)),
}


class _Residual(torch.nn.Module):
    def __init__(self, inner):
        super().__init__()
        self.inner = inner

    def forward(self, x):
        return self.inner(x) + x


class _SelfAttention(torch.nn.Module):
    def __init__(self, d):
        super().__init__()
        self.mha = torch.nn.MultiheadAttention(d, 1, batch_first=True, dtype=D)

    def forward(self, x):
        return self.mha(x, x, x, need_weights=False)[0]


def _torch_model(spec, in_shape, params):
    """The torch module of the spec, holding the given parameters."""
    mods, stack, shape = [], [], tuple(in_shape)
    for layer in spec["layers"]:
        op = layer[0]
        if op == "res_begin":
            stack.append(mods)
            mods = []
        elif op == "res_end":
            inner = torch.nn.Sequential(*mods)
            mods = stack.pop()
            mods.append(_Residual(inner))
        elif op == "unflatten":
            mods.append(torch.nn.Unflatten(1, (layer[1], shape[0] // layer[1])))
            shape = (layer[1], shape[0] // layer[1])
        elif op == "linear":
            fin = shape[-1]
            mods.append(torch.nn.Linear(fin, layer[1], dtype=D))
            shape = shape[:-1] + (layer[1],)
        elif op == "attention":
            mods.append(_SelfAttention(shape[-1]))
        elif op == "relu":
            mods.append(torch.nn.ReLU())
        elif op == "flatten":
            mods.append(torch.nn.Flatten())
            shape = (int(np.prod(shape)),)
    model = torch.nn.Sequential(*mods)
    with torch.no_grad():
        for tp, p in zip(model.parameters(), params):
            tp.copy_(torch.tensor(np.asarray(p, np.float64)).reshape(tp.shape))
    return model


def _setup(name, seed=3, B=5):
    spec, in_shape = SPECS[name]
    params = [p.astype(np.float64) for p in W.init_params(spec, in_shape, seed, 0, "torch")]
    rng = np.random.default_rng([seed, 5])
    x = rng.standard_normal((B,) + tuple(in_shape))
    y = rng.integers(0, spec["num_classes"], size=B)
    return spec, in_shape, params, x, y


@pytest.mark.parametrize("name", list(SPECS))
def test_param_count_and_order_match_torch(name):
    spec, in_shape, params, _, _ = _setup(name)
    model = _torch_model(spec, in_shape, params)
    tshapes = [tuple(p.shape) for p in model.parameters()]
    assert tshapes == [s for s, _ in W.param_shapes(spec, in_shape)]
    assert oracle.count_params(spec, in_shape) == sum(int(np.prod(s)) for s in tshapes)


@pytest.mark.parametrize("name", list(SPECS))
def test_forward_matches_torch_modules(name):
    spec, in_shape, params, x, _ = _setup(name)
    model = _torch_model(spec, in_shape, params)
    ref = model(torch.tensor(x)).detach().numpy()
    got, _ = oracle.forward(spec, params, x, "f64")
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("name", list(SPECS))
def test_gradients_match_central_differences(name):
    spec, in_shape, params, x, y = _setup(name, B=3)
    _, _, grads = oracle.step(spec, params, x, y, 0.0, "f64")
    rng = np.random.default_rng(11)
    eps = 1e-6
    for t, p in enumerate(params):
        for _ in range(4):
            idx = tuple(rng.integers(0, n) for n in p.shape)
            plus = [q.copy() for q in params]
            minus = [q.copy() for q in params]
            plus[t][idx] += eps
            minus[t][idx] -= eps
            fd = (oracle.loss_only(spec, plus, x, y) - oracle.loss_only(spec, minus, x, y)) / (2 * eps)
            g = grads[t][idx]
            assert abs(fd - g) <= 1e-7 * max(1.0, abs(fd)) + 1e-8 * np.max(np.abs(grads[t])), (name, t, idx, fd, g)


class _StoredSoftmax(torch.autograd.Function):
    """P = softmax(S) stored in `kind`; the backward uses the stored P (the
    Jacobian of softmax, P * (dP - rowsum(P * dP)))."""

    @staticmethod
    def forward(ctx, s, kind):
        p = _round(torch.softmax(s, dim=-1), kind)
        ctx.save_for_backward(p)
        return p

    @staticmethod
    def backward(ctx, dp):
        (p,) = ctx.saved_tensors
        return p * (dp - (p * dp).sum(dim=-1, keepdim=True)), None


def reference_step(spec, params, x, y, mode):
    """Loss and gradients by torch autograd with the reading's rounding nodes
    (see test_oracle_rounding); the attention core: Q, K, V read as operands,
    S and P stored fp32, A stored and read as an operand by the out-projection,
    dA and dQKV stored and read as operands."""
    operand = mode
    store = "f64" if mode == "f64" else "f32"
    ps = [torch.tensor(np.asarray(p, dtype=np.float64), dtype=D, requires_grad=True) for p in params]
    h = torch.tensor(np.asarray(x, dtype=np.float64), dtype=D)
    layers = spec["layers"]
    pi, skips = 0, []
    for li, layer in enumerate(layers):
        op = layer[0]
        ends = li + 1 < len(layers) and layers[li + 1][0] == "res_end"
        if op == "linear":
            hin = value_round(grad_round(h, store), operand)
            z = grad_round(F.linear(hin, value_round(ps[pi], operand), ps[pi + 1]), operand)
            if ends:
                z = z + grad_round(value_round(skips[-1], operand), operand)
            h = value_round(z, store)
            pi += 2
        elif op == "attention":
            Wi, bi, Wo, bo = ps[pi:pi + 4]
            d = h.shape[-1]
            hin = value_round(grad_round(h, store), operand)
            qkv = F.linear(hin, value_round(Wi, operand), bi)
            qkv = value_round(grad_round(grad_round(qkv, operand), store), store)
            q, k, v = (value_round(qkv[..., j * d:(j + 1) * d], operand) for j in range(3))
            s = value_round((q @ k.transpose(-1, -2)) / np.sqrt(d), store)
            p = _StoredSoftmax.apply(s, store)
            a = grad_round(grad_round(p @ v, operand), store)
            aq = value_round(value_round(a, store), operand)
            z = grad_round(F.linear(aq, value_round(Wo, operand), bo), operand)
            if ends:
                z = z + grad_round(value_round(skips[-1], operand), operand)
            h = value_round(z, store)
            pi += 4
        elif op == "res_begin":
            h = grad_round(h, store)
            skips.append(h)
        elif op == "res_end":
            skips.pop()
        elif op == "relu":
            h = F.relu(h)
        elif op == "flatten":
            h = h.reshape(h.shape[0], -1)
        elif op == "unflatten":
            h = h.reshape(h.shape[0], layer[1], -1)
    logits = grad_round(h, store)
    loss = F.cross_entropy(logits, torch.tensor(np.asarray(y, dtype=np.int64)))
    loss.backward()
    return float(loss.detach()), [_round(p.grad, store).numpy() for p in ps]


@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("name", list(SPECS))
def test_rounding_points_match_autograd_with_rounding_nodes(name, mode):
    spec, in_shape, params, x, y = _setup(name, B=6)
    params = [p.astype(np.float32) for p in params]
    x = x.astype(np.float32)
    lo, _, go = oracle.step(spec, params, x, y, 0.0, mode)
    lr, gr = reference_step(spec, params, x, y, mode)
    assert abs(lo - lr) <= 1e-12 * abs(lr)
    for t, (a, b) in enumerate(zip(go, gr)):
        a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
        e = np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)
        assert e <= 2.0 ** -20, f"{name} {mode} tensor {t}: {e:.3g}"


def test_bf16_rounding_is_visible_in_attention_gradients():
    spec, in_shape, params, x, y = _setup("two_attn", B=6)
    _, _, g16 = oracle.step(spec, params, x, y, 0.0, "bf16")
    _, _, g32 = oracle.step(spec, params, x, y, 0.0, "f32")
    for t, (a, b) in enumerate(zip(g16, g32)):
        e = np.max(np.abs(np.asarray(a) - b)) / np.max(np.abs(b))
        assert e > 64 * 2.0 ** -20, t
