"""Pins for the CPU oracle: it is checked against things other than itself.

* library routines: torch's bf16 conversion, scipy's 2-D correlation,
  logsumexp and softmax, Python's exact rationals;
* closed forms: ln C for zero logits, multinomial logistic regression's
  gradient, the adjoint identity of convolution;
* central finite differences of the fp64 loss on tiny models;
* hand-built max-pool windows (ties) and parameter counts printed in the paper.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.signal
import scipy.special

import oracle
from paper_2408_01331_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# bf16 rounding and the fp32 fma
# ---------------------------------------------------------------------------
def _bits(u32):
    return np.array(u32, dtype=np.uint32).view(np.float32)


def _bf16_bits(f32):
    return (np.asarray(f32, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint32)


@pytest.mark.parametrize("pattern,expect", [
    (0x3F800000, 0x3F80),   # 1.0 exact
    (0x3F807FFF, 0x3F80),   # just below half an ulp: down
    (0x3F808000, 0x3F80),   # exactly half, kept bit even: down
    (0x3F808001, 0x3F81),   # just above half: up
    (0x3F818000, 0x3F82),   # exactly half, kept bit odd: up to even
    (0xBF818000, 0xBF82),   # same, negative
    (0x7F7FFFFF, 0x7F80),   # largest finite rounds to +inf
    (0x7F800000, 0x7F80),   # +inf stays
    (0x00008000, 0x0000),   # subnormal half-way, even: to +0
    (0x00018000, 0x0002),   # subnormal half-way, odd: up
    (0x80000000, 0x8000),   # -0
])
def test_bf16_rne_handpicked(pattern, expect):
    got = _bf16_bits(oracle.to_bf16(_bits([pattern])))[0]
    assert got == expect, hex(got)


def test_bf16_nan_stays_nan():
    x = _bits([0x7F800001, 0xFFC00000])
    assert np.all(np.isnan(oracle.to_bf16(x)))


def test_bf16_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    a = rng.standard_normal(200000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 200000)
    a = a.astype(np.float32)
    # force many exact half-way cases
    u = a.view(np.uint32)
    u[::3] = (u[::3] & 0xFFFF0000) | 0x8000
    ours = oracle.to_bf16(a)
    ref = torch.from_numpy(a.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_fma32_exact_against_rationals():
    rng = np.random.default_rng(3)
    n = 4000
    a = rng.standard_normal(n).astype(np.float32)
    b = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    c = rng.standard_normal(n).astype(np.float32)
    # constructed double-rounding cases: a*b = 2^-24 - 2^-70 and c = 1 + 2^-23, so
    # fl64(a*b + c) is the fp32 midpoint 1 + 3*2^-24 and rounding it once more to
    # even would give 1 + 2^-22, while the exact sum lies below the midpoint
    a[:50] = np.float32(1.0 + 2.0 ** -23)
    b[:50] = np.float32(2.0 ** -24 * (1.0 - 2.0 ** -23))
    c[:50] = np.float32(1.0 + 2.0 ** -23)
    a[50:100] = -a[:50]
    b[50:100] = b[:50]
    c[50:100] = -c[:50]
    got = oracle.fma32(a, b, c)
    naive = (a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64)).astype(np.float32)
    assert np.all(naive[:100] != got[:100])     # the midpoint fix-up is exercised
    assert np.all(got[:50] == np.float32(1.0 + 2.0 ** -23))
    for i in range(n):
        exact = Fraction(float(a[i])) * Fraction(float(b[i])) + Fraction(float(c[i]))
        # correct rounding: the nearest fp32, ties to even
        r = np.float32(float(exact))
        cands = [np.nextafter(r, np.float32(-np.inf)), r, np.nextafter(r, np.float32(np.inf))]
        dists = [abs(Fraction(float(v)) - exact) for v in cands]
        best = min(dists)
        winners = [v for v, d in zip(cands, dists) if d == best]
        if len(winners) > 1:
            winners = [v for v in winners if (int(np.float32(v).view(np.uint32)) & 1) == 0]
        assert got[i].view(np.uint32) == np.float32(winners[0]).view(np.uint32), i


# ---------------------------------------------------------------------------
# softmax cross-entropy
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("C", [10, 100])
def test_ce_zero_logits_is_ln_C(C):
    loss, dz = oracle.softmax_ce(np.zeros((5, C)), np.arange(5) % C)
    assert abs(loss - math.log(C)) < 1e-15
    assert abs(loss - {10: 2.302585093, 100: 4.605170186}[C]) < 1e-9


def test_ce_against_scipy():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((33, 17)) * 4
    y = rng.integers(0, 17, 33)
    loss, dz = oracle.softmax_ce(z, y)
    ref = np.mean(scipy.special.logsumexp(z, axis=1) - z[np.arange(33), y])
    assert abs(loss - ref) < 1e-12
    P = scipy.special.softmax(z, axis=1)
    Y = np.eye(17)[y]
    np.testing.assert_allclose(dz, (P - Y) / 33, atol=1e-15)
    np.testing.assert_allclose(dz.sum(axis=1), 0, atol=1e-15)


def test_ce_finite_differences():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((4, 6))
    y = rng.integers(0, 6, 4)
    _, dz = oracle.softmax_ce(z, y)
    eps = 1e-6
    for b in range(4):
        for c in range(6):
            zp, zm = z.copy(), z.copy()
            zp[b, c] += eps
            zm[b, c] -= eps
            fd = (oracle.softmax_ce(zp, y)[0] - oracle.softmax_ce(zm, y)[0]) / (2 * eps)
            assert abs(fd - dz[b, c]) < 1e-9


# ---------------------------------------------------------------------------
# Linear: one layer is multinomial logistic regression
# ---------------------------------------------------------------------------
def test_single_linear_is_logistic_regression():
    rng = np.random.default_rng(4)
    B, F, C = 9, 7, 5
    spec = {"layers": [("linear", C)], "num_classes": C}
    Wt = rng.standard_normal((C, F))
    bt = rng.standard_normal(C)
    x = rng.standard_normal((B, F))
    y = rng.integers(0, C, B)
    logits, cache = oracle.forward(spec, [Wt, bt], x, "f64")
    loss, dz = oracle.softmax_ce(logits, y)
    gW, gb = oracle.backward(spec, [Wt, bt], cache, dz, "f64")
    P = scipy.special.softmax(x @ Wt.T + bt, axis=1)
    Y = np.eye(C)[y]
    np.testing.assert_allclose(gW, (P - Y).T @ x / B, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gb, (P - Y).mean(axis=0), rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# Convolution
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("pad,k", [(0, 5), (1, 3), (2, 3), (0, 1)])
def test_conv_forward_against_scipy(pad, k):
    rng = np.random.default_rng(5 + pad + k)
    n, c, o, H, Wd = 2, 3, 4, 7, 6
    h = rng.standard_normal((n, c, H, Wd))
    Wt = rng.standard_normal((o, c, k, k))
    b = rng.standard_normal(o)
    z = oracle.conv2d_fwd(h, Wt, b, pad)
    for ni in range(n):
        for oi in range(o):
            ref = b[oi] + sum(
                scipy.signal.correlate2d(np.pad(h[ni, ci], pad), Wt[oi, ci], mode="valid")
                for ci in range(c))
            np.testing.assert_allclose(z[ni, oi], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("pad,k", [(0, 5), (1, 3)])
def test_conv_backward_adjoint(pad, k):
    """<conv(x; W), g> = <x, dh(g)> = <W, dW(x, g)> (the map is bilinear in x and W)."""
    rng = np.random.default_rng(11)
    n, c, o, H, Wd = 2, 3, 4, 8, 9
    h = rng.standard_normal((n, c, H, Wd))
    Wt = rng.standard_normal((o, c, k, k))
    z = oracle.conv2d_fwd(h, Wt, np.zeros(o), pad)
    g = rng.standard_normal(z.shape)
    dW, db, dh = oracle.conv2d_bwd(g, h, Wt, pad)
    lhs = float(np.sum(z * g))
    assert abs(lhs - float(np.sum(h * dh))) < 1e-9 * max(1, abs(lhs))
    assert abs(lhs - float(np.sum(Wt * dW))) < 1e-9 * max(1, abs(lhs))
    np.testing.assert_allclose(db, g.sum(axis=(0, 2, 3)), rtol=1e-13)


# ---------------------------------------------------------------------------
# Max-pool and ReLU
# ---------------------------------------------------------------------------
def test_maxpool_ties_first_in_row_major_order():
    h = np.zeros((1, 1, 4, 6))
    h[0, 0, 0:2, 0:2] = [[1, 3], [3, 2]]        # two-way tie (0,1),(1,0) -> index 1
    h[0, 0, 0:2, 2:4] = [[5, 5], [5, 5]]        # four-way tie -> index 0
    h[0, 0, 0:2, 4:6] = [[-1, -2], [7, 7]]      # tie in the second row -> index 2
    h[0, 0, 2:4, 0:2] = [[0, 0], [0, 9]]        # unique max -> index 3
    h[0, 0, 2:4, 2:4] = [[-3, -1], [-1, -2]]    # all negative, tie -> index 1
    h[0, 0, 2:4, 4:6] = [[4, 1], [4, 4]]        # three-way tie -> index 0
    out, am = oracle.maxpool2_fwd(h)
    np.testing.assert_array_equal(am[0, 0], [[1, 0, 2], [3, 1, 0]])
    np.testing.assert_array_equal(out[0, 0], [[3, 5, 7], [9, -1, 4]])
    g = oracle.maxpool2_bwd(np.arange(1, 7, dtype=float).reshape(1, 1, 2, 3), am, h.shape)
    expect = np.zeros((4, 6))
    expect[0, 1] = 1
    expect[0, 2] = 2
    expect[1, 4] = 3
    expect[3, 1] = 4
    expect[2, 3] = 5
    expect[2, 4] = 6
    np.testing.assert_array_equal(g[0, 0], expect)


def test_maxpool_floor_mode_odd_sizes():
    h = np.arange(2 * 5 * 7, dtype=float).reshape(1, 2, 5, 7)
    out, am = oracle.maxpool2_fwd(h)
    assert out.shape == (1, 2, 2, 3)
    assert np.all(am == 3)
    g = oracle.maxpool2_bwd(np.ones(out.shape), am, h.shape)
    assert g[:, :, 4, :].sum() == 0 and g[:, :, :, 6].sum() == 0
    assert g.sum() == out.size


def test_relu_derivative_at_zero_is_zero():
    z = np.array([[-1.0, 0.0, 2.0]])
    y = oracle.relu_fwd(z)
    np.testing.assert_array_equal(oracle.relu_bwd(np.ones_like(z), y), [[0, 0, 1]])


# ---------------------------------------------------------------------------
# Whole models: central finite differences in fp64
# ---------------------------------------------------------------------------
def _fd_check(spec, in_shape, seed, n_samples=None, eps=1e-6, tol=2e-6):
    rng = np.random.default_rng(seed)
    params = [p.astype(np.float64) for p in W.init_params(spec, in_shape, seed, 0)]
    B = 3
    x = rng.standard_normal((B,) + tuple(in_shape))
    y = rng.integers(0, spec["num_classes"], B)
    logits, cache = oracle.forward(spec, params, x, "f64")
    _, dz = oracle.softmax_ce(logits, y)
    grads = oracle.backward(spec, params, cache, dz, "f64")
    checked = 0
    for t, (p, g) in enumerate(zip(params, grads)):
        flat = list(range(p.size))
        if n_samples is not None and p.size > n_samples:
            flat = list(rng.choice(p.size, n_samples, replace=False))
        for j in flat:
            idx = np.unravel_index(j, p.shape)
            old = p[idx]
            p[idx] = old + eps
            lp = oracle.loss_only(spec, params, x, y)
            p[idx] = old - eps
            lm = oracle.loss_only(spec, params, x, y)
            p[idx] = old
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - g[idx]) <= tol * max(1.0, abs(fd)), (t, idx, fd, g[idx])
            checked += 1
    return checked


def test_fd_mlp_two_hidden():
    spec = {"layers": [("linear", 7), ("relu",), ("linear", 5), ("relu",), ("linear", 4)],
            "num_classes": 4}
    assert _fd_check(spec, (6,), 21) > 100


def test_fd_cnn_conv_relu_pool():
    spec = {"layers": [("conv", 3, 3, 1), ("relu",), ("pool",),
                       ("conv", 4, 3, 0), ("relu",), ("pool",), ("flatten",),
                       ("linear", 5), ("relu",), ("linear", 3)], "num_classes": 3}
    assert _fd_check(spec, (2, 9, 10), 22, n_samples=12) > 50


def test_fd_lenet_like_small():
    spec = {"layers": [("conv", 2, 5, 0), ("relu",), ("pool",), ("flatten",), ("linear", 3)],
            "num_classes": 3}
    assert _fd_check(spec, (1, 10, 10), 23, n_samples=20) > 20


# Residual blocks: inner(x) + x, with a ReLU after the block applied to the sum
_RES_SPEC = {"layers": [("linear", 6), ("relu",),
                        ("res_begin",), ("linear", 6), ("res_end",), ("relu",),
                        ("res_begin",), ("linear", 5), ("relu",), ("linear", 6), ("res_end",), ("relu",),
                        ("linear", 4)], "num_classes": 4}


def test_fd_residual_blocks():
    # the backward (both paths into a block's input) against the forward's own loss
    assert _fd_check(_RES_SPEC, (7,), 24) > 150


def test_residual_forward_matches_torch_modules():
    # the forward against an nn.Module graph with the skip written as x + inner(x)
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(25)
    params = [p.astype(np.float64) for p in W.init_params(_RES_SPEC, (7,), 25, 0)]
    x = rng.standard_normal((5, 7))
    lin = lambda i, h: torch.nn.functional.linear(h, torch.from_numpy(params[2 * i]), torch.from_numpy(params[2 * i + 1]))
    h = torch.relu(lin(0, torch.from_numpy(x)))
    h = torch.relu(lin(1, h) + h)
    h = torch.relu(lin(3, torch.relu(lin(2, h))) + h)
    ref = lin(4, h).numpy()
    got, _ = oracle.forward(_RES_SPEC, params, x, "f64")
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_residual_with_zero_inner_layers_is_the_identity():
    # zero weights and biases inside a block: the block passes x through, so the
    # model equals the one without the block (forward, and gradients of the rest)
    spec = {"layers": [("linear", 6), ("relu",), ("res_begin",), ("linear", 6), ("res_end",), ("relu",),
                       ("linear", 4)], "num_classes": 4}
    plain = {"layers": [("linear", 6), ("relu",), ("linear", 4)], "num_classes": 4}
    rng = np.random.default_rng(26)
    params = [p.astype(np.float64) for p in W.init_params(spec, (7,), 26, 0)]
    params[2][:] = 0.0
    params[3][:] = 0.0
    x = rng.standard_normal((5, 7))
    y = rng.integers(0, 4, 5)
    keep = [params[0], params[1], params[4], params[5]]
    z1, c1 = oracle.forward(spec, params, x, "f64")
    z0, c0 = oracle.forward(plain, keep, x, "f64")
    np.testing.assert_array_equal(z1, z0)
    g1 = oracle.backward(spec, params, c1, oracle.softmax_ce(z1, y)[1], "f64")
    g0 = oracle.backward(plain, keep, c0, oracle.softmax_ce(z0, y)[1], "f64")
    for a, b in zip([g1[0], g1[1], g1[4], g1[5]], g0):
        np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-15)


_RES_CNN = {"layers": [("conv", 3, 3, 1), ("relu",),
                       ("res_begin",), ("conv", 4, 3, 1), ("relu",), ("conv", 3, 3, 1), ("res_end",), ("relu",),
                       ("pool",), ("flatten",), ("linear", 3)], "num_classes": 3}


def test_fd_residual_conv_block():
    assert _fd_check(_RES_CNN, (2, 6, 6), 28, n_samples=12) > 50


def test_residual_conv_forward_matches_torch_modules():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    rng = np.random.default_rng(29)
    params = [p.astype(np.float64) for p in W.init_params(_RES_CNN, (2, 6, 6), 29, 0)]
    t = [torch.from_numpy(p) for p in params]
    x = rng.standard_normal((3, 2, 6, 6))
    h = torch.relu(F.conv2d(torch.from_numpy(x), t[0], t[1], padding=1))
    h = torch.relu(F.conv2d(torch.relu(F.conv2d(h, t[2], t[3], padding=1)), t[4], t[5], padding=1) + h)
    ref = F.linear(F.max_pool2d(h, 2).flatten(1), t[6], t[7]).numpy()
    got, _ = oracle.forward(_RES_CNN, params, x, "f64")
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_residual_spec_errors():
    params = [p.astype(np.float64) for p in W.init_params(_RES_SPEC, (7,), 27, 0)]
    x = np.zeros((2, 7))
    bad = {"layers": [("linear", 6), ("res_begin",), ("linear", 5), ("res_end",), ("linear", 4)],
           "num_classes": 4}
    with pytest.raises(ValueError):
        oracle.forward(bad, [p.astype(np.float64) for p in W.init_params(bad, (7,), 27, 0)], x, "f64")
    assert oracle.count_params(_RES_SPEC, (7,)) == sum(p.size for p in params)


# ---------------------------------------------------------------------------
# Shapes and parameter counts
# ---------------------------------------------------------------------------
def _golden_counts():
    out = {}
    with open(os.path.join(GOLDEN, "param_counts.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                name, val = line.split()[:2]
                out[name] = int(val)
    return out


def test_param_counts_against_paper_table():
    g = _golden_counts()
    lenet = W.lenet4().specs[0]
    lenet6 = {"layers": [("conv", 6, 5, 0)] + list(lenet["layers"][1:]), "num_classes": 10}
    n = oracle.count_params(lenet6, (1, 28, 28))
    assert n == g["lenet_c6_pad0"]
    assert n + 2 * (6 + 16) == g["paper_lenet_table2"]
    pad2 = {"layers": [("conv", 6, 5, 2)] + list(lenet["layers"][1:3]) +
            [("conv", 16, 5, 0)] + list(lenet["layers"][4:]), "num_classes": 10}
    assert oracle.count_params(pad2, (1, 28, 28)) == g["lenet_c6_pad2_variant"]
    mlp = W.mlp2_tiny()
    assert oracle.count_params(mlp.specs[0], (784,)) == g["mlp_784_128_10"]
    assert oracle.count_params(mlp.specs[1], (784,)) == g["mlp_784_64_10"]


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_param_count_agrees_with_generator(name):
    wl = W.get(name)
    for i, spec in enumerate(wl.specs[:4]):
        n = sum(int(np.prod(s)) for s, _ in W.param_shapes(spec, wl.in_shape))
        assert n == oracle.count_params(spec, wl.in_shape)


# ---------------------------------------------------------------------------
# SGD and training
# ---------------------------------------------------------------------------
def test_sgd_lr_zero_leaves_params_bitwise():
    rng = np.random.default_rng(8)
    p = [rng.standard_normal(50).astype(np.float32)]
    g = [rng.standard_normal(50).astype(np.float32)]
    q = oracle.sgd_update(p, g, 0.0)
    assert np.array_equal(p[0].view(np.uint32), q[0].view(np.uint32))


def test_sgd_is_theta_minus_lr_g():
    rng = np.random.default_rng(9)
    p = [rng.standard_normal(1000).astype(np.float32)]
    g = [rng.standard_normal(1000).astype(np.float32)]
    q = oracle.sgd_update(p, g, 0.01)[0]
    ref = p[0].astype(np.float64) - np.float64(np.float32(0.01)) * g[0].astype(np.float64)
    assert np.max(np.abs(q - ref)) <= np.max(np.spacing(np.abs(q)))


def test_training_reduces_loss_on_a_fixed_batch():
    wl = W.mlp2_tiny()
    x, y = W.make_batch(wl, 0)
    p0 = W.init_params(wl.specs[0], wl.in_shape, 0, 0)
    losses, _, _ = oracle.train(wl.specs[0], p0, [(x, y)] * 30, 0.05, "f32")
    assert losses[-1] < 0.5 * losses[0]


def test_bf16_mode_equals_f32_mode_on_prerounded_operands():
    """A one-layer model: bf16 mode only rounds the operands, so pre-rounding them
    and running in f32 mode gives the same logits bit for bit."""
    rng = np.random.default_rng(12)
    spec = {"layers": [("linear", 10)], "num_classes": 10}
    x = rng.standard_normal((8, 32)).astype(np.float32)
    Wt = rng.standard_normal((10, 32)).astype(np.float32)
    b = rng.standard_normal(10).astype(np.float32)
    lb, _ = oracle.forward(spec, [Wt, b], x, "bf16")
    lf, _ = oracle.forward(spec, [oracle.to_bf16(Wt), b], oracle.to_bf16(x), "f32")
    assert np.array_equal(lb, lf)
    l32, _ = oracle.forward(spec, [Wt, b], x, "f32")
    assert not np.array_equal(lb, l32)
    assert np.max(np.abs(lb - l32)) < 0.1


def test_f32_mode_close_to_f64():
    wl = W.lenet4()
    spec = wl.specs[0]
    p = W.init_params(spec, wl.in_shape, 0, 0)
    x, y = W.make_batch(W.shrink(wl, batch=8), 0)
    l32, _, g32 = oracle.step(spec, p, x, y, 0.01, "f32")
    l64, _, g64 = oracle.step(spec, [q.astype(np.float64) for q in p], x, y, 0.01, "f64")
    assert abs(l32 - l64) < 1e-6
    for a, b in zip(g32, g64):
        assert np.max(np.abs(a - b)) <= 1e-5 * np.max(np.abs(b)) + 1e-12


# ---------------------------------------------------------------------------
# Ill-conditioned discrete decisions
# ---------------------------------------------------------------------------
def test_flags_mark_relu_inputs_within_fp32_rounding_of_zero():
    spec = {"layers": [("linear", 3), ("relu",), ("linear", 2)], "num_classes": 2}
    W1 = np.array([[1.0, -1.0], [1.0, 1.0], [2.0 ** -30, 0.0]], dtype=np.float32)
    b1 = np.zeros(3, dtype=np.float32)
    W2 = np.ones((2, 3), dtype=np.float32)
    b2 = np.zeros(2, dtype=np.float32)
    x = np.array([[0.5, 0.5], [1.0, 2.0]], dtype=np.float32)
    flags = {}
    oracle.forward(spec, [W1, b1, W2, b2], x, "f32", flags)
    # unit 0: z = 0 exactly for sample 0; unit 2: z = 2^-31 << u * |h||w| is not
    # the case (|z| equals the magnitude sum, so it is well conditioned)
    assert flags[0] == {0}


def test_flags_mark_near_tied_pool_windows():
    spec = {"layers": [("conv", 1, 1, 0), ("pool",), ("flatten",), ("linear", 2)], "num_classes": 2}
    Wc = np.ones((1, 1, 1, 1), dtype=np.float32)
    bc = np.zeros(1, dtype=np.float32)
    Wl = np.ones((2, 1), dtype=np.float32)
    bl = np.zeros(2, dtype=np.float32)
    near = np.array([[[[1.0, 1.0 + 2.0 ** -26], [0.5, 0.25]]]], dtype=np.float64)
    far = np.array([[[[1.0, 1.5], [0.5, 0.25]]]], dtype=np.float64)
    f1, f2 = {}, {}
    oracle.forward(spec, [Wc, bc, Wl, bl], near, "f64", f1)
    oracle.forward(spec, [Wc, bc, Wl, bl], far, "f64", f2)
    assert f1.get(0) == {0} and not f2.get(0)
