"""Pins of the oracle's per-model optimizers (CPU): SGD with momentum and Adam
against torch.optim's own implementations in float64, and closed forms."""
import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")


def _rand(seed, shapes):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(s) for s in shapes]


SHAPES = [(7, 5), (7,), (3, 2, 3, 3)]


def _torch_run(opt_factory, params, grads_seq):
    ps = [torch.tensor(p, dtype=torch.float64, requires_grad=True) for p in params]
    opt = opt_factory(ps)
    for grads in grads_seq:
        for p, g in zip(ps, grads):
            p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    return [p.detach().numpy() for p in ps], opt


def test_momentum_matches_torch_sgd():
    params = _rand(1, SHAPES)
    grads_seq = [_rand(10 + k, SHAPES) for k in range(4)]
    lr, mu = 0.05, 0.9
    ref, _ = _torch_run(lambda ps: torch.optim.SGD(ps, lr=lr, momentum=mu), params, grads_seq)
    p, b = params, [np.zeros(s) for s in SHAPES]
    for g in grads_seq:
        p, b = oracle.momentum_update(p, g, b, lr, mu, mode="f64")
    for a, r in zip(p, ref):
        np.testing.assert_allclose(a, r, rtol=1e-13, atol=1e-14)


def test_adam_matches_torch_adam():
    params = _rand(2, SHAPES)
    grads_seq = [_rand(20 + k, SHAPES) for k in range(5)]
    lr, b1, b2, eps = 1e-2, 0.8, 0.95, 1e-6
    ref, _ = _torch_run(lambda ps: torch.optim.Adam(ps, lr=lr, betas=(b1, b2), eps=eps), params, grads_seq)
    p, m, v = params, [np.zeros(s) for s in SHAPES], [np.zeros(s) for s in SHAPES]
    for t, g in enumerate(grads_seq, start=1):
        p, m, v = oracle.adam_update(p, g, m, v, t, lr, b1, b2, eps, mode="f64")
    for a, r in zip(p, ref):
        np.testing.assert_allclose(a, r, rtol=1e-12, atol=1e-13)


def test_momentum_zero_is_sgd_and_first_momentum_step_is_sgd():
    params = _rand(3, SHAPES)
    g = _rand(4, SHAPES)
    sgd = oracle.sgd_update(params, g, 0.1, mode="f64")
    m0, _ = oracle.momentum_update(params, g, [np.zeros(s) for s in SHAPES], 0.1, 0.0, mode="f64")
    m9, b = oracle.momentum_update(params, g, [np.zeros(s) for s in SHAPES], 0.1, 0.9, mode="f64")
    for a, c, d, bb, gg in zip(sgd, m0, m9, b, g):
        np.testing.assert_array_equal(a, c)
        np.testing.assert_array_equal(a, d)      # b starts at 0: the first step is plain SGD
        np.testing.assert_array_equal(bb, gg)


def test_adam_first_step_closed_form():
    """At t = 1 the bias corrections cancel: theta moves by lr * g / (|g| + eps)."""
    params = _rand(5, SHAPES)
    g = _rand(6, SHAPES)
    lr, eps = 1e-3, 1e-8
    p, m, v = oracle.adam_update(params, g, [np.zeros(s) for s in SHAPES], [np.zeros(s) for s in SHAPES], 1, lr,
                                 0.9, 0.999, eps, mode="f64")
    for a, p0, gg, mm, vv in zip(p, params, g, m, v):
        np.testing.assert_allclose(p0 - a, lr * gg / (np.abs(gg) + eps), rtol=1e-9)
        np.testing.assert_allclose(mm, 0.1 * gg, rtol=1e-12)
        np.testing.assert_allclose(vv, 0.001 * gg * gg, rtol=1e-12)


def test_fp32_modes_round_every_stored_value():
    params = [np.asarray(a, dtype=np.float32) for a in _rand(7, SHAPES)]
    g = [np.asarray(a, dtype=np.float32) for a in _rand(8, SHAPES)]
    zeros = [np.zeros(s, np.float32) for s in SHAPES]
    p, m, v = oracle.adam_update(params, g, zeros, zeros, 1, 1e-3, 0.9, 0.999, 1e-8, mode="f32")
    assert all(a.dtype == np.float32 for a in p + m + v)
    p64, m64, _ = oracle.adam_update(params, g, zeros, zeros, 1, 1e-3, 0.9, 0.999, 1e-8, mode="f64")
    for a, b in zip(m, m64):
        np.testing.assert_array_equal(a, b.astype(np.float32))


def test_step_opt_sgd_equals_step():
    from paper_2408_01331_amd import workloads as W
    wl = W.get("mlp2")
    x, y = W.make_batch(wl, 0)
    th = W.init_params(wl.specs[0], wl.in_shape, wl.seed, 0)
    l1, p1, g1 = oracle.step(wl.specs[0], th, x, y, 0.01)
    l2, p2, g2, st = oracle.step_opt(wl.specs[0], th, x, y, 0.01, {"kind": "sgd"}, {})
    assert l1 == l2 and st["t"] == 1
    for a, b in zip(p1, p2):
        np.testing.assert_array_equal(a, b)
