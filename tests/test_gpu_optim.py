"""GPU: per-model optimizers (plain SGD, SGD with momentum, Adam) fused into
the same step, and per-model checkpoint / resume with optimizer state.

Every model of a fused step with mixed optimizers must equal, bit for bit
(losses, parameters, gradients, optimizer state), the same model trained
alone with its optimizer, and match the oracle's torch.optim-pinned updates.
A run interrupted by a checkpoint and resumed in a fresh context must equal
the uninterrupted run bit for bit.
"""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W
from _parity import TOL, UPDATE_TOL, compare_run, flagged_masks, fro_err, tensor_err, theta0

pytestmark = pytest.mark.gpu

# Adam moves every weight by about lr per step whatever the gradient's size, so
# a gradient element within rounding of zero may move either way. In the
# multi-step runs below the rate is kept small enough that such an element
# stays inside the bound of flagged parameters; test_optimizer_step_strict
# compares one step at the workload's own rate with those elements flagged.
OPTS = [dict(kind="sgd"), dict(kind="momentum", momentum=0.9),
        dict(kind="adam", betas=(0.9, 0.999), eps=1e-8, lr_scale=0.005)]


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _case(name):
    if name == "mlp64_8":
        return W.shrink(W.get("mlp64"), n_models=8)
    if name == "mlp8_b1100":
        # more than 1024 rows: the weight gradients are split-K, their
        # updates (each model's optimizer and rate) done by the reduction
        return W.shrink(W.get("mlp8"), batch=1100)
    if name == "cifar16_4":
        return W.shrink(W.get("cifar16"), n_models=4, batch=64)
    return W.get(name)


def _opt(i):
    return OPTS[i % len(OPTS)]


def _rates(wl):
    return np.array([wl.lr * _opt(i).get("lr_scale", 1.0) for i in range(wl.n_models)], np.float32)


def _set(h, i, o):
    h.set_optimizer(i, o["kind"], o.get("momentum", 0.0), o.get("betas", (0.9, 0.999)), o.get("eps", 1e-8))


def _run(wl, steps, models=None, masks=None, start=0, h=None):
    """Train `models` of wl (all by default) for `steps` steps from step `start`,
    each model with its optimizer and rate. Returns (losses, params, grads, states)."""
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    idx = list(range(wl.n_models)) if models is None else list(models)
    own = h is None
    if own:
        h = Hybrid([wl.specs[i] for i in idx], wl.batch, wl.in_shape, wl.precision)
        for k, i in enumerate(idx):
            h.set_params(k, flatten_params(theta0(wl, i)))
            _set(h, k, _opt(i))
    h.keep_grads(True)
    rates = _rates(wl)[idx]
    losses = []
    for s in range(start, start + steps):
        if masks is not None:
            h.set_active(masks[s])
        x, y = W.make_batch(wl, s)
        h.load_batch(x, y)
        losses.append(h.step(rates))
    params = {i: h.get_params(k) for k, i in enumerate(idx)}
    grads = {i: h.get_grads(k) for k, i in enumerate(idx)}
    states = {i: h.get_opt_state(k) for k, i in enumerate(idx)}
    if own:
        h.close()
    return np.array(losses), params, grads, states


@pytest.mark.parametrize("name", ["mlp8", "lenet4", "mlp64_8", "cifar16_4", "mlp8_b1100"])
def test_mixed_optimizers_equal_each_model_alone_bitwise(name):
    _need_gpu()
    wl = _case(name)
    steps = 3
    losses, params, grads, states = _run(wl, steps)
    for i in range(wl.n_models):
        la, pa, ga, sa = _run(wl, steps, models=[i])
        assert np.array_equal(_bits(losses[:, i]), _bits(la[:, 0])), f"model {i}: losses"
        assert np.array_equal(_bits(params[i]), _bits(pa[i])), f"model {i}: params"
        assert np.array_equal(_bits(grads[i]), _bits(ga[i])), f"model {i}: grads"
        assert states[i][1] == sa[i][1] == steps
        assert np.array_equal(_bits(states[i][0]), _bits(sa[i][0])), f"model {i}: optimizer state"
        k = {"sgd": 0, "momentum": 1, "adam": 2}[_opt(i)["kind"]]
        assert states[i][0].size == k * params[i].size


def _oracle(wl, i, steps):
    import oracle
    o = dict(_opt(i))
    o.setdefault("betas", (0.9, 0.999))
    o.setdefault("eps", 1e-8)
    o.setdefault("momentum", 0.0)
    lr = float(_rates(wl)[i])
    params = [np.array(p, dtype=np.float32) for p in theta0(wl, i)]
    losses, flags, st, grads = [], {}, {}, None
    for s in range(steps):
        x, y = W.make_batch(wl, s)
        loss, params, grads, st = oracle.step_opt(wl.specs[i], params, x, y, lr, o, st, wl.precision, flags)
        losses.append(loss)
    return (np.array(losses), params, grads, flags), st


@pytest.mark.parametrize("name,models", [("mlp8", None), ("lenet4", None), ("mlp64_8", [0, 1, 2, 5]),
                                         ("cifar16_4", [1, 2]), ("mlp8_b1100", None)])
def test_mixed_optimizers_match_the_oracle(name, models):
    _need_gpu()
    from paper_2408_01331_amd.unifiednn import split_params
    wl = _case(name)
    steps = 3
    losses, params, grads, states = _run(wl, steps)
    models = list(range(wl.n_models)) if models is None else models
    for i in models:
        orc, st = _oracle(wl, i, steps)
        shapes = [sh for sh, _ in W.param_shapes(wl.specs[i], wl.in_shape)]
        gpu = (losses, {i: split_params(params[i], shapes)}, {i: split_params(grads[i], shapes)})
        worst = compare_run(wl, gpu, {i: orc}, [i])
        # optimizer state: momentum buffer or Adam's moments, per tensor, over
        # the parameters of units the oracle did not flag (as the updates)
        s, n = states[i][0], params[i].size
        fm = flagged_masks(wl.specs[i], orc[1], orc[3])
        worst["state_fro"] = 0.0
        for k, key in enumerate(("s1", "s2")[: s.size // n]):
            for t, (a, b) in enumerate(zip(split_params(s[k * n:(k + 1) * n], shapes), st[key])):
                e = fro_err(np.asarray(a)[~fm[t]], np.asarray(b)[~fm[t]])
                worst["state_fro"] = max(worst["state_fro"], e)
                assert e <= UPDATE_TOL[wl.precision], f"model {i} {key} tensor {t}: {e:.3g}"
        print(f"\n[{wl.name} model {i} {_opt(i)['kind']}] " + ", ".join(f"{k}={v:.3g}" for k, v in worst.items()),
              flush=True)


def _flat_state(st, key, shapes):
    return np.concatenate([np.asarray(a, np.float32).ravel() for a in st[key]])


def _oracle_update(o, lr, params, grads, st):
    """The oracle's optimizer step of one model (fp32 mode): new params and state."""
    import oracle
    if o["kind"] == "momentum":
        p, b = oracle.momentum_update(params, grads, st["s1"], lr, o["momentum"], "f32")
        return p, {"t": st["t"] + 1, "s1": b}
    b1, b2 = o["betas"]
    p, m, v = oracle.adam_update(params, grads, st["s1"], st["s2"], st["t"] + 1, lr, b1, b2, o["eps"], "f32")
    return p, {"t": st["t"] + 1, "s1": m, "s2": v}


@pytest.mark.parametrize("kind", ["momentum", "adam"])
@pytest.mark.parametrize("name,models", [("mlp8", None), ("lenet4", None), ("mlp64_8", [0, 3, 7]),
                                         ("cifar16_4", [0, 3])])
def test_optimizer_step_strict(name, models, kind):
    """One step of momentum / Adam at the workload's own rate, both sides from
    the oracle's parameters and optimizer state after a first step (injected
    into the library with un_set_params / un_set_opt_state): loss, gradient,
    new parameters, update and new state within the gate per tensor (max
    relative error). Flagged: the oracle's ill-conditioned ReLU / pool units,
    and elements whose update is an ill-conditioned function of the gradient
    at the gradient's own tolerance eps = tol * max|g| (the oracle's update at
    g - eps or g + eps moves by more than tol * max|update|; for Adam, the
    elements whose gradient is within eps of a sign change); those are held
    to the oracle's own spread over [g - eps, g + eps]."""
    _need_gpu()
    import oracle
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params, split_params
    wl = _case(name)
    tol = TOL[wl.precision]
    o = {"kind": kind, "momentum": 0.9, "betas": (0.9, 0.999), "eps": 1e-8}
    models = list(range(wl.n_models)) if models is None else models
    x0, y0 = W.make_batch(wl, 0)
    x1, y1 = W.make_batch(wl, 1)
    start = {}
    for i in range(wl.n_models):
        _, p1, _, st1 = oracle.step_opt(wl.specs[i], theta0(wl, i), x0, y0, wl.lr, o, {}, wl.precision)
        start[i] = (p1, st1)
    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        h.keep_grads(True)
        for i in range(wl.n_models):
            p1, st1 = start[i]
            h.set_params(i, flatten_params(p1))
            _set(h, i, o)
            keys = ("s1",) if kind == "momentum" else ("s1", "s2")
            h.set_opt_state(i, np.concatenate([_flat_state(st1, k, None) for k in keys]), st1["t"])
        h.load_batch(x1, y1)
        losses = h.step(wl.lr)
        got = {i: (h.get_params(i), h.get_grads(i), h.get_opt_state(i)) for i in models}
    worst = {"loss": 0.0, "param": 0.0, "update": 0.0, "grad": 0.0, "state": 0.0, "ill_elements": 0,
             "ill_param": 0.0}
    for i in models:
        p1, st1 = start[i]
        flags = {}
        lo, p2, g2, st2 = oracle.step_opt(wl.specs[i], p1, x1, y1, wl.lr, o, st1, wl.precision, flags)
        le = abs(losses[i] - lo) / abs(lo)
        worst["loss"] = max(worst["loss"], le)
        assert le <= tol, f"model {i}: loss {losses[i]} vs {lo}"
        shapes = [sh for sh, _ in W.param_shapes(wl.specs[i], wl.in_shape)]
        pg, gg = split_params(got[i][0], shapes), split_params(got[i][1], shapes)
        n = got[i][0].size
        sg = [split_params(got[i][2][0][k * n:(k + 1) * n], shapes) for k in range(len(st2) - 1)]
        assert got[i][2][1] == st2["t"] == 2
        fm = flagged_masks(wl.specs[i], p2, flags)
        # the update's own conditioning at the gradient's tolerance
        eps = [tol * np.max(np.abs(g)) for g in g2]
        lo_p, _ = _oracle_update(o, wl.lr, p1, [np.asarray(g) - e for g, e in zip(g2, eps)], st1)
        hi_p, _ = _oracle_update(o, wl.lr, p1, [np.asarray(g) + e for g, e in zip(g2, eps)], st1)
        for t in range(len(p2)):
            u_o = np.asarray(p2[t], np.float64) - p1[t]
            spread = np.maximum(np.abs(np.asarray(lo_p[t], np.float64) - p2[t]),
                                np.abs(np.asarray(hi_p[t], np.float64) - p2[t]))
            ill = spread > tol * np.max(np.abs(u_o))
            keep = ~fm[t] & ~ill
            worst["ill_elements"] += int(np.count_nonzero(ill & ~fm[t]))
            checks = [("param", pg[t], p2[t]), ("update", np.asarray(pg[t], np.float64) - p1[t], u_o),
                      ("grad", gg[t], g2[t])]
            checks += [("state", sg[k][t], st2[key][t]) for k, key in enumerate(("s1", "s2")[:len(sg)])]
            for key, a, b in checks:
                mask = ~fm[t] if key == "grad" else keep
                e = tensor_err(a, b, mask)
                worst[key] = max(worst[key], e)
                assert e <= tol, f"model {i} tensor {t}: {key} err {e:.3g} > {tol}"
            sel = ill & ~fm[t]
            if sel.any():
                d = np.abs(np.asarray(pg[t], np.float64) - p2[t])[sel]
                assert np.all(d <= 1.5 * spread[sel] + tol * np.max(np.abs(u_o))), f"model {i} tensor {t}: ill"
                worst["ill_param"] = max(worst["ill_param"], float(np.max(d / (spread[sel] + 1e-30))))
    print(f"\n[{wl.name} {kind} one step at lr {wl.lr}] " + ", ".join(f"{k}={v:.3g}" for k, v in worst.items()),
          flush=True)


def test_adam_counts_only_the_steps_a_model_takes():
    """A model outside the active set takes no update and its Adam step count
    does not advance: it equals the model trained alone on its own steps."""
    _need_gpu()
    wl = W.get("mlp8")
    masks = [np.ones(8, bool), np.array([i % 2 == 0 for i in range(8)]), np.ones(8, bool)]
    losses, params, grads, states = _run(wl, 3, masks=masks)
    for i in (1, 2, 5):       # momentum / adam models, some of them sat out step 1
        on = [s for s in range(3) if masks[s][i]]
        from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
        with Hybrid([wl.specs[i]], wl.batch, wl.in_shape, wl.precision) as h:
            h.set_params(0, flatten_params(theta0(wl, i)))
            _set(h, 0, _opt(i))
            for s in on:
                x, y = W.make_batch(wl, s)
                h.load_batch(x, y)
                h.step(np.array([_rates(wl)[i]], np.float32))
            assert np.array_equal(_bits(params[i]), _bits(h.get_params(0))), f"model {i}"
            st, step = h.get_opt_state(0)
            assert step == states[i][1] == len(on)
            assert np.array_equal(_bits(states[i][0]), _bits(st))


@pytest.mark.parametrize("name", ["mlp8", "lenet4"])
def test_checkpoint_resume_equals_the_uninterrupted_run(name, tmp_path):
    _need_gpu()
    from paper_2408_01331_amd import checkpoint as C
    from paper_2408_01331_amd.unifiednn import Hybrid
    wl = W.get(name)
    full = _run(wl, 4)
    # two steps, one checkpoint file per model, a fresh context, two more steps
    from paper_2408_01331_amd.unifiednn import flatten_params
    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        for i in range(wl.n_models):
            h.set_params(i, flatten_params(theta0(wl, i)))
            _set(h, i, _opt(i))
        _run(wl, 2, h=h)
        for i in range(wl.n_models):
            C.save(h, i, str(tmp_path / f"m{i}.safetensors"))
    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as g:
        for i in range(wl.n_models):
            C.load(g, i, str(tmp_path / f"m{i}.safetensors"))
        resumed = _run(wl, 2, start=2, h=g)
    assert np.array_equal(_bits(resumed[0]), _bits(full[0][2:]))
    for i in range(wl.n_models):
        assert np.array_equal(_bits(resumed[1][i]), _bits(full[1][i])), f"model {i}: params"
        assert np.array_equal(_bits(resumed[3][i][0]), _bits(full[3][i][0])), f"model {i}: state"
        assert resumed[3][i][1] == full[3][i][1] == 4
    # a checkpoint also resumes a model alone, in a hybrid of one
    j = 2
    with Hybrid([wl.specs[j]], wl.batch, wl.in_shape, wl.precision) as a:
        C.load(a, 0, str(tmp_path / f"m{j}.safetensors"))
        for s in (2, 3):
            x, y = W.make_batch(wl, s)
            a.load_batch(x, y)
            a.step(np.array([_rates(wl)[j]], np.float32))
        assert np.array_equal(_bits(a.get_params(0)), _bits(full[1][j]))


def test_optimizer_errors_and_reset():
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    wl = W.get("mlp2")
    x, y = W.make_batch(wl, 0)
    with U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        with pytest.raises(ValueError):
            h.set_optimizer(0, "lion")
        for bad in (dict(kind="momentum", momentum=1.5), dict(kind="adam", betas=(0.9, 1.0)),
                    dict(kind="adam", eps=0.0)):
            with pytest.raises(U.UnError) as e:
                _set(h, 0, bad)
            assert e.value.status == U.UN_ERR_INVALID
        h.set_optimizer(0, "adam")
        n = h.get_params(0).size
        assert h.get_opt_state(0)[0].size == 2 * n and h.get_opt_state(0)[1] == 0
        with pytest.raises(U.UnError) as e:
            h.set_opt_state(0, np.zeros(n, np.float32), 3)
        assert e.value.status == U.UN_ERR_BUFSIZE
        h.load_batch(x, y)
        h.step(0.001)
        s, t = h.get_opt_state(0)
        assert t == 1 and np.any(s != 0)
        assert h.get_opt_state(1)[0].size == 0 and h.get_opt_state(1)[1] == 1   # plain SGD counts too
        h.set_optimizer(0, "adam")          # a fresh optimizer: zero state, count 0
        s, t = h.get_opt_state(0)
        assert t == 0 and not np.any(s)
