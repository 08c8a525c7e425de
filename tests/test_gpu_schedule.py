"""GPU: active sets of the fused step (un_set_active) and the schedules built on
them (Trainer section of the paper: scheduling policies, and the Model
Separator handing a finished model back while the others go on).

A model outside the active set neither runs nor changes; a model inside it
sees exactly the step it would see alone. So every model of a masked run must
equal, bit for bit, the same model trained alone (N=1) on the batches of the
steps it was active in, and match the oracle trained on those batches.
"""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W
from paper_2408_01331_amd.scheduler import Schedule, train
from _parity import compare_run, oracle_spread, theta0

pytestmark = pytest.mark.gpu


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _masks(n, steps):
    """A mask per step with gaps inside the model range (so the concatenated
    first-layer GEMM splits into several runs), a lone model, repeats (no
    re-plan), and a final all-active step (so every model's gradients are
    those of its last active step)."""
    full = np.ones(n, dtype=bool)
    gappy = np.array([i % 3 != 1 for i in range(n)])
    lone = np.zeros(n, dtype=bool)
    lone[n // 2] = True
    ends = np.zeros(n, dtype=bool)
    ends[[0, n - 1]] = True
    seq = [full, gappy, lone, lone, ends, ~gappy, full]
    return seq[:steps - 1] + [full] if steps < len(seq) else seq


def _run_masked(wl, masks, lr=None):
    """Train all models of `wl` on the GPU, step s under masks[s].

    Returns (losses [steps, N], params {i: flat}, grads {i: flat}, snapshots)
    where snapshots[s] holds every model's flat parameters after step s."""
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    lr = wl.lr if lr is None else lr
    losses, snaps = [], []
    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        h.keep_grads(True)
        for i in range(wl.n_models):
            h.set_params(i, flatten_params(theta0(wl, i)))
        cur = None
        for s, m in enumerate(masks):
            if cur is None or not np.array_equal(cur, m):
                h.set_active(m)
                cur = m
            x, y = W.make_batch(wl, s)
            h.load_batch(x, y)
            losses.append(h.step(lr))
            snaps.append({i: h.get_params(i).copy() for i in range(wl.n_models)})
        params = {i: h.get_params(i) for i in range(wl.n_models)}
        grads = {i: h.get_grads(i) for i in range(wl.n_models)}
    return np.array(losses), params, grads, snaps


def _run_alone(wl, i, steps, lr=None):
    """Model i of `wl` alone (N=1) on the batches of the listed global steps."""
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    lr = wl.lr if lr is None else lr
    with Hybrid([wl.specs[i]], wl.batch, wl.in_shape, wl.precision) as h:
        h.keep_grads(True)
        h.set_params(0, flatten_params(theta0(wl, i)))
        losses = []
        for s in steps:
            x, y = W.make_batch(wl, s)
            h.load_batch(x, y)
            losses.append(h.step(lr)[0])
        return np.array(losses, dtype=np.float32), h.get_params(0), h.get_grads(0)


def _case(name):
    if name == "mlp64_8":
        return W.shrink(W.get("mlp64"), n_models=8)
    if name == "cifar16_4":
        return W.shrink(W.get("cifar16"), n_models=4, batch=64)
    return W.get(name)


# f32 and bf16 (bf16 shadows of the master weights must be refreshed when the
# active set changes), MLPs (concatenated first layer) and CNNs.
CASES = ["mlp8", "lenet4", "mlp64_8", "cifar16_4"]


@pytest.mark.parametrize("name", CASES)
def test_masked_steps_equal_each_model_alone_bitwise(name):
    _need_gpu()
    wl = _case(name)
    masks = _masks(wl.n_models, 7)
    print(f"\n[{wl.name}] masks {[np.flatnonzero(m).tolist() for m in masks]}", flush=True)
    losses, params, grads, snaps = _run_masked(wl, masks)
    for i in range(wl.n_models):
        on = [s for s, m in enumerate(masks) if m[i]]
        # losses: NaN exactly where the model sat out
        assert np.all(np.isnan(losses[[s for s in range(len(masks)) if s not in on], i]))
        assert np.all(np.isfinite(losses[on, i]))
        # parameters frozen while out
        for s in range(1, len(masks)):
            if not masks[s][i]:
                assert np.array_equal(_bits(snaps[s][i]), _bits(snaps[s - 1][i])), f"model {i} moved at step {s}"
        la, pa, ga = _run_alone(wl, i, on)
        assert np.array_equal(_bits(losses[on, i]), _bits(la)), f"model {i}: losses differ from alone"
        assert np.array_equal(_bits(params[i]), _bits(pa)), f"model {i}: params differ from alone"
        assert np.array_equal(_bits(grads[i]), _bits(ga)), f"model {i}: grads differ from alone"


@pytest.mark.parametrize("name,models", [("mlp8", None), ("mlp64_8", [0, 1, 4, 7]), ("cifar16_4", [1, 2])])
def test_masked_run_matches_the_oracle_on_each_models_batches(name, models):
    _need_gpu()
    from paper_2408_01331_amd.unifiednn import split_params
    wl = _case(name)
    masks = _masks(wl.n_models, 7)
    losses, params, grads, _ = _run_masked(wl, masks)
    models = list(range(wl.n_models)) if models is None else models
    for i in models:
        on = [s for s, m in enumerate(masks) if m[i]]
        orc, spread = _oracle_on_steps(wl, i, on)   # model i alone on the batches of its active steps
        shapes = [sh for sh, _ in W.param_shapes(wl.specs[i], wl.in_shape)]
        L = np.full((len(on), wl.n_models), np.nan, dtype=np.float32)
        L[:, i] = losses[on, i]
        gpu = (L, {i: split_params(params[i], shapes)}, {i: split_params(grads[i], shapes)})
        worst = compare_run(wl, gpu, {i: orc}, [i], spread={i: spread})
        print(f"\n[{wl.name} model {i}, steps {on}] " + ", ".join(f"{k}={v:.3g}" for k, v in worst.items()),
              flush=True)


def _oracle_on_steps(wl, i, steps):
    """Model i alone on the batches of the listed steps, and the spread of the
    oracle's two evaluation orders over them."""
    import oracle
    batches = [W.make_batch(wl, s) for s in steps]
    out = oracle.train_models(wl.specs, {i: theta0(wl, i)}, batches, wl.lr, wl.precision, models=[i],
                              with_flags=True)
    return out[i], oracle_spread(wl.specs[i], theta0(wl, i), batches, wl.lr, wl.precision, out[i][3], out[i][:3])


def test_fcfs_schedule_releases_each_model_as_trained_alone():
    """First come first serve, two at a time: each model is handed back (Model
    Separator) the moment its epochs are done, while the others continue, and
    equals that model trained alone on the batches of its steps."""
    _need_gpu()
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    wl = W.get("mlp8")
    sched = Schedule([1, 2, 1, 1, 2, 1, 1, 1], steps_per_epoch=2, policy="fcfs", capacity=2)
    plan = sched.plan()
    released, order, at = {}, [], []

    def release(i, p):
        released[i] = p.copy()
        order.append(i)
        at.append(sched.steps)

    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        for i in range(wl.n_models):
            h.set_params(i, flatten_params(theta0(wl, i)))
        losses = train(h, sched, lambda s: W.make_batch(wl, s), wl.lr, on_release=release)
        final = {i: h.get_params(i) for i in range(wl.n_models)}
    assert order == sched.finished and sorted(order) == list(range(wl.n_models))
    assert at[0] < len(plan)                     # released while others still train
    assert losses.shape == (len(plan), wl.n_models)
    for i in range(wl.n_models):
        on = [s for s, m in enumerate(plan) if m[i]]
        _, pa, _ = _run_alone(wl, i, on)
        assert np.array_equal(_bits(released[i]), _bits(pa)), f"model {i}: released params differ from alone"
        assert np.array_equal(_bits(final[i]), _bits(pa)), f"model {i}: changed after release"


def test_active_set_errors_leave_state_unchanged():
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    wl = W.get("mlp2")
    x, y = W.make_batch(wl, 0)
    with U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        h.keep_grads(True)
        with pytest.raises(U.UnError) as e:
            h.set_active([False, False])
        assert e.value.status == U.UN_ERR_INVALID
        with pytest.raises(ValueError):
            h.set_active([True])
        h.load_batch(x, y)
        l0 = h.step(0.01)                       # still both models
        assert np.all(np.isfinite(l0))
        h.set_active([False, True])
        with pytest.raises(U.UnError) as e:     # no step since the set changed
            h.get_grads(1)
        assert e.value.status == U.UN_ERR_STATE
        p0 = h.get_params(0)
        l1 = h.step(0.01)
        assert np.isnan(l1[0]) and np.isfinite(l1[1])
        with pytest.raises(U.UnError) as e:     # model 0 did not run
            h.get_grads(0)
        assert e.value.status == U.UN_ERR_STATE
        assert h.get_grads(1).size == h.get_params(1).size
        assert np.array_equal(_bits(h.get_params(0)), _bits(p0))
        h.set_active([True, True])
        assert np.all(np.isfinite(h.step(0.01)))
