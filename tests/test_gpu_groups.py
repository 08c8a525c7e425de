"""GPU: models on different datasets in one hybrid (input groups,
un_create_grouped). Algorithm 2 gives every sub-model its own batches and the
Model Unifier lists input size and batch size among a sub-model's
hyper-parameters; the paper's own runs mix LeNet on MNIST with ResNets on
CIFAR. Each input group is one dataset with its own batch size and sample
shape, loaded once and read by its models.

Every model must match the oracle trained alone on its own group's batches,
and equal bit for bit the same model trained alone in a one-model context on
that data."""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W
from _parity import compare_run, compare_step, oracle_spread

pytestmark = pytest.mark.gpu

L, RELU, POOL, FLAT, RB, RE = (lambda n: ("linear", n)), ("relu",), ("pool",), ("flatten",), ("res_begin",), \
    ("res_end",)
# (sample shape, batch, classes, specs): MNIST-shaped, CIFAR-shaped, flat features
GROUPS = [
    ((1, 28, 28), 128, 10, [
        {"layers": [("conv", 6, 5, 0), RELU, POOL, ("conv", 16, 5, 0), RELU, POOL, FLAT, L(120), RELU, L(10)],
         "num_classes": 10},
        {"layers": [FLAT, L(64), RELU, L(10)], "num_classes": 10},
    ]),
    ((3, 32, 32), 64, 10, [
        {"layers": [("conv", 16, 3, 1), RELU, POOL, ("conv", 32, 3, 1), RELU, POOL, FLAT, L(10)], "num_classes": 10},
        {"layers": [("conv", 16, 3, 1), RELU, POOL, RB, ("conv", 16, 3, 1), RE, RELU, ("conv", 8, 3, 1), RELU, POOL,
                    FLAT, L(10)], "num_classes": 10},
    ]),
    ((104,), 37, 13, [
        {"layers": [L(37), RELU, L(129), RELU, L(13)], "num_classes": 13},
        {"layers": [L(200), RELU, L(13)], "num_classes": 13},
        {"layers": [L(13)], "num_classes": 13},
    ]),
]
LR = 0.02


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _layout(precision, groups=GROUPS):
    """specs, group_of, inputs, per-model one-model workloads, per-group workloads."""
    specs, group_of, inputs, model_wl, group_wl = [], [], [], [], []
    for g, (shape, batch, classes, gspecs) in enumerate(groups):
        inputs.append((batch, shape))
        group_wl.append(W.Workload(f"group{g}", len(gspecs), batch, shape, precision, gspecs, LR, 3, 20 + g,
                                   init="torch"))
        for s in gspecs:
            i = len(specs)
            specs.append(s)
            group_of.append(g)
            model_wl.append(W.Workload(f"model{i}", 1, batch, shape, precision, [s], LR, 3, 100 + i, init="torch"))
    return specs, group_of, inputs, model_wl, group_wl


def _theta(mwl):
    return W.init_params(mwl.specs[0], mwl.in_shape, mwl.seed, 0, mwl.init)


def _run(precision, steps, models=None, labels=None):
    """The grouped hybrid (or the listed models only, each with its group's
    data) for `steps` steps. Returns (losses [steps, n], params, grads)."""
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params, split_params
    specs, group_of, inputs, model_wl, group_wl = _layout(precision)
    idx = list(range(len(specs))) if models is None else list(models)
    used = sorted({group_of[i] for i in idx})
    remap = {g: k for k, g in enumerate(used)}
    with Hybrid([specs[i] for i in idx], None, None, precision, inputs=[inputs[g] for g in used],
                group_of=[remap[group_of[i]] for i in idx]) as h:
        h.keep_grads(True)
        for k, i in enumerate(idx):
            h.set_params(k, flatten_params(_theta(model_wl[i])))
        losses = []
        for s in range(steps):
            for g in used:
                x, y = W.make_batch(group_wl[g], s)
                h.load_batch(x, y, group=remap[g])
            if labels is not None:
                h.load_labels([labels(i, s) for i in idx])
            losses.append(h.step(LR))
        params, grads = {}, {}
        for k, i in enumerate(idx):
            shapes = [sh for sh, _ in W.param_shapes(specs[i], inputs[group_of[i]][1])]
            params[i] = split_params(h.get_params(k), shapes)
            grads[i] = split_params(h.get_grads(k), shapes)
    return np.array(losses), params, grads


def _oracle(precision, i, steps, labels=None):
    import oracle
    specs, group_of, inputs, model_wl, group_wl = _layout(precision)
    batches = []
    for s in range(steps):
        x, y = W.make_batch(group_wl[group_of[i]], s)
        batches.append((x, y if labels is None else labels(i, s)))
    flags = {}
    th = _theta(model_wl[i])
    ref = oracle.train(specs[i], th, batches, LR, precision, flags)
    spread = oracle_spread(specs[i], th, batches, LR, precision, flags, ref)
    return (ref[0], ref[1], ref[2], flags), spread


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_grouped_models_match_the_oracle(precision):
    _need_gpu()
    specs, group_of, inputs, model_wl, _ = _layout(precision)
    for steps in (1, 3):
        losses, params, grads = _run(precision, steps)
        for i in range(len(specs)):
            orc, spread = _oracle(precision, i, steps)
            gpu = (losses[:, i:i + 1], {0: params[i]}, {0: grads[i]})
            cmp = compare_step if steps == 1 else compare_run
            worst = cmp(model_wl[i], gpu, {0: orc}, [0], spread={0: spread})
            print(f"\n[groups {precision} {steps} steps model {i} (group {group_of[i]}, batch "
                  f"{inputs[group_of[i]][0]})] " + ", ".join(f"{k}={v:.3g}" for k, v in worst.items()), flush=True)


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_grouped_model_equals_itself_alone_bitwise(precision):
    _need_gpu()
    specs = _layout(precision)[0]
    merged = _run(precision, 2)
    for i in range(len(specs)):
        alone = _run(precision, 2, models=[i])
        assert np.array_equal(_bits(merged[0][:, i]), _bits(alone[0][:, 0])), f"model {i}: losses"
        for a, b in zip(merged[1][i], alone[1][i]):
            assert np.array_equal(_bits(a), _bits(b)), f"model {i}: params"
        for a, b in zip(merged[2][i], alone[2][i]):
            assert np.array_equal(_bits(a), _bits(b)), f"model {i}: grads"


def test_grouped_per_model_labels():
    """Per-model label rows of different lengths (each model's own batch) equal
    the model alone with those labels, and match the oracle."""
    _need_gpu()
    specs, group_of, inputs, model_wl, _ = _layout("bf16")

    def labels(i, s):
        rng = np.random.default_rng([7, i, s])
        return rng.integers(0, specs[i]["num_classes"], size=inputs[group_of[i]][0]).astype(np.int32)

    merged = _run("bf16", 2, labels=labels)
    for i in (0, 3, 6):
        alone = _run("bf16", 2, models=[i], labels=labels)
        assert np.array_equal(_bits(merged[0][:, i]), _bits(alone[0][:, 0]))
        orc, spread = _oracle("bf16", i, 2, labels)
        compare_run(model_wl[i], (merged[0][:, i:i + 1], {0: merged[1][i]}, {0: merged[2][i]}), {0: orc}, [0],
                    spread={0: spread})


def test_group_errors_change_nothing():
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    specs, group_of, inputs, model_wl, group_wl = _layout("f32")
    with pytest.raises(U.UnError) as e:
        U.Hybrid(specs, None, None, "f32", inputs=inputs, group_of=[0] * (len(specs) - 1) + [5])
    assert e.value.status == U.UN_ERR_RANGE
    with pytest.raises(U.UnError) as e:                     # group 2 holds no model
        U.Hybrid(specs[:4], None, None, "f32", inputs=inputs, group_of=group_of[:4])
    assert e.value.status == U.UN_ERR_INVALID
    with U.Hybrid(specs, None, None, "f32", inputs=inputs, group_of=group_of) as h:
        x, y = W.make_batch(group_wl[0], 0)
        with pytest.raises(U.UnError) as e:
            h.load_batch(x, y)                              # no group given, several groups
        assert e.value.status == U.UN_ERR_INVALID
        h.load_batch(x, y, group=0)
        with pytest.raises(U.UnError) as e:
            h.step(LR)                                      # groups 1 and 2 not loaded yet
        assert e.value.status == U.UN_ERR_STATE
        x1, y1 = W.make_batch(group_wl[1], 0)
        h.load_batch(x1, y1, group=1)
        x2, y2 = W.make_batch(group_wl[2], 0)
        bad = y2.copy()
        bad[0] = 13                                         # the flat group has 13 classes
        with pytest.raises(U.UnError) as e:
            h.load_batch(x2, bad, group=2)
        assert e.value.status == U.UN_ERR_RANGE
        with pytest.raises(U.UnError) as e:
            h.load_batch(x2, y2, group=3)
        assert e.value.status == U.UN_ERR_RANGE
        h.load_batch(x2, y2, group=2)
        losses = h.step(LR)
        assert np.all(np.isfinite(losses))


def test_grouped_plan_bytes_equal_the_arena_and_active_sets():
    """un_plan_bytes_grouped equals the arena; a whole group sitting out leaves
    its models untouched and the others equal to their alone runs."""
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    from paper_2408_01331_amd.unifiednn import flatten_params
    specs, group_of, inputs, model_wl, group_wl = _layout("bf16")
    plan, _ = U.un_plan_bytes(specs, None, None, "bf16", inputs=inputs, group_of=group_of)
    with U.Hybrid(specs, None, None, "bf16", inputs=inputs, group_of=group_of) as h:
        assert U.un_arena_bytes(h.ctx) == plan
        for i in range(len(specs)):
            h.set_params(i, flatten_params(_theta(model_wl[i])))
        h.set_active(np.array([g != 1 for g in group_of]))
        for s in range(2):
            for g in range(3):
                x, y = W.make_batch(group_wl[g], s)
                h.load_batch(x, y, group=g)
            losses = h.step(LR)
            assert np.all(np.isnan(losses[[i for i in range(len(specs)) if group_of[i] == 1]]))
        for i in range(len(specs)):
            p = h.get_params(i)
            if group_of[i] == 1:
                assert np.array_equal(_bits(p), _bits(flatten_params(_theta(model_wl[i]))))
            else:
                alone = _run("bf16", 2, models=[i])
                assert np.array_equal(_bits(p), _bits(flatten_params(alone[1][i])))
