"""Memory estimate (un_plan_bytes, host only) and admission of models onto a
GPU budget. CPU: the planner runs without a device."""
import numpy as np
import pytest

from paper_2408_01331_amd import admission as A
from paper_2408_01331_amd import unifiednn as U
from paper_2408_01331_amd import workloads as W


def _need_lib():
    try:
        U.lib()
    except OSError as e:  # not built
        pytest.skip(f"library not built: {e}")


def _params(wl, idx):
    return sum(int(np.prod(s)) for i in idx for s, _ in W.param_shapes(wl.specs[i], wl.in_shape))


@pytest.mark.parametrize("name", ["mlp8", "lenet4", "cifar16", "mlp64", "resnet8"])
def test_fused_footprint_is_one_input_plus_the_models(name):
    _need_lib()
    wl = W.get(name)
    r = A.memory_report(wl.specs, wl.batch, wl.in_shape, wl.precision)
    # the shared input is held once instead of N times
    assert r["fused_bytes"] < r["separate_total"]
    in_bytes = wl.batch * int(np.prod(wl.in_shape)) * 4          # the fp32 staging copy alone
    assert r["saved_bytes"] >= (wl.n_models - 1) * in_bytes
    # every parameter has at least its fp32 master weight and its gradient
    assert r["fused_bytes"] >= 8 * _params(wl, range(wl.n_models))
    # the optimizer state is two fp32 values per parameter (rows padded to 8)
    p = _params(wl, range(wl.n_models))
    assert 8 * p <= r["optimizer_state_bytes"] <= 8 * p * 1.25 + 256 * 4 * 8 * wl.n_models


def test_footprint_grows_with_every_model():
    _need_lib()
    wl = W.get("mlp8")
    prev = 0
    for k in range(1, wl.n_models + 1):
        b = A.plan_bytes(wl.specs[:k], wl.batch, wl.in_shape, wl.precision)
        assert b > prev
        prev = b
    assert A.plan_bytes(wl.specs, wl.batch, wl.in_shape, wl.precision, optimizer_state=True) > prev


def test_admission_fcfs_and_size_order():
    _need_lib()
    wl = W.get("mlp8")
    sizes = [A.plan_bytes([s], wl.batch, wl.in_shape, wl.precision) for s in wl.specs]
    three = A.plan_bytes(wl.specs[:3], wl.batch, wl.in_shape, wl.precision)
    got, used = A.admit(wl.specs, wl.batch, wl.in_shape, wl.precision, three)
    assert got[:3] == [0, 1, 2] and used <= three
    # a later, smaller model may still fit after a larger one was refused
    for i in got[3:]:
        assert A.plan_bytes([wl.specs[j] for j in sorted(got)], wl.batch, wl.in_shape, wl.precision) <= three
    # smallest first admits at least as many models under the same budget
    by_size = sorted(range(wl.n_models), key=lambda i: sizes[i])
    got_s, _ = A.admit(wl.specs, wl.batch, wl.in_shape, wl.precision, three, order=by_size)
    assert len(got_s) >= len(got)
    assert A.admit(wl.specs, wl.batch, wl.in_shape, wl.precision, min(sizes) - 1) == ([], 0)


def test_plan_errors_match_create_validation():
    _need_lib()
    with pytest.raises(U.UnError) as e:
        U.un_plan_bytes([{"layers": [("linear", 10)], "num_classes": 5}], 8, (16,), "f32")
    assert e.value.status in (U.UN_ERR_INVALID, U.UN_ERR_UNSUPPORTED)
