"""GPU: un_step_scratch, the step whose workspace (split-K partials of conv
and long-contraction Linear weight gradients, loss partials) lives in the
library's static device array instead of the
context's arena, for callers that cannot allocate. It must equal un_step bit
for bit, call after call, with a smaller input after a larger one (the array
keeps the previous call's contents), and refuse a context whose workspace
does not fit, changing nothing."""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W
from _parity import theta0

pytestmark = pytest.mark.gpu


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _pair(wl):
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    hs = []
    for _ in range(2):
        h = Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision)
        for i in range(wl.n_models):
            h.set_params(i, flatten_params(theta0(wl, i)))
        h.keep_grads(True)
        hs.append(h)
    return hs


def _compare(wl, ref, got, step):
    for i in range(wl.n_models):
        assert np.array_equal(_bits(ref.get_params(i)), _bits(got.get_params(i))), f"step {step} model {i}: params"
        assert np.array_equal(_bits(ref.get_grads(i)), _bits(got.get_grads(i))), f"step {step} model {i}: grads"


def test_scratch_step_equals_un_step_large_then_small():
    _need_gpu()
    from paper_2408_01331_amd.unifiednn import un_step_scratch
    big = W.shrink(W.get("cifar16"), n_models=4, batch=64)      # bf16 CNNs, several split-K partial sets
    small = W.shrink(W.get("cifar16"), n_models=3, batch=24)    # fewer models, smaller batch and workspace
    lenet = W.get("lenet4")                                     # fp32 CNNs
    attn = W.get("attn8")                                       # split-K Linear weight gradients, attention
    cases = [(attn, _pair(attn)), (big, _pair(big)), (small, _pair(small)), (lenet, _pair(lenet))]
    try:
        for rnd in range(2):
            for wl, (ref, got) in cases:
                x, y = W.make_batch(wl, rnd)
                ref.load_batch(x, y)
                got.load_batch(x, y)
                lr_ = ref.step(wl.lr)
                lg = un_step_scratch(got.ctx, wl.lr, wl.n_models)
                print(f"[{wl.name} b{wl.batch} call {rnd}] losses {lg.tolist()}", flush=True)
                assert np.array_equal(_bits(lr_), _bits(lg)), f"{wl.name} call {rnd}: losses"
                _compare(wl, ref, got, rnd)
    finally:
        for _, hs in cases:
            for h in hs:
                h.close()


def test_scratch_step_refuses_a_workspace_that_does_not_fit():
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    wl = W.get("cifar16")
    with U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        x, y = W.make_batch(wl, 0)
        h.load_batch(x, y)
        before = h.get_params(0)
        with pytest.raises(U.UnError) as e:
            U.un_step_scratch(h.ctx, wl.lr, wl.n_models)
        assert e.value.status == U.UN_ERR_UNSUPPORTED
        assert np.array_equal(_bits(before), _bits(h.get_params(0)))
        h.step(wl.lr)                                           # un_step still works
