"""GPU: the runtime around the step - a step captured as a HIP graph and
replayed, a caller-supplied stream, batches already in device memory, and the
per-model refresh of the weight copies in un_set_params. Every check is
bitwise against the plain un_step path (same kernels, same order)."""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W
from _parity import theta0

pytestmark = pytest.mark.gpu


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def _case(name):
    if name == "mlp64_8":
        return W.shrink(W.get("mlp64"), n_models=8)
    if name == "cifar16_4":
        return W.shrink(W.get("cifar16"), n_models=4, batch=64)
    return W.get(name)


def _hybrid(wl):
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    h = Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision)
    for i in range(wl.n_models):
        h.set_params(i, flatten_params(theta0(wl, i)))
    h.keep_grads(True)
    return h


def _state(h, wl):
    return [(_bits(h.get_params(i)), _bits(h.get_grads(i))) for i in range(wl.n_models)]


@pytest.mark.parametrize("name", ["mlp2", "lenet4", "mlp64_8", "cifar16_4"])
def test_graph_replays_equal_eager_steps(name):
    """Four replays of one captured step, each on a new batch loaded between
    them (eager work and host synchronisation in between), equal four eager
    steps bit for bit: losses after every step, parameters and gradients at
    the end."""
    _need_gpu()
    wl = _case(name)
    steps = 4
    with _hybrid(wl) as a, _hybrid(wl) as g:
        eager, replay = [], []
        for s in range(steps):
            x, y = W.make_batch(wl, s)
            a.load_batch(x, y)
            eager.append(a.step(wl.lr))
        x, y = W.make_batch(wl, 0)
        g.load_batch(x, y)
        g.capture(wl.lr)
        for s in range(steps):
            x, y = W.make_batch(wl, s)
            g.load_batch(x, y)
            replay.append(g.replay())
            _ = g.get_params(0)                       # eager device work between replays
            assert np.array_equal(_bits(replay[-1]), _bits(eager[s])), f"step {s}: losses"
        for (pa, ga), (pg, gg) in zip(_state(a, wl), _state(g, wl)):
            assert np.array_equal(pa, pg) and np.array_equal(ga, gg)


def test_graph_goes_stale_and_refuses():
    _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    wl = W.get("mlp8")
    with _hybrid(wl) as h:
        with pytest.raises(U.UnError) as e:
            h.replay()
        assert e.value.status == U.UN_ERR_STATE
        x, y = W.make_batch(wl, 0)
        h.load_batch(x, y)
        h.capture(wl.lr)
        h.replay()
        h.keep_grads(False)
        with pytest.raises(U.UnError) as e:
            h.replay()
        assert e.value.status == U.UN_ERR_STATE
        h.keep_grads(True)
        h.replay()
        h.set_active(np.arange(wl.n_models) % 2 == 0)
        with pytest.raises(U.UnError) as e:
            h.replay()
        assert e.value.status == U.UN_ERR_STATE
        h.capture(wl.lr)                                 # recapture with the new active set
        losses = h.replay()
        assert np.all(np.isnan(losses[1::2])) and np.all(np.isfinite(losses[0::2]))
        h.set_optimizer(1, "adam")
        with pytest.raises(U.UnError) as e:
            h.capture(wl.lr)
        assert e.value.status == U.UN_ERR_UNSUPPORTED


def test_contexts_on_one_caller_stream():
    """Two contexts stepped on one PyTorch stream, enqueued without host
    synchronisation, equal the same contexts on their own streams."""
    torch = _need_gpu()
    wl = W.get("mlp8")
    ref, got = [], []
    stream = torch.cuda.Stream()
    for shared in (False, True):
        hs = [_hybrid(wl), _hybrid(wl)]
        if shared:
            for h in hs:
                h.set_stream(stream.cuda_stream)
        for s in range(3):
            x, y = W.make_batch(wl, s)
            for h in hs:
                h.load_batch(x, y)
            for h in hs:
                h.step(wl.lr, losses=False)
        out = ref if not shared else got
        for h in hs:
            out.append(_state(h, wl))
            h.set_stream(None)
            h.close()
    for a, b in zip(ref, got):
        for (pa, ga), (pb, gb) in zip(a, b):
            assert np.array_equal(pa, pb) and np.array_equal(ga, gb)


@pytest.mark.parametrize("name", ["mlp8", "cifar16_4"])
def test_load_batch_device_equals_host_load(name):
    torch = _need_gpu()
    from paper_2408_01331_amd.unifiednn import un_load_batch_device
    wl = _case(name)
    with _hybrid(wl) as a, _hybrid(wl) as d:
        for s in range(2):
            x, y = W.make_batch(wl, s)
            a.load_batch(x, y)
            xd = torch.from_numpy(x).cuda()
            yd = torch.from_numpy(y).cuda()
            torch.cuda.synchronize()                      # the writes are ordered before the call
            un_load_batch_device(d.ctx, xd.data_ptr(), yd.data_ptr())
            la, ld = a.step(wl.lr), d.step(wl.lr)
            assert np.array_equal(_bits(la), _bits(ld))
        for (pa, ga), (pd, gd) in zip(_state(a, wl), _state(d, wl)):
            assert np.array_equal(pa, pd) and np.array_equal(ga, gd)


@pytest.mark.parametrize("name", ["mlp64_8", "cifar16_4"])
def test_set_params_refreshes_only_that_models_copies(name):
    """Setting model 1's parameters mid-run refreshes model 1's bf16 (and conv
    transposed) copies only: the other models continue bit for bit as if
    nothing happened, and model 1 continues as a fresh run from the new values."""
    _need_gpu()
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params
    wl = _case(name)
    new = flatten_params([p * np.float32(0.5) for p in theta0(wl, 1)])
    with _hybrid(wl) as base, _hybrid(wl) as h:
        for s in range(4):
            x, y = W.make_batch(wl, s)
            if s == 2:
                h.set_params(1, new)
            for c in (base, h):
                c.load_batch(x, y)
                c.step(wl.lr)
        sb, sh = _state(base, wl), _state(h, wl)
        for i in range(wl.n_models):
            if i != 1:
                assert np.array_equal(sb[i][0], sh[i][0]), f"model {i}"
        with Hybrid([wl.specs[1]], wl.batch, wl.in_shape, wl.precision) as a:
            a.set_params(0, new)
            for s in (2, 3):
                x, y = W.make_batch(wl, s)
                a.load_batch(x, y)
                a.step(wl.lr)
            assert np.array_equal(_bits(a.get_params(0)), sh[1][0])
