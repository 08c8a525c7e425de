"""GPU: the host-side estimate is exactly what a context allocates."""
import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W

pytestmark = pytest.mark.gpu


def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("name", ["mlp2", "mlp8", "lenet4", "cifar16", "mlp64", "resnet8"])
def test_plan_bytes_equal_the_arena_and_the_device_allocation(name):
    torch = _need_gpu()
    from paper_2408_01331_amd import unifiednn as U
    wl = W.get(name)
    arena, state = U.un_plan_bytes(wl.specs, wl.batch, wl.in_shape, wl.precision)
    with U.Hybrid(wl.specs[:1], wl.batch, wl.in_shape, wl.precision):
        pass                                   # runtime set-up outside the measurement
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    with U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        got = U.un_arena_bytes(h.ctx)
        free1, _ = torch.cuda.mem_get_info()
        h.set_optimizer(0, "adam")             # first state-holding optimizer: the state allocation
        free2, _ = torch.cuda.mem_get_info()
    assert got == arena
    # the free-memory counter moves in pages and the runtime's own pieces come
    # and go: equal within a few MiB
    slack = 16 << 20
    assert abs((free0 - free1) - arena) <= slack, (free0 - free1, arena)
    assert abs((free1 - free2) - state) <= slack, (free1 - free2, state)
