"""Scheduling policies of the fused step as active-set sequences (CPU only).

Each expected sequence is written out from the policy's definition (Trainer
section of the paper): who trains in which step, and in what order the models
are released.
"""
import numpy as np
import pytest

from paper_2408_01331_amd.scheduler import Schedule, train


def _runs(masks):
    """Compress a mask sequence into [(active tuple, number of steps)]."""
    out = []
    for m in masks:
        a = tuple(int(i) for i in np.flatnonzero(m))
        if out and out[-1][0] == a:
            out[-1] = (a, out[-1][1] + 1)
        else:
            out.append((a, 1))
    return out


def _finish_order(s):
    while not s.done():
        s.advance(s.mask())
    return s.finished


def test_fused_keeps_every_unfinished_model():
    s = Schedule([1, 2, 3], steps_per_epoch=2, policy="fused")
    assert _runs(s.plan()) == [((0, 1, 2), 2), ((1, 2), 2), ((2,), 2)]
    assert _finish_order(s) == [0, 1, 2]


def test_fcfs_runs_in_arrival_order_to_completion():
    s = Schedule([2, 1, 1], steps_per_epoch=2, policy="fcfs")
    assert _runs(s.plan()) == [((0,), 4), ((1,), 2), ((2,), 2)]
    assert _finish_order(s) == [0, 1, 2]
    # two at a time: a freed slot goes to the next arrival
    s2 = Schedule([2, 1, 1], steps_per_epoch=2, policy="fcfs", capacity=2)
    assert _runs(s2.plan()) == [((0, 1), 2), ((0, 2), 2)]


def test_priority_lowest_value_first_ties_take_epoch_turns():
    s = Schedule([1, 2, 1, 1], steps_per_epoch=2, policy="priority", priorities=[2, 1, 1, 3])
    # models 1 and 2 (priority 1) alternate one epoch each, then 0, then 3
    assert _runs(s.plan()) == [((1,), 2), ((2,), 2), ((1,), 2), ((0,), 2), ((3,), 2)]
    assert _finish_order(s) == [2, 1, 0, 3]


def test_shortest_job_first_by_epochs_and_by_size():
    s = Schedule([3, 1, 2], steps_per_epoch=1, policy="sjf", sjf_by="epochs")
    assert _runs(s.plan()) == [((1,), 1), ((2,), 2), ((0,), 3)]
    s2 = Schedule([1, 1, 1], steps_per_epoch=1, policy="sjf", sjf_by="size", sizes=[10, 30, 20])
    assert _finish_order(s2) == [0, 2, 1]
    with pytest.raises(ValueError):
        Schedule([1], 1, policy="sjf", sjf_by="size")


def test_round_robin_turns_of_one_epoch():
    s = Schedule([2, 1, 2], steps_per_epoch=2, policy="rr")
    assert _runs(s.plan()) == [((0,), 2), ((1,), 2), ((2,), 2), ((0,), 2), ((2,), 2)]
    assert _finish_order(s) == [1, 0, 2]


def test_zero_epoch_jobs_and_bad_arguments():
    s = Schedule([0, 1], steps_per_epoch=3, policy="rr")
    assert _runs(s.plan()) == [((1,), 3)]
    with pytest.raises(ValueError):
        Schedule([1], 1, policy="lottery")
    with pytest.raises(ValueError):
        Schedule([1], 0)


class _FakeHybrid:
    """Records what train() asks of the library."""

    def __init__(self, n):
        self.n, self.sets, self.steps, self.loaded = n, [], 0, []

    def set_active(self, m):
        self.sets.append(tuple(np.flatnonzero(m)))

    def load_batch(self, x, y):
        self.loaded.append(x)

    def step(self, lr):
        self.steps += 1
        return np.zeros(self.n, dtype=np.float32)

    def get_params(self, i):
        return np.full(3, float(i), dtype=np.float32)


def test_train_sets_the_active_set_only_on_change_and_releases_in_order():
    h = _FakeHybrid(3)
    released = []
    losses = train(h, Schedule([1, 2, 1], steps_per_epoch=2, policy="fcfs"), lambda s: (s, None), 0.1,
                   on_release=lambda i, p: released.append((i, float(p[0]))))
    assert h.steps == 8 and losses.shape == (8, 3)
    assert h.sets == [(0,), (1,), (2,)]
    assert h.loaded == list(range(8))            # the step index picks the batch
    assert released == [(0, 0.0), (1, 1.0), (2, 2.0)]
