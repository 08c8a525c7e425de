"""Schedules of the fused step: which sub-models train in each step.

The paper's trainer (Trainer section) lets the provider pick a scheduling
policy; a sub-model whose training is done is handed back through the Model
Separator while the others go on. With one fused step for many models, a
policy is a sequence of active sets (`un_set_active`): the kernels never
change, only which models are in the step. Policies:

* ``fused``    - every unfinished model in every step (the hybrid training
  algorithm, Algorithm 2, with all sub-models at once);
* ``fcfs``     - first come first serve: models in arrival order (index
  order), ``capacity`` at a time, each to completion;
* ``priority`` - the lowest priority value first; models of equal priority
  take turns of one epoch (round robin among them);
* ``sjf``      - shortest job first, the job length being the number of
  epochs (``sjf_by="epochs"``) or the model size (``sjf_by="size"``); a
  started job runs to completion, ties go in arrival order;
* ``rr``       - round robin: the unfinished models take turns of one epoch.

A job is ``epochs[i]`` epochs of ``steps_per_epoch`` steps. ``capacity`` is
how many models a non-fused policy runs at once (the paper's policies run one
at a time: capacity 1). This is host-side bookkeeping only; `train` drives a
`Hybrid` with it.
"""
from __future__ import annotations

import numpy as np

POLICIES = ("fused", "fcfs", "priority", "sjf", "rr")


class Schedule:
    def __init__(self, epochs, steps_per_epoch, policy="fused", priorities=None, sizes=None, sjf_by="epochs",
                 capacity=1):
        if policy not in POLICIES:
            raise ValueError(f"unknown policy {policy!r}; one of {POLICIES}")
        if steps_per_epoch <= 0 or capacity <= 0:
            raise ValueError("steps_per_epoch and capacity must be positive")
        self.n = len(epochs)
        self.policy = policy
        self.spe = int(steps_per_epoch)
        self.capacity = int(capacity)
        self.remaining = np.array([int(e) * self.spe for e in epochs], dtype=np.int64)
        if np.any(self.remaining < 0):
            raise ValueError("negative epoch count")
        self.priorities = np.zeros(self.n) if priorities is None else np.asarray(priorities, dtype=np.float64)
        if policy == "sjf":
            if sjf_by == "epochs":
                self.length = np.asarray(epochs, dtype=np.float64)
            elif sjf_by == "size":
                if sizes is None:
                    raise ValueError("sjf_by='size' needs sizes")
                self.length = np.asarray(sizes, dtype=np.float64)
            else:
                raise ValueError("sjf_by is 'epochs' or 'size'")
        self.queue = [i for i in range(self.n) if self.remaining[i] > 0]  # turn order (rr, priority ties)
        self.running = []      # models of the current turn / current jobs
        self.turn_left = 0     # steps left in the current turn (rr, priority)
        self.finished = []     # released models, in order
        self.steps = 0

    def done(self):
        return not np.any(self.remaining > 0)

    def _unfinished(self):
        return [i for i in range(self.n) if self.remaining[i] > 0]

    def _pick(self):
        """Choose the running set when the current one has to be replaced."""
        live = self._unfinished()
        k = self.capacity
        if self.policy == "fcfs":
            keep = [i for i in self.running if self.remaining[i] > 0]
            fresh = [i for i in live if i not in keep]
            self.running = keep + fresh[:k - len(keep)]
        elif self.policy == "sjf":
            keep = [i for i in self.running if self.remaining[i] > 0]
            fresh = sorted((i for i in live if i not in keep), key=lambda i: (self.length[i], i))
            self.running = keep + fresh[:k - len(keep)]
        elif self.policy == "rr":
            self.queue = [i for i in self.queue if self.remaining[i] > 0]
            self.running = self.queue[:k]
            self.turn_left = self.spe
        elif self.policy == "priority":
            best = min(self.priorities[i] for i in live)
            self.queue = [i for i in self.queue if self.remaining[i] > 0]
            group = [i for i in self.queue if self.priorities[i] == best]
            self.running = group[:k]
            self.turn_left = self.spe

    def mask(self):
        """Active set of the next step (all False once every job is done)."""
        m = np.zeros(self.n, dtype=bool)
        if self.done():
            return m
        if self.policy == "fused":
            return self.remaining > 0
        need = not self.running or any(self.remaining[i] == 0 for i in self.running)
        if self.policy in ("rr", "priority") and self.turn_left == 0:
            need = True
        if need:
            self._pick()
        m[self.running] = True
        return m

    def advance(self, mask):
        """Account one step of the models in `mask`; return the models it finished."""
        mask = np.asarray(mask, dtype=bool)
        self.remaining[mask] -= 1
        self.steps += 1
        done_now = [i for i in np.flatnonzero(mask) if self.remaining[i] == 0]
        self.finished.extend(int(i) for i in done_now)
        if self.policy in ("rr", "priority"):
            self.turn_left -= 1
            if self.turn_left == 0 or any(self.remaining[i] == 0 for i in self.running):
                # end of the turn (one epoch) or a job done: the turn's models go
                # to the back of the queue
                ran = [i for i in self.queue if i in self.running]
                self.queue = [i for i in self.queue if i not in self.running] + ran
                self.turn_left = 0
        return [int(i) for i in done_now]

    def plan(self):
        """The whole sequence of active sets (a copy of this schedule is run)."""
        import copy
        s = copy.deepcopy(self)
        out = []
        while not s.done():
            m = s.mask()
            out.append(m)
            s.advance(m)
        return out


def train(hybrid, schedule, batch, lr, on_release=None):
    """Run `schedule` on a `Hybrid`: before each step the active set is set
    when it changed, the step's batch is loaded (`batch(step)` -> (x, y)), and
    every model that finishes is released: `on_release(i, params)` receives its
    parameters while the others go on. Returns the per-step losses [steps, N]
    (NaN for models outside the step's active set)."""
    losses, cur = [], None
    while not schedule.done():
        m = schedule.mask()
        if cur is None or not np.array_equal(m, cur):
            hybrid.set_active(m)
            cur = m
        x, y = batch(schedule.steps)
        hybrid.load_batch(x, y)
        losses.append(hybrid.step(lr))
        for i in schedule.advance(m):
            if on_release is not None:
                on_release(i, hybrid.get_params(i))
    return np.array(losses)
