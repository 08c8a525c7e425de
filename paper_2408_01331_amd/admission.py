"""Memory estimate and admission of models onto one GPU, before anything is
created on the device.

The paper's trainer assigns a hybrid to a GPU with enough free memory and
sizes the hybrid as the largest of its sub-models, because its scheduler
trains them one after another (Trainer section, memory requirement). A fused
step holds all of its models at once: its footprint is the planner's arena -
the shared input batch once, plus every model's parameters, copies,
activations and gradients - which `un_plan_bytes` computes exactly on the
host. Admission is then a packing question: which models, in the scheduler's
order, fit the budget together.
"""
from __future__ import annotations

from .unifiednn import un_plan_bytes


def plan_bytes(specs, batch, in_shape, precision, optimizer_state=False):
    """Device bytes of one context for ``specs`` (plus the optimizer state
    allocation when ``optimizer_state``)."""
    arena, state = un_plan_bytes(list(specs), batch, in_shape, precision)
    return arena + (state if optimizer_state else 0)


def memory_report(specs, batch, in_shape, precision):
    """Fused footprint against N separate contexts (one per model, each with
    its own copy of the input batch)."""
    fused, state = un_plan_bytes(list(specs), batch, in_shape, precision)
    separate = [un_plan_bytes([s], batch, in_shape, precision)[0] for s in specs]
    return {"fused_bytes": fused, "separate_bytes": separate, "separate_total": sum(separate),
            "saved_bytes": sum(separate) - fused, "optimizer_state_bytes": state}


def admit(specs, batch, in_shape, precision, budget_bytes, order=None, optimizer_state=False):
    """Greedy admission in ``order`` (default: arrival order, i.e. first come
    first serve; pass a size order for shortest-job-first): each model joins
    if the fused context of the admitted set plus it still fits
    ``budget_bytes``; a model that does not fit is skipped and later ones are
    still tried. Returns (admitted indices in admission order, their bytes)."""
    order = list(range(len(specs))) if order is None else list(order)
    taken, used = [], 0
    for i in order:
        cand = taken + [i]
        b = plan_bytes([specs[j] for j in sorted(cand)], batch, in_shape, precision, optimizer_state)
        if b <= budget_bytes:
            taken, used = cand, b
    return taken, used
