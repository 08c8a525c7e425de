"""Shared helpers of the parity tests: run a workload on the GPU library and on
the CPU oracle from the same seeded inputs, and compare them.

Error metrics (fixed here, used by every parity test):
* loss:   |a - b| / |b| per model per step;
* tensor: max |a - b| / max |b| per parameter tensor (element-wise ratios are
  ill-posed for weights near zero), or the Frobenius ratio |a - b| / |b|;
* update: the same metrics on the change theta_k - theta_0, which isolates the
  accumulated gradient from the (identical) starting point.
compare_step and compare_run say which applies where.
"""
import numpy as np

import oracle
from paper_2408_01331_amd import workloads as W

TOL = {"f32": 1e-4, "bf16": 2e-2}
UPDATE_TOL = {"f32": 1e-2, "bf16": 0.2}


def theta0(wl, i):
    return W.init_params(wl.specs[i], wl.in_shape, wl.seed, i)


def run_gpu(wl, steps, lr=None, theta=None, models=None):
    """Train all models of `wl` for `steps` steps on the GPU.

    Returns (losses [steps, N], params {i: [arrays]}, grads {i: [arrays]} of the
    last step) for the models listed (all by default)."""
    from paper_2408_01331_amd.unifiednn import Hybrid, flatten_params, split_params
    lr = wl.lr if lr is None else lr
    idx = range(wl.n_models) if models is None else models
    with Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        h.keep_grads(True)
        for i in range(wl.n_models):
            p = theta0(wl, i) if theta is None or i not in theta else theta[i]
            h.set_params(i, flatten_params(p))
        losses = []
        for s in range(steps):
            x, y = W.make_batch(wl, s)
            h.load_batch(x, y)
            losses.append(h.step(lr))
        params, grads = {}, {}
        for i in idx:
            shapes = [sh for sh, _ in W.param_shapes(wl.specs[i], wl.in_shape)]
            params[i] = split_params(h.get_params(i), shapes)
            grads[i] = split_params(h.get_grads(i), shapes) if steps > 0 else None
    return np.array(losses), params, grads


def run_oracle(wl, steps, models, lr=None, theta=None):
    lr = wl.lr if lr is None else lr
    batches = [W.make_batch(wl, s) for s in range(steps)]
    th = {i: (theta0(wl, i) if theta is None or i not in theta else theta[i]) for i in range(wl.n_models)}
    return oracle.train_models(wl.specs, th, batches, lr, wl.precision, models=models, with_flags=True)


def tensor_err(a, b, mask=None):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b))
    d = np.abs(a - b)
    if mask is not None:
        d = d[mask]
        if d.size == 0:
            return 0.0
    return float(np.max(d) / den) if den > 0 else float(np.max(d))


def flagged_masks(params, flags):
    """Per tensor, True where a parameter belongs to an output unit whose ReLU or
    max-pool decision the oracle found ill-conditioned in fp32: the unit's weight
    row and bias entry, and the next layer's weights that read the unit (its
    input column, input channel, or the block of flattened features of that
    channel). After a flip those parameters drift apart for the remaining steps."""
    masks = [np.zeros(np.shape(p), dtype=bool) for p in params]
    for wi, units in flags.items():
        nxt = wi + 2 if wi + 2 < len(params) else None
        for u in units:
            masks[wi][u, ...] = True
            masks[wi + 1][u] = True
            if nxt is None:
                continue
            Wn = params[nxt]
            if np.ndim(Wn) == 4 or np.ndim(params[wi]) == 2:
                masks[nxt][:, u, ...] = True
            else:  # conv -> flatten -> linear: channel u owns a contiguous block of features
                S = np.shape(Wn)[1] // np.shape(params[wi])[0]
                masks[nxt][:, u * S:(u + 1) * S] = True
    return masks


# A flipped decision changes one sample's contribution to the flagged unit's
# gradient; those parameters are held to this bound instead of the strict one.
FLAGGED_TOL = 1e-2


def fro_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def _losses(wl, losses_g, i, losses_o, tol, worst):
    le = np.abs(losses_g[:, i] - losses_o) / np.abs(losses_o)
    worst["loss"] = max(worst["loss"], float(le.max()))
    assert le.max() <= tol, f"model {i}: loss rel err {le.max():.3g} > {tol} ({losses_g[:, i]} vs {losses_o})"


def compare_step(wl, gpu, orc, models, tol=None):
    """One step from identical parameters: per-tensor max relative error <= tol
    on losses, parameters, updates and gradients, except at units whose ReLU /
    max-pool decision the oracle flagged as ill-conditioned in fp32 (those
    parameters within FLAGGED_TOL; their gradients are not compared)."""
    tol = TOL[wl.precision] if tol is None else tol
    losses_g, params_g, grads_g = gpu
    assert losses_g.shape[0] == 1
    worst = {"loss": 0.0, "param": 0.0, "update": 0.0, "grad": 0.0, "flagged_param": 0.0, "flagged_units": 0}
    for i in models:
        losses_o, params_o, grads_o, flags = orc[i]
        _losses(wl, losses_g, i, losses_o, tol, worst)
        th0 = theta0(wl, i)
        fm = flagged_masks(params_o, flags)
        worst["flagged_units"] += sum(len(v) for v in flags.values())
        for t, (pg, po, gg, go) in enumerate(zip(params_g[i], params_o, grads_g[i], grads_o)):
            strict = ~fm[t]
            for key, a, b in (("param", pg, po), ("update", pg - th0[t], po - th0[t]), ("grad", gg, go)):
                e = tensor_err(a, b, strict)
                worst[key] = max(worst[key], e)
                assert e <= tol, f"model {i} tensor {t}: {key} err {e:.3g} > {tol}"
            if fm[t].any():
                ef = tensor_err(pg, po, fm[t])
                worst["flagged_param"] = max(worst["flagged_param"], ef)
                assert ef <= FLAGGED_TOL, f"model {i} tensor {t}: flagged param err {ef:.3g}"
    return worst


def compare_run(wl, gpu, orc, models, tol=None, update_tol=None):
    """k free-running steps. Once one fp32 decision has legitimately come out the
    other way, the trajectories differ by a few ulps of a single unit, which can
    tip further near-zero decisions; no fp32 order of evaluation can bound the
    per-element error of every parameter after many steps. So:
      losses: max relative error <= tol at every step;
      parameters: Frobenius relative error <= tol per tensor, and per-element
        max relative error <= FLAGGED_TOL (guard against localised gross errors);
      updates theta_k - theta_0 and last-step gradients: Frobenius relative
        error <= update_tol per tensor (UPDATE_TOL by default), over the
        parameters of units the oracle did not flag. A flipped decision at a
        flagged unit changes one sample's share of that unit's gradient; an
        optimizer that normalises the step per element (Adam) turns that into
        a change of the whole step of those parameters, however small the
        share, so their updates are held by the per-element guard only.
    """
    tol = TOL[wl.precision] if tol is None else tol
    # One flipped decision moves its unit's row of one step's update by a few
    # per cent (Frobenius share ~1e-3); bf16 storage adds 1-ulp activation
    # differences that compound over steps. Kernel-level gradient accuracy is
    # held to `tol` by compare_step.
    update_tol = UPDATE_TOL[wl.precision] if update_tol is None else update_tol
    losses_g, params_g, grads_g = gpu
    worst = {"loss": 0.0, "param_fro": 0.0, "param_max": 0.0, "update_fro": 0.0, "grad_fro": 0.0,
             "flagged_units": 0}
    for i in models:
        losses_o, params_o, grads_o, flags = orc[i]
        _losses(wl, losses_g, i, losses_o, tol, worst)
        worst["flagged_units"] += sum(len(v) for v in flags.values())
        th0 = theta0(wl, i)
        fm = flagged_masks(params_o, flags)
        for t, (pg, po, gg, go) in enumerate(zip(params_g[i], params_o, grads_g[i], grads_o)):
            keep = ~fm[t]
            ug, uo = np.asarray(pg - th0[t])[keep], np.asarray(po - th0[t])[keep]
            checks = (("param_fro", fro_err(pg, po), tol), ("param_max", tensor_err(pg, po), FLAGGED_TOL),
                      ("update_fro", fro_err(ug, uo), update_tol),
                      ("grad_fro", fro_err(np.asarray(gg)[keep], np.asarray(go)[keep]), update_tol))
            for key, e, bound in checks:
                worst[key] = max(worst[key], e)
                assert e <= bound, f"model {i} tensor {t}: {key} {e:.3g} > {bound}"
    return worst
