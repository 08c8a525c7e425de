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

# The gate: max relative error on losses and parameters.
TOL = {"f32": 1e-4, "bf16": 2e-2}
# Extras (one step: update and gradient, max relative error; k steps: update
# theta_k - theta_0 and the last step's gradient, Frobenius) are bounded by
# SPREAD_FACTOR times the distance between the oracle and the same oracle
# evaluated in fp32 arithmetic (oracle_spread), and never tighter than a floor:
# the gate for one step; EXTRA_FLOOR for k steps, the scale of a trajectory in
# which one discrete decision (a bf16 rounding of a stored value, a ReLU / pool
# decision) went the other way once: at batch 6 one flipped bf16 value moves a
# weight gradient by about 2^-8 / sqrt(6), and the runs part from there.
SPREAD_FACTOR = 4.0
EXTRA_FLOOR = {"f32": 1e-2, "bf16": 0.1}
UPDATE_TOL = EXTRA_FLOOR
# A flipped decision changes one sample's contribution to the flagged unit's
# gradient; those parameters are held to this bound instead of the strict one.
FLAGGED_TOL = 1e-2


def theta0(wl, i):
    return W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)


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


def perturb_ulp(params, seed):
    """Move a random half of the elements of each tensor by one fp32 ulp, up or
    down at random (an input transformation: no arithmetic of the method)."""
    rng = np.random.default_rng([seed, 77])
    out = []
    for p in params:
        p = np.asarray(p, dtype=np.float32)
        pick = rng.random(p.shape) < 0.5
        toward = np.where(rng.random(p.shape) < 0.5, np.inf, -np.inf).astype(np.float32)
        out.append(np.where(pick, np.nextafter(p, toward), p).astype(np.float32))
    return out


def oracle_spread(spec, th0, batches, lr, mode, flags, ref):
    """How far two evaluation orders the reading allows lie apart: the oracle's
    trajectory with fp32 accumulation (float32 BLAS) against its reference
    trajectory `ref` = (losses, params, grads) (fp64 accumulation), over the
    units `flags` never marked, per tensor: the parameters ("param", max
    relative error), the update theta_k - theta_0 and the last step's
    gradient, each as max relative error ("update", "grad") and as Frobenius
    relative error ("update_fro", "grad_fro"), and the loss of every step. In bf16 the stored values are discrete (roundings, ReLU and
    pool decisions), so differences of order compound over the steps; this is
    the scale below which no evaluation order can be told apart from another."""
    loss_a, p, g = oracle.train(spec, th0, batches, lr, mode, None, "f32")
    masks = flagged_masks(spec, ref[1], flags)
    out = {"param": [], "update": [], "grad": [], "update_fro": [], "grad_fro": []}
    for t, (a, b, ga, gb, t0) in enumerate(zip(p, ref[1], g, ref[2], th0)):
        keep = ~masks[t]
        ua, ub = np.asarray(a, np.float64) - t0, np.asarray(b, np.float64) - t0
        out["param"].append(tensor_err(a, b, keep))
        out["update"].append(tensor_err(ua, ub, keep))
        out["grad"].append(tensor_err(ga, gb, keep))
        out["update_fro"].append(fro_err(ua[keep], ub[keep]))
        out["grad_fro"].append(fro_err(np.asarray(ga)[keep], np.asarray(gb)[keep]))
    out["loss"] = (np.abs(np.asarray(loss_a) - ref[0]) / np.abs(ref[0])).tolist()
    return out


def run_oracle(wl, steps, models, lr=None, theta=None, spread=False):
    """Each listed model trained alone by the oracle. Returns {i: (losses,
    params, grads, flags)} or, with spread, also {i: oracle_spread}."""
    lr = wl.lr if lr is None else lr
    batches = [W.make_batch(wl, s) for s in range(steps)]
    th = {i: (theta0(wl, i) if theta is None or i not in theta else theta[i]) for i in range(wl.n_models)}
    out = oracle.train_models(wl.specs, th, batches, lr, wl.precision, models=models, with_flags=True)
    if not spread:
        return out
    sp = {i: oracle_spread(wl.specs[i], th[i], batches, lr, wl.precision, out[i][3], out[i][:3]) for i in out}
    return out, sp


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


def _param_layers(spec):
    """The parameterised layers of a spec, in order, as dicts:
    ``out_w``/``out_b``: the tensors whose row / entry u produce output unit u
    (feature, channel or token feature); ``in_w``: the weight that reads the
    layer's input (an attention layer reads through its in-projection and
    produces through its out-projection); ``view``: how the previous
    parameterised layer's unit u appears in this layer's input -
    "same" (column / input channel u), "img_flat" (a flattened NCHW channel:
    a block of H*W features), "seq_flat" (a flattened [T, d] sequence: every
    d-th feature) or "unflat" (flat features read as tokens of d: feature
    u mod d); ``skip_end``: for a layer whose output starts a residual block,
    the index of the block's last parameterised layer (its output is the sum)
    and the view of the skip."""
    L = spec["layers"]
    ents, t, state, view = [], 0, "flat", "same"
    for li, layer in enumerate(L):
        op = layer[0]
        if op in ("linear", "conv", "attention"):
            n = 4 if op == "attention" else 2
            ents.append({"li": li, "in_w": t, "out_w": t + n - 2, "out_b": t + n - 1, "view": view})
            t += n
            view = "same"
            if op == "conv":
                state = "image"
        elif op == "flatten":
            if state != "flat":
                view = "img_flat" if state == "image" else "seq_flat"
            state = "flat"
        elif op == "unflatten":
            if ents:
                view = "unflat"
            state = "seq"
    for k, e in enumerate(ents):
        nxt = ents[k + 1]["li"] if k + 1 < len(ents) else len(L)
        rb = [j for j in range(e["li"] + 1, nxt) if L[j][0] == "res_begin"]
        if rb:
            j, depth = rb[0] + 1, 1
            while depth:
                depth += {"res_begin": 1, "res_end": -1}.get(L[j][0], 0)
                j += 1
            last = max(q for q, f in enumerate(ents) if f["li"] < j - 1)
            sv = "unflat" if any(L[q][0] == "unflatten" for q in range(e["li"] + 1, rb[0])) else "same"
            e["skip_end"] = (last, sv)
    return ents


def _units_seen(view, u, n_prev, w_next):
    """Input columns (or channels) of the next weight that read unit u of a
    layer with n_prev output units, under the view between them."""
    if view == "same":
        return [u]
    if view == "unflat":
        return [u % w_next.shape[1]]
    if view == "seq_flat":
        return list(range(u, w_next.shape[1], n_prev))
    S = w_next.shape[1] // n_prev                      # img_flat: channel u's block of features
    return list(range(u * S, (u + 1) * S))


def flagged_masks(spec, params, flags):
    """Per tensor, True where a parameter belongs to, or reads, an output unit
    whose ReLU or max-pool decision the oracle found ill-conditioned in fp32.
    For a flagged unit u of a layer: the layer's weight row and bias entry u,
    and the next layer's weights that read u (its input column or channel, the
    features of a flattened channel or token feature, or the token feature of
    a flat unit read as a sequence). When the layer's output is the input of
    a residual block, u also reaches the block's sum through the skip: the
    block's last layer's rows of u are marked, and so is everything that reads
    the sum's unit, recursively (back-to-back blocks). After a flip those
    parameters drift apart for the remaining steps."""
    masks = [np.zeros(np.shape(p), dtype=bool) for p in params]
    ents = _param_layers(spec)
    by_out = {e["out_w"]: k for k, e in enumerate(ents)}

    def mark(k, u, seen):
        if (k, u) in seen:
            return
        seen.add((k, u))
        e = ents[k]
        n_prev = np.shape(params[e["out_w"]])[0]
        masks[e["out_w"]][u, ...] = True
        masks[e["out_b"]][u] = True
        if k + 1 < len(ents):
            nx = ents[k + 1]
            for col in _units_seen(nx["view"], u, n_prev, params[nx["in_w"]]):
                masks[nx["in_w"]][:, col, ...] = True
        if "skip_end" in e:
            last, sv = e["skip_end"]
            mark(last, u % np.shape(params[ents[last]["out_w"]])[0] if sv == "unflat" else u, seen)

    for wi, units in flags.items():
        for u in units:
            mark(by_out[wi], u, set())
    return masks


def fro_err(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a - b))


def _losses(wl, losses_g, i, losses_o, tol, worst):
    le = np.abs(losses_g[:, i] - losses_o) / np.abs(losses_o)
    worst["loss"] = max(worst["loss"], float(le.max()))
    assert le.max() <= tol, f"model {i}: loss rel err {le.max():.3g} > {tol} ({losses_g[:, i]} vs {losses_o})"


def compare_step(wl, gpu, orc, models, tol=None, spread=None, extra_floor=None):
    """One step from identical parameters: per-tensor max relative error <= tol
    on losses and parameters (the gate), and on updates and gradients, except
    at units whose ReLU / max-pool decision the oracle flagged as
    ill-conditioned in fp32 (those parameters within FLAGGED_TOL; their
    gradients are not compared). With `spread` (oracle_spread of one step), an
    update or gradient tensor whose two evaluation orders already lie further
    apart than tol / SPREAD_FACTOR is held to SPREAD_FACTOR times that spread.
    extra_floor replaces tol as the extras' floor (a network in which a single
    discrete decision going the other way moves a gradient row by more than
    the gate)."""
    tol = TOL[wl.precision] if tol is None else tol
    losses_g, params_g, grads_g = gpu
    assert losses_g.shape[0] == 1
    worst = {"loss": 0.0, "param": 0.0, "update": 0.0, "grad": 0.0, "flagged_param": 0.0, "flagged_units": 0}
    for i in models:
        losses_o, params_o, grads_o, flags = orc[i]
        _losses(wl, losses_g, i, losses_o, tol, worst)
        th0 = theta0(wl, i)
        fm = flagged_masks(wl.specs[i], params_o, flags)
        worst["flagged_units"] += sum(len(v) for v in flags.values())
        for t, (pg, po, gg, go) in enumerate(zip(params_g[i], params_o, grads_g[i], grads_o)):
            strict = ~fm[t]
            for key, a, b in (("param", pg, po), ("update", pg - th0[t], po - th0[t]), ("grad", gg, go)):
                e = tensor_err(a, b, strict)
                worst[key] = max(worst[key], e)
                bound = tol
                if key != "param":
                    floor = tol if extra_floor is None else max(tol, extra_floor)
                    bound = floor
                    if spread is not None and i in spread:
                        bound = max(floor, SPREAD_FACTOR * spread[i][key][t])
                assert e <= bound, f"model {i} tensor {t}: {key} err {e:.3g} > {bound:.3g}"
            if fm[t].any():
                ef = tensor_err(pg, po, fm[t])
                worst["flagged_param"] = max(worst["flagged_param"], ef)
                assert ef <= FLAGGED_TOL, f"model {i} tensor {t}: flagged param err {ef:.3g}"
    return worst


def extra_bound(wl, spread, i, key, t):
    """Bound of a multi-step extra (update or gradient, Frobenius) of model i's
    tensor t: SPREAD_FACTOR times the spread between the oracle's two
    evaluation orders, never below EXTRA_FLOOR."""
    floor = EXTRA_FLOOR[wl.precision]
    if spread is None or i not in spread or not spread[i]:
        return floor
    return max(floor, SPREAD_FACTOR * spread[i][key][t])


def compare_run(wl, gpu, orc, models, tol=None, spread=None):
    """k free-running steps against the oracle that trained each model alone.

    The gate (the stated metric): losses within `tol` relative error at every
    step, and every parameter tensor within max |a - b| / max |b| <= tol over
    the units the oracle never flagged in any step; the parameters of flagged
    units within FLAGGED_TOL (once an fp32 decision has legitimately come out
    the other way, the trajectories of those units part by more than rounding).
    A model in which the oracle flagged any decision may fork there as a
    whole (the flipped unit feeds every later layer in the following steps):
    with `spread` given, its never-flagged parameters are held to
    max(tol, SPREAD_FACTOR * the oracle's own parameter spread), the distance
    its two evaluation orders reach when they fork the same way.

    Extras, Frobenius relative error over the never-flagged units: the update
    theta_k - theta_0 and the last step's gradient, each within extra_bound
    (the spread of the oracle's two evaluation orders, oracle_spread, measured
    in the same test when `spread` is given). Returns the worst values, and
    for the extras their worst ratio to the bound."""
    tol = TOL[wl.precision] if tol is None else tol
    losses_g, params_g, grads_g = gpu
    worst = {"loss": 0.0, "param_max": 0.0, "flagged_param": 0.0, "update_fro": 0.0, "grad_fro": 0.0,
             "extra_vs_bound": 0.0, "flagged_units": 0}
    for i in models:
        losses_o, params_o, grads_o, flags = orc[i]
        _losses(wl, losses_g, i, losses_o, tol, worst)
        worst["flagged_units"] += sum(len(v) for v in flags.values())
        th0 = theta0(wl, i)
        fm = flagged_masks(wl.specs[i], params_o, flags)
        forked = any(len(v) for v in flags.values())
        for t, (pg, po, gg, go) in enumerate(zip(params_g[i], params_o, grads_g[i], grads_o)):
            keep = ~fm[t]
            e = tensor_err(pg, po, keep)
            worst["param_max"] = max(worst["param_max"], e)
            pbound = tol
            if forked and spread is not None and i in spread and "param" in spread[i]:
                pbound = max(tol, SPREAD_FACTOR * spread[i]["param"][t])
            assert e <= pbound, f"model {i} tensor {t}: param max rel err {e:.3g} > {pbound:.3g} (never-flagged units)"
            if fm[t].any():
                ef = tensor_err(pg, po, fm[t])
                worst["flagged_param"] = max(worst["flagged_param"], ef)
                assert ef <= FLAGGED_TOL, f"model {i} tensor {t}: flagged param err {ef:.3g} > {FLAGGED_TOL}"
            ug, uo = np.asarray(pg - th0[t])[keep], np.asarray(po - th0[t])[keep]
            for key, err in (("update_fro", fro_err(ug, uo)),
                             ("grad_fro", fro_err(np.asarray(gg)[keep], np.asarray(go)[keep]))):
                bound = extra_bound(wl, spread, i, key, t)
                worst[key] = max(worst[key], err)
                worst["extra_vs_bound"] = max(worst["extra_vs_bound"], err / bound)
                assert err <= bound, f"model {i} tensor {t}: {key} {err:.3g} > {bound:.3g}"
    return worst
