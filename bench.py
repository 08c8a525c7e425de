"""Benchmark of the fused N-model training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload mlp64] [--also cifar16,resnet8]
    python bench.py --copy-probe      # calibration copy for the HBM byte counters only

Prints ONE JSON line. A step is one fused forward + softmax-CE + backward +
SGD pass of all N models over one resident synthetic batch (un_step with no
loss read-back). `value` is model-samples/s = N * batch * K / elapsed.

Alongside: the dominant kernel class against its roofline (algorithmic FLOPs
or bytes per launch divided by its HIP-event time on the library's stream;
HBM traffic per launch from the committed counter summary under profiles/
when it was taken on the current kernels), the other workloads named by
--also, the same N models stepped as N separate one-model contexts back to
back (the unfused baseline), and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2408_01331_amd import workloads as W  # noqa: E402

PEAK = {"bf16_mfma_tflops": 2500.0, "f32_mfma_tflops": 157.3, "hbm_gbs": 8000.0}
KCLASS = ["gemm_fwd", "gemm_bwd", "conv_fwd", "conv_dgrad", "conv_wgrad", "ce", "sgd", "other", "attn"]


# ---------------------------------------------------------------------------
# Algorithmic work per step (the definition, not what the kernels happen to do)
# ---------------------------------------------------------------------------
def algorithmic_work(wl):
    """Algorithmic FLOPs and HBM bytes per step and kernel class, from the layer shapes.

    FLOPs: 2 per multiply-add of forward, weight gradient and data gradient
    (none for the first layer), with no padding counted. Bytes: the minimum
    under fusion, each tensor moved once per use: a stored activation is
    written once and read by the next layer's forward and by this layer's
    weight gradient; its gradient likewise; the weights the products read are
    read once per use (forward, data gradient); the fused update reads and
    writes the fp32 master (8 B per parameter) plus the bf16 copy (2 B) in bf16
    mode. A residual block adds one read of its input x (the forward of its
    last layer) and one of its output gradient (the data gradient of its first
    layer). Returns (flops, bytes, n_params)."""
    B = wl.batch
    es = 2 if wl.precision == "bf16" else 4
    upd = 10 if wl.precision == "bf16" else 8
    flops = {k: 0.0 for k in KCLASS}
    nbytes = {k: 0.0 for k in KCLASS}
    n_params = 0
    for spec in wl.specs:
        shape = tuple(wl.in_shape)
        first = True
        layers = spec["layers"]
        for li, layer in enumerate(layers):
            op = layer[0]
            ends = li + 1 < len(layers) and layers[li + 1][0] == "res_end"
            begins = li > 0 and layers[li - 1][0] == "res_begin"
            if op in ("linear", "attention"):
                # a sequence (T, d): token-wise products over B * T rows
                R, K = (B * shape[0], shape[1]) if len(shape) == 2 else (B, int(np.prod(shape)))
                last = li == len(layers) - 1
                # (N, rows stored fp32?) per projection: Linear, or in- and out-projection
                projs = [(layer[1], last)] if op == "linear" else [(3 * K, False), (K, False)]
                for pj, (N, fp32_out) in enumerate(projs):
                    f = 2.0 * R * K * N
                    flops["gemm_fwd"] += f
                    nbytes["gemm_fwd"] += R * K * es + N * K * es + N * 4 + R * N * (4 if fp32_out else es)
                    flops["gemm_bwd"] += f                               # weight gradient + update
                    nbytes["gemm_bwd"] += R * N * es + R * K * es + (N * K + N) * upd
                    if not (first and pj == 0):                          # data gradient
                        flops["gemm_bwd"] += f
                        nbytes["gemm_bwd"] += R * N * es + N * K * es + R * K * es
                    n_params += K * N + N
                if op == "attention":
                    T, d = shape
                    # core: S = Q K^T and A = P V forward; dP, dQ, dK, dV backward
                    flops["attn"] += 4.0 * B * T * T * d + 8.0 * B * T * T * d
                    nbytes["attn"] += B * T * 3 * d * es + B * T * d * es + B * T * T * 4          # forward, P fp32
                    nbytes["attn"] += B * T * 3 * d * es * 2 + B * T * d * es + B * T * T * 4      # backward
                else:
                    N = layer[1]
                    if last:                                             # softmax-CE: logits in, dZ out
                        nbytes["ce"] += B * N * 4 + B * N * es
                    shape = (shape[0], N) if len(shape) == 2 else (N,)
                out_el = R * shape[-1]
                nbytes["gemm_fwd"] += out_el * es if ends else 0         # skip input
                nbytes["gemm_bwd"] += R * K * es if begins else 0        # skip gradient
                first = False
            elif op == "conv":
                C, H, Wd = shape
                O, k, pad = layer[1], layer[2], layer[3]
                OH, OW = H + 2 * pad - k + 1, Wd + 2 * pad - k + 1
                pool = li + 1 < len(layers) and layers[li + 1][0] == "pool" or \
                    li + 2 < len(layers) and layers[li + 1][0] == "relu" and layers[li + 2][0] == "pool"
                out_el = B * (OH // 2) * (OW // 2) * O if pool else B * OH * OW * O
                out_b = out_el * (es + 1 if pool else es)                # pooled values + argmax byte
                in_b = B * H * Wd * C * es
                w_b = O * C * k * k * es
                f = 2.0 * B * OH * OW * O * C * k * k
                flops["conv_fwd"] += f
                nbytes["conv_fwd"] += in_b + w_b + out_b
                flops["conv_wgrad"] += f
                nbytes["conv_wgrad"] += out_b + in_b
                nbytes["other"] += (O * C * k * k + O) * upd           # update (split-K reduction kernel)
                if not first:
                    flops["conv_dgrad"] += f
                    nbytes["conv_dgrad"] += out_b + w_b + in_b
                nbytes["conv_fwd"] += out_el * es if ends else 0         # skip input
                nbytes["conv_dgrad"] += in_b if begins else 0            # skip gradient
                n_params += O * C * k * k + O
                shape = (O, OH, OW)
                first = False
            elif op == "pool":
                C, H, Wd = shape
                shape = (C, H // 2, Wd // 2)
            elif op == "flatten":
                shape = (int(np.prod(shape)),)
            elif op == "unflatten":
                shape = (layer[1], int(np.prod(shape)) // layer[1])
    return flops, nbytes, n_params


def run_gpu(wl, steps, warmup, repeats=0):
    """Time `steps` steps after `warmup`; then `repeats` more windows of the
    same steps (their ms per step, a noise indicator beside the reported
    window) and a pass with per-launch HIP events."""
    import torch
    from paper_2408_01331_amd import unifiednn as U

    torch.cuda.set_device(0)
    h = U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision)
    for i in range(wl.n_models):
        h.set_params(i, U.flatten_params(W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)))
    x, y = W.make_batch(wl, 0)
    h.load_batch(x, y)                       # resident in HBM before timing
    for _ in range(warmup):
        h.step(wl.lr, losses=False)
    h.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        h.step(wl.lr, losses=False)
    h.sync()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    windows = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(steps):
            h.step(wl.lr, losses=False)
        h.sync()
        torch.cuda.synchronize()
        windows.append((time.perf_counter() - t1) / steps * 1e3)

    # the same K steps again with every launch bracketed by HIP events on the
    # library's stream (per-kernel durations for the roofline)
    U.un_profile_enable(h.ctx, True)
    for _ in range(steps):
        h.step(wl.lr, losses=False)
    h.sync()
    kern = {}
    for k, name in enumerate(KCLASS):
        ms, n = U.un_profile_read(h.ctx, k)
        if n:
            kern[name] = {"ms_per_step": ms / steps, "launches_per_step": n / steps, "avg_launch_ms": ms / n}
    U.un_profile_enable(h.ctx, False)
    losses = h.step(wl.lr, losses=True)
    arena = U.un_arena_bytes(h.ctx)
    h.close()
    if repeats:
        return elapsed, kern, losses, arena, windows
    return elapsed, kern, losses, arena


def run_unfused(wl, steps, warmup):
    """N separate one-model contexts stepped back to back (same kernels, no
    fusion): (a) each model's step waited for before the next one starts, and
    (b) all contexts on one stream, every step enqueued without host
    synchronisation (ordered by the stream alone). Returns (seconds of (a),
    seconds of (b), summed arena bytes)."""
    import torch
    from paper_2408_01331_amd import unifiednn as U

    hs = []
    x, y = W.make_batch(wl, 0)
    for i in range(wl.n_models):
        h = U.Hybrid([wl.specs[i]], wl.batch, wl.in_shape, wl.precision)
        h.set_params(0, U.flatten_params(W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)))
        h.load_batch(x, y)
        hs.append(h)
    for _ in range(warmup):
        for h in hs:
            h.step(wl.lr, losses=False)
    for h in hs:
        h.sync()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        for h in hs:
            h.step(wl.lr, losses=False)
            h.sync()        # back to back: each model's step completes before the next starts
    torch.cuda.synchronize()
    synced = time.perf_counter() - t0
    stream = torch.cuda.Stream()
    for h in hs:
        h.set_stream(stream.cuda_stream)
    for h in hs:
        h.step(wl.lr, losses=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        for h in hs:
            h.step(wl.lr, losses=False)
    torch.cuda.synchronize()
    queued = time.perf_counter() - t0
    arena = sum(U.un_arena_bytes(h.ctx) for h in hs)
    for h in hs:
        h.set_stream(None)
        h.close()
    return synced, queued, arena


def run_latency(wl, steps, warmup):
    """ms per step of a launch-latency-bound workload, enqueued step by step
    (un_step) and replayed from one captured graph (un_graph_step)."""
    import torch
    from paper_2408_01331_amd import unifiednn as U

    torch.cuda.set_device(0)
    out = {}
    with U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision) as h:
        for i in range(wl.n_models):
            h.set_params(i, U.flatten_params(W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)))
        x, y = W.make_batch(wl, 0)
        h.load_batch(x, y)
        h.capture(wl.lr)
        for mode in ("eager", "graph"):
            run = (lambda: h.step(wl.lr, losses=False)) if mode == "eager" else (lambda: h.replay(losses=False))
            for _ in range(warmup):
                run()
            h.sync()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                run()
            h.sync()
            torch.cuda.synchronize()
            out[f"ms_per_step_{mode}"] = (time.perf_counter() - t0) / steps * 1e3
    out["model_samples_per_s_graph"] = wl.n_models * wl.batch / (out["ms_per_step_graph"] / 1e3)
    out["steps"] = steps
    return out


def copy_probe(nbytes=1 << 30, reps=4):
    """A plain device-to-device copy of known size (calibrates the HBM byte
    counters: FETCH_SIZE / WRITE_SIZE read for it vs. the bytes it moves)."""
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)      # one elementwise kernel: reads and writes nbytes
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": nbytes, "copy_probe_bytes_written": nbytes, "copies": reps}),
          flush=True)


def source_digest():
    """sha256 of the kernel, planner and interface sources (identifies the
    launches a counter summary was taken on)."""
    from paper_2408_01331_amd.profile_summary import sources_digest
    return sources_digest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed counter
    summary, or None when there is none or the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None, None
    rec = json.load(open(path))
    if rec.get("sources_sha256") != source_digest():
        return None, path
    return rec["hbm_bytes_per_launch"], path


def cpu_baseline(wl, budget_s=12.0, single_thread_s=6.0):
    """The oracle (as it stands) on a bounded sample: whole one-model steps on
    the same batch, models taken in turn (cycling) until the budget is spent;
    then the same with the BLAS library limited to one thread."""
    import oracle

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    x, y = W.make_batch(wl, 0)
    params = {}
    t0 = time.perf_counter()
    done = 0
    while True:
        i = done % wl.n_models
        if i not in params:
            params[i] = W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)
        oracle.step(wl.specs[i], params[i], x, y, wl.lr, wl.precision)
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    one = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t1, n1 = time.perf_counter(), 0
            while True:
                i = n1 % wl.n_models
                oracle.step(wl.specs[i], params.setdefault(i, W.init_params(wl.specs[i], wl.in_shape, wl.seed, i,
                                                                            wl.init)), x, y, wl.lr, wl.precision)
                n1 += 1
                if time.perf_counter() - t1 > single_thread_s:
                    break
            one = {"value": n1 * wl.batch / (time.perf_counter() - t1), "cores": 1,
                   "sample": f"{n1} one-model steps with BLAS limited to 1 thread"}
    except Exception:
        pass
    return {"value": done * wl.batch / el, "unit": "model-samples/s",
            "cores": blas_threads if blas_threads else cores, "host_cpus": cores, "kind": "oracle",
            "sample": f"{done} one-model steps (models 0..{min(done, wl.n_models) - 1} of {wl.n_models} in turn, "
                      f"batch {wl.batch}) in {el:.1f} s, numpy fp64 with BLAS threads={blas_threads}",
            "single_thread": one}


def measure(wl, steps, warmup, repeats=0):
    """Time `steps` fused steps of workload `wl`; per-kernel rooflines. With
    repeats, that many more windows of the same steps are timed and reported
    beside the first (median, min, max ms per step): the run-to-run spread."""
    flops, nbytes, n_params = algorithmic_work(wl)
    out = run_gpu(wl, steps, warmup, repeats)
    elapsed, kern, losses, arena = out[:4]
    ms_step = elapsed / steps * 1e3
    value = wl.n_models * wl.batch / (ms_step / 1e3)
    mfma_peak = PEAK["bf16_mfma_tflops"] if wl.precision == "bf16" else PEAK["f32_mfma_tflops"]
    total_flops = sum(flops.values())
    # One entry per kernel: the forward and the backward grouped GEMM are two
    # instantiations of gemm_kernel (row-major operands / k-major operands
    # with the update in the epilogue), timed and bounded apart.
    sym = {"gemm_fwd": ["gemm_fwd"], "gemm_bwd": ["gemm_bwd"], "conv_fwd": ["conv_fwd"],
           "conv_dgrad": ["conv_dgrad"], "conv_wgrad": ["conv_wgrad"], "ce": ["ce"], "sgd": ["sgd"],
           "other": ["other"], "attn": ["attn"]}
    per_sym = {}
    for name, classes in sym.items():
        ms = sum(kern[c]["ms_per_step"] for c in classes if c in kern)
        n = sum(kern[c]["launches_per_step"] for c in classes if c in kern)
        if n:
            per_sym[name] = {"ms_per_step": ms, "launches_per_step": n, "avg_launch_ms": ms / n,
                             "flops_per_step": sum(flops[c] for c in classes),
                             "bytes_per_step": sum(nbytes[c] for c in classes)}
    dom = max(per_sym, key=lambda k: per_sym[k]["ms_per_step"])
    d = per_sym[dom]
    # The kernel's bound: its algorithmic arithmetic intensity against the
    # ridge point of the peaks. achieved = algorithmic work of one launch (the
    # step's work / launches per step) over the average launch duration, both
    # from HIP events on the library's stream.
    ridge = mfma_peak * 1e12 / (PEAK["hbm_gbs"] * 1e9)
    ai = d["flops_per_step"] / d["bytes_per_step"] if d["bytes_per_step"] else float("inf")
    launch_s = d["avg_launch_ms"] / 1e3
    if ai < ridge:
        achieved = d["bytes_per_step"] / d["launches_per_step"] / launch_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    else:
        achieved = d["flops_per_step"] / d["launches_per_step"] / launch_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": mfma_peak, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    kname = f"{dom}_{wl.precision}"
    # counter summaries are named for the kernel and the workload's short name (mlp64, cifar16, ...)
    traffic, tpath = measured_traffic(kname, wl.name.split("_")[0])
    roof["traffic"] = traffic
    roof["traffic_unit"] = "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE scaled by a plain copy)"
    roof["kernel"] = dom
    roof["avg_launch_ms"] = d["avg_launch_ms"]
    roof["launches_per_step"] = d["launches_per_step"]
    roof["algorithmic_flops_per_launch"] = d["flops_per_step"] / d["launches_per_step"]
    roof["algorithmic_bytes_per_launch"] = d["bytes_per_step"] / d["launches_per_step"]
    roof["arith_intensity"] = ai
    roof["ridge"] = ridge
    roof["mfma_frac"] = d["flops_per_step"] / d["launches_per_step"] / launch_s / 1e12 / mfma_peak
    per_kernel = {}
    for k, v in kern.items():
        e = dict(v)
        if flops.get(k):
            e["achieved_tflops"] = flops[k] / (v["ms_per_step"] / 1e3) / 1e12
        if nbytes.get(k):
            e["achieved_gbs"] = nbytes[k] / (v["ms_per_step"] / 1e3) / 1e9
        per_kernel[k] = e
    return {
        "value": value, "ms_per_step": ms_step, "steps": steps, "warmup": warmup,
        "config": {"workload": wl.name, "description": wl.description, "n_models": wl.n_models,
                   "batch": wl.batch, "in_shape": list(wl.in_shape), "params": n_params,
                   "parallelism": "none (one GPU, N models fused)"},
        "dtype": wl.precision,
        "mfma_util_step": total_flops / (ms_step / 1e3) / 1e12 / mfma_peak,
        "train_gflop_per_step": total_flops / 1e9,
        "roofline": roof, "kernels": per_kernel, "arena_bytes": arena,
        "final_losses_mean": float(np.mean(losses)),
        **({"repeat_windows_ms_per_step": {"n": repeats, "median": float(np.median(out[4])),
                                           "min": float(np.min(out[4])), "max": float(np.max(out[4]))}}
           if repeats else {}),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mlp64", choices=list(W.WORKLOADS))
    ap.add_argument("--also", default="cifar16,resnet8,attn8",
                    help="comma-separated workloads also timed and reported under other_workloads ('' for none)")
    ap.add_argument("--latency", default="mlp2,mlp8,lenet4",
                    help="launch-latency-bound workloads timed with and without graph replay ('' for none)")
    ap.add_argument("--repeats", type=int, default=3,
                    help="further timing windows of the headline workload, reported as their median / min / max")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy (calibration run for the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}); the N-model step is a "
              "single-GPU path and multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe()
        return

    wl = W.get(args.workload)
    rec = measure(wl, args.steps, args.warmup, repeats=args.repeats)
    out = {
        "metric": "model-samples/sec (N x batch / step time) at 1 GPU",
        "value": rec["value"],
        "unit": "model-samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": rec["dtype"],
        "data": "synthetic (seeded N(0,1) inputs, uniform labels; random-init weights)",
    }
    out.update({k: rec[k] for k in ("config", "mfma_util_step", "train_gflop_per_step", "roofline", "kernels",
                                    "arena_bytes", "final_losses_mean")})
    if "repeat_windows_ms_per_step" in rec:
        out["repeat_windows_ms_per_step"] = rec["repeat_windows_ms_per_step"]
    others = {}
    for name in [w for w in args.also.split(",") if w and w != wl.name]:
        owl = W.get(name)
        others[name] = measure(owl, args.steps, args.warmup)
    if others:
        out["other_workloads"] = others
    lat = {}
    for name in [w for w in args.latency.split(",") if w]:
        lat[name] = run_latency(W.get(name), args.steps, args.warmup)
    if lat:
        out["latency_workloads"] = lat
    if not args.no_unfused:
        usteps = max(3, args.steps // 5)
        ue, uq, uarena = run_unfused(wl, usteps, 2)
        out["unfused_baseline"] = {
            "value": wl.n_models * wl.batch / (ue / usteps), "unit": "model-samples/s",
            "ms_per_round": ue / usteps * 1e3, "arena_bytes_sum": uarena,
            "what": f"{wl.n_models} one-model contexts, each stepped and synchronised in turn",
            "queued": {"value": wl.n_models * wl.batch / (uq / usteps), "ms_per_round": uq / usteps * 1e3,
                       "what": "the same contexts on one stream, all steps enqueued without host synchronisation"}}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
