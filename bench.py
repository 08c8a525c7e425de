"""Benchmark of the fused N-model training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload mlp64]

Prints ONE JSON line. A step is one fused forward + softmax-CE + backward +
SGD pass of all N models over one resident synthetic batch (un_step with no
loss read-back). `value` is model-samples/s = N * batch * K / elapsed.

Alongside: the dominant kernel class against its roofline (algorithmic FLOPs
or bytes per step divided by its HIP-event time on the library's stream), the
same N models stepped as N separate one-model contexts back to back (the
unfused baseline), and the CPU oracle timed on a bounded sample.
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
KCLASS = ["gemm_fwd", "gemm_bwd", "conv_fwd", "conv_dgrad", "conv_wgrad", "ce", "sgd", "other"]


# ---------------------------------------------------------------------------
# Algorithmic work per step (the definition, not what the kernels happen to do)
# ---------------------------------------------------------------------------
def algorithmic_work(wl):
    """FLOPs per kernel class and SGD bytes, per step, from the layer shapes."""
    B = wl.batch
    flops = {k: 0.0 for k in KCLASS}
    n_params = 0
    for spec in wl.specs:
        shape = tuple(wl.in_shape)
        first = True
        for layer in spec["layers"]:
            op = layer[0]
            if op == "linear":
                K = int(np.prod(shape))
                N = layer[1]
                flops["gemm_fwd"] += 2.0 * B * K * N
                flops["gemm_bwd"] += 2.0 * B * K * N          # wgrad
                if not first:
                    flops["gemm_bwd"] += 2.0 * B * K * N      # dgrad
                n_params += K * N + N
                shape = (N,)
                first = False
            elif op == "conv":
                C, H, Wd = shape
                O, k, pad = layer[1], layer[2], layer[3]
                OH, OW = H + 2 * pad - k + 1, Wd + 2 * pad - k + 1
                f = 2.0 * B * OH * OW * O * C * k * k
                flops["conv_fwd"] += f
                flops["conv_wgrad"] += f
                if not first:
                    flops["conv_dgrad"] += f
                n_params += O * C * k * k + O
                shape = (O, OH, OW)
                first = False
            elif op == "pool":
                C, H, Wd = shape
                shape = (C, H // 2, Wd // 2)
            elif op == "flatten":
                shape = (int(np.prod(shape)),)
    # SGD per parameter: read master + grad, write master (12 B), then the copies
    # the GEMMs read: bf16 shadow (2 B) and transposed copy (2 B) in bf16 mode,
    # transposed fp32 copy (4 B) in fp32 mode.
    per_param = 12 + (4 if wl.precision == "bf16" else 4)
    return flops, n_params, n_params * per_param


def run_gpu(wl, steps, warmup):
    import torch
    from paper_2408_01331_amd import unifiednn as U

    torch.cuda.set_device(0)
    h = U.Hybrid(wl.specs, wl.batch, wl.in_shape, wl.precision)
    for i in range(wl.n_models):
        h.set_params(i, U.flatten_params(W.init_params(wl.specs[i], wl.in_shape, wl.seed, i)))
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
    return elapsed, kern, losses, arena


def run_unfused(wl, steps, warmup):
    """N separate one-model contexts stepped back to back (same kernels, no fusion)."""
    import torch
    from paper_2408_01331_amd import unifiednn as U

    hs = []
    x, y = W.make_batch(wl, 0)
    for i in range(wl.n_models):
        h = U.Hybrid([wl.specs[i]], wl.batch, wl.in_shape, wl.precision)
        h.set_params(0, U.flatten_params(W.init_params(wl.specs[i], wl.in_shape, wl.seed, i)))
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
    elapsed = time.perf_counter() - t0
    arena = sum(U.un_arena_bytes(h.ctx) for h in hs)
    for h in hs:
        h.close()
    return elapsed, arena


def cpu_baseline(wl, budget_s=15.0):
    """The oracle (as it stands) on a bounded sample: whole models, one step each."""
    import oracle

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    x, y = W.make_batch(wl, 0)
    t0 = time.perf_counter()
    done = 0
    for i in range(wl.n_models):
        p = W.init_params(wl.specs[i], wl.in_shape, wl.seed, i)
        oracle.step(wl.specs[i], p, x, y, wl.lr, wl.precision)
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": done * wl.batch / el, "unit": "model-samples/s",
            "cores": blas_threads if blas_threads else cores, "host_cpus": cores, "kind": "oracle",
            "sample": f"one step of models 0..{done - 1} of {wl.n_models} (batch {wl.batch}), "
                      f"{el:.1f} s, numpy fp64 with BLAS threads={blas_threads}"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mlp64", choices=list(W.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}); the N-model step is a "
              "single-GPU path and multi-GPU runs are not part of this build.", file=sys.stderr)
        sys.exit(2)

    wl = W.get(args.workload)
    flops, n_params, sgd_bytes = algorithmic_work(wl)
    elapsed, kern, losses, arena = run_gpu(wl, args.steps, args.warmup)
    ms_step = elapsed / args.steps * 1e3
    value = wl.n_models * wl.batch / (ms_step / 1e3)

    mfma_peak = PEAK["bf16_mfma_tflops"] if wl.precision == "bf16" else PEAK["f32_mfma_tflops"]
    total_flops = sum(flops.values())
    # Kernel symbols: the grouped GEMM serves both gemm_fwd and gemm_bwd launches.
    sym = {"gemm": ["gemm_fwd", "gemm_bwd"], "conv_fwd": ["conv_fwd"], "conv_dgrad": ["conv_dgrad"],
           "conv_wgrad": ["conv_wgrad"], "ce": ["ce"], "sgd": ["sgd"], "other": ["other"]}
    per_sym = {}
    for name, classes in sym.items():
        ms = sum(kern[c]["ms_per_step"] for c in classes if c in kern)
        n = sum(kern[c]["launches_per_step"] for c in classes if c in kern)
        if n:
            per_sym[name] = {"ms_per_step": ms, "launches_per_step": n, "avg_launch_ms": ms / n,
                             "flops_per_step": sum(flops[c] for c in classes)}
    dom = max((k for k in per_sym if k != "other"), key=lambda k: per_sym[k]["ms_per_step"])
    d = per_sym[dom]
    if dom in ("sgd", "ce"):
        achieved = (sgd_bytes if dom == "sgd" else 0.0) / (d["ms_per_step"] / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    else:
        achieved = d["flops_per_step"] / (d["ms_per_step"] / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": mfma_peak, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    roof["kernel"] = dom
    roof["avg_launch_ms"] = d["avg_launch_ms"]
    per_kernel = {}
    for k, v in kern.items():
        e = dict(v)
        if k == "sgd":
            e["achieved_gbs"] = sgd_bytes / (v["ms_per_step"] / 1e3) / 1e9
        elif flops.get(k):
            e["achieved_tflops"] = flops[k] / (v["ms_per_step"] / 1e3) / 1e12
        per_kernel[k] = e

    out = {
        "metric": "model-samples/sec (N x batch / step time) at 1 GPU",
        "value": value,
        "unit": "model-samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.precision,
        "data": "synthetic (seeded N(0,1) inputs, uniform labels; random-init weights)",
        "config": {"workload": wl.name, "description": wl.description, "n_models": wl.n_models,
                   "batch": wl.batch, "in_shape": list(wl.in_shape), "params": n_params,
                   "parallelism": "none (one GPU, N models fused)"},
        "mfma_util_step": total_flops / (ms_step / 1e3) / 1e12 / mfma_peak,
        "train_gflop_per_step": total_flops / 1e9,
        "roofline": roof,
        "kernels": per_kernel,
        "arena_bytes": arena,
        "final_losses_mean": float(np.mean(losses)),
    }
    if not args.no_unfused:
        ue, uarena = run_unfused(wl, max(3, args.steps // 5), 2)
        usteps = max(3, args.steps // 5)
        out["unfused_baseline"] = {
            "value": wl.n_models * wl.batch / (ue / usteps), "unit": "model-samples/s",
            "ms_per_round": ue / usteps * 1e3, "arena_bytes_sum": uarena,
            "what": f"{wl.n_models} one-model contexts, each stepped and synchronised in turn"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
