"""Summaries of rocprofv3 output for the committed profiles.

    python -m paper_2408_01331_amd.profile_summary stats DIR
        kernel table (calls, average/min/max microseconds, share) from the
        *_kernel_stats.csv of a `rocprofv3 --kernel-trace --stats` run

    python -m paper_2408_01331_amd.profile_summary traffic --kernel NAME --workload W \\
        --fetch DIR --write DIR --copy-fetch DIR --copy-write DIR --out FILE
        HBM bytes per launch of the kernels whose name contains NAME, from one
        `rocprofv3 --pmc FETCH_SIZE` and one `--pmc WRITE_SIZE` run of the
        benchmark, each scaled by what the same counter reads for a plain
        elementwise copy of known size (`bench.py --copy-probe`)

    python -m paper_2408_01331_amd.profile_summary pmc --trace DIR --counters DIR [DIR ...]
        per kernel instantiation: dispatches, average kernel time (from the
        kernel trace), and per dispatch the counters of `rocprofv3 --pmc`
        runs, with MFMA throughput from the MFMA op counters, MFMA-busy and
        wait shares, and the HBM request mix (32 / 64 / 128-byte reads)
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


SOURCES = ("paper_2408_01331_amd/csrc/kernels.hip", "paper_2408_01331_amd/csrc/un_api.cpp",
           "paper_2408_01331_amd/csrc/internal.h", "include/unifiednn.h")


def sources_digest():
    """sha256 over the kernel, planner and interface sources, in a fixed order:
    a counter summary holds for the launches those sources produce."""
    h = hashlib.sha256()
    for rel in SOURCES:
        h.update(rel.encode())
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    return h.hexdigest()


def _one(pattern):
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        sys.exit(f"no file matches {pattern}")
    return files[0]


def stats(d):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*kernel_stats.csv")))))
    print("| kernel | calls | avg µs | min µs | max µs | share |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        name = r["Name"].replace("unsigned short", "bf16")
        print(f"| `{name[:80]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
              f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | {float(r['Percentage']):.1f} % |")


def per_dispatch(d, counter):
    """{dispatch id: (kernel name, counter value summed over its rows)}"""
    acc = collections.defaultdict(float)
    names = {}
    for r in csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))):
        if r["Counter_Name"] != counter:
            continue
        acc[r["Dispatch_Id"]] += float(r["Counter_Value"])
        names[r["Dispatch_Id"]] = r["Kernel_Name"]
    return {k: (names[k], v) for k, v in acc.items()}


def copy_factor(d, counter, nbytes):
    """Counter KiB per byte moved, from the largest elementwise dispatch of the copy probe."""
    disp = per_dispatch(d, counter)
    vals = [v for n, v in disp.values() if "elementwise" in n]
    if not vals:
        sys.exit(f"no elementwise copy dispatch in {d}")
    return max(vals) * 1024.0 / nbytes


def traffic(a):
    probe_bytes = 1 << 30
    ff = copy_factor(a.copy_fetch, "FETCH_SIZE", probe_bytes)
    wf = copy_factor(a.copy_write, "WRITE_SIZE", probe_bytes)
    f = [v for n, v in per_dispatch(a.fetch, "FETCH_SIZE").values() if a.kernel in n]
    w = [v for n, v in per_dispatch(a.write, "WRITE_SIZE").values() if a.kernel in n]
    if not f or not w:
        sys.exit(f"no dispatch of {a.kernel}")
    fkib, wkib = sum(f) / len(f), sum(w) / len(w)
    rec = {
        "kernel": a.kernel, "workload": a.workload,
        "sources_sha256": sources_digest(),
        "dispatches": [len(f), len(w)],
        "fetch_kib_per_dispatch": fkib, "write_kib_per_dispatch": wkib,
        "copy_fetch_factor": ff, "copy_write_factor": wf,
        "hbm_bytes_per_launch": fkib * 1024.0 / ff + wkib * 1024.0 / wf,
    }
    with open(a.out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def per_kernel(d):
    """{kernel name: {counter: [value per dispatch]}} of a --pmc run."""
    rows = collections.defaultdict(lambda: collections.defaultdict(float))
    names = {}
    for r in csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))):
        rows[r["Dispatch_Id"]][r["Counter_Name"]] += float(r["Counter_Value"])
        names[r["Dispatch_Id"]] = r["Kernel_Name"]
    out = collections.defaultdict(lambda: collections.defaultdict(list))
    for disp, cs in rows.items():
        for c, v in cs.items():
            out[names[disp]][c].append(v)
    return out


def short(name):
    return name.replace("unsigned short", "bf16").split("(")[0].replace("void ", "")


def pmc(a):
    """MFMA / wait / request-mix table per kernel instantiation."""
    trace = list(csv.DictReader(open(_one(os.path.join(a.trace, "**", "*kernel_stats.csv")))))
    avg_ns = {r["Name"]: float(r["AverageNs"]) for r in trace}
    merged = collections.defaultdict(dict)
    for d in a.counters:
        for k, cs in per_kernel(d).items():
            for c, vals in cs.items():
                merged[k][c] = sum(vals) / len(vals)
    peak_bf16 = 2500.0  # TFLOP/s, dense bf16 MFMA
    rows = []
    for k, cs in merged.items():
        if not any(x in k for x in a.match):
            continue
        t = avg_ns.get(k)
        rec = {"kernel": short(k), "avg_us": t / 1e3 if t else None}
        rec.update({c: v for c, v in sorted(cs.items())})
        mops = cs.get("SQ_INSTS_VALU_MFMA_MOPS_BF16")
        if mops is not None and t:
            rec["mfma_tflops"] = mops * 512 / (t * 1e-9) / 1e12
            rec["mfma_frac_bf16_peak"] = rec["mfma_tflops"] / peak_bf16
        wave = cs.get("SQ_WAVE_CYCLES")
        if wave:
            for c in ("SQ_WAIT_ANY", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_VMEM", "SQ_VALU_MFMA_BUSY_CYCLES"):
                if c in cs:
                    rec[c + "/SQ_WAVE_CYCLES"] = cs[c] / wave
        waves = cs.get("SQ_WAVES")
        if waves and "SQ_INSTS_VALU" in cs:
            # vector instructions per wave, and the time the whole dispatch's
            # vector instructions take to issue: a wave64 instruction occupies
            # its SIMD for 4 cycles; 1024 SIMDs at 2.4 GHz
            rec["valu_per_wave"] = cs["SQ_INSTS_VALU"] / waves
            rec["valu_issue_us"] = cs["SQ_INSTS_VALU"] * 4 / (1024 * 2.4e9) * 1e6
            if t:
                rec["valu_issue_frac"] = rec["valu_issue_us"] / (t / 1e3)
            if "SQ_INSTS_SALU" in cs:
                rec["salu_per_wave"] = cs["SQ_INSTS_SALU"] / waves
            if "SQ_INSTS_MFMA" in cs:
                rec["mfma_insts_per_wave"] = cs["SQ_INSTS_MFMA"] / waves
        if cs.get("SQ_BUSY_CYCLES") and "SQ_VALU_MFMA_BUSY_CYCLES" in cs:
            rec["MFMA_BUSY/SQ_BUSY"] = cs["SQ_VALU_MFMA_BUSY_CYCLES"] / cs["SQ_BUSY_CYCLES"]
        rd = cs.get("TCC_EA0_RDREQ_sum")
        if rd:
            b128 = cs.get("TCC_BUBBLE_sum", 0.0)
            b32 = cs.get("TCC_EA0_RDREQ_32B_sum", 0.0)
            rec["read_req_mix_32_64_128"] = [b32 / rd, (rd - b32 - b128) / rd, b128 / rd]
            rec["read_bytes_from_requests"] = b32 * 32 + (rd - b32 - b128) * 64 + b128 * 128
        rows.append(rec)
    rows.sort(key=lambda r: -(r["avg_us"] or 0))
    print(json.dumps(rows, indent=1))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    m = sub.add_parser("pmc")
    m.add_argument("--trace", required=True)
    m.add_argument("--counters", nargs="+", required=True)
    m.add_argument("--match", nargs="+", default=["gemm_kernel", "conv_", "reduce_kernel", "elementwise"])
    t = sub.add_parser("traffic")
    for k in ("kernel", "workload", "fetch", "write", "copy_fetch", "copy_write", "out"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    a = ap.parse_args()
    if a.cmd == "stats":
        stats(a.dir)
    elif a.cmd == "pmc":
        pmc(a)
    else:
        traffic(a)


if __name__ == "__main__":
    main()
