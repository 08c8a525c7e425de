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
        "kernels_sha256": hashlib.sha256(
            open(os.path.join(ROOT, "paper_2408_01331_amd", "csrc", "kernels.hip"), "rb").read()).hexdigest(),
        "dispatches": [len(f), len(w)],
        "fetch_kib_per_dispatch": fkib, "write_kib_per_dispatch": wkib,
        "copy_fetch_factor": ff, "copy_write_factor": wf,
        "hbm_bytes_per_launch": fkib * 1024.0 / ff + wkib * 1024.0 / wf,
    }
    with open(a.out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    t = sub.add_parser("traffic")
    for k in ("kernel", "workload", "fetch", "write", "copy_fetch", "copy_write", "out"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    a = ap.parse_args()
    if a.cmd == "stats":
        stats(a.dir)
    else:
        traffic(a)


if __name__ == "__main__":
    main()
