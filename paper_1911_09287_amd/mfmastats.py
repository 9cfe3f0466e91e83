"""Matrix-core counters of the contraction kernels from a rocprofv3 counter run.

Measurement tool (not used by the library).  Inputs:

* the ``*_counter_collection.csv`` of ``rocprofv3 --pmc MfmaFlopsF32 MfmaUtil``
  run on ``bench.py`` (every dispatch of the run; all at one compression rate);
* the ``*_kernel_trace.csv`` of a plain ``rocprofv3 --kernel-trace`` run of the
  benchmark's headline command: the kernel durations are taken from there,
  between the first two marker dispatches (the timed steps), because a counter
  run serialises dispatches and stretches them;
* optionally the benchmark's JSON line, for the algorithmic flops per launch
  (8 real flops per complex multiply-add over the kept bins).

For each contraction pass (library kernel name) it prints the dispatches, the
executed matrix-core flops per dispatch (``MfmaFlopsF32`` = 512 x
``SQ_INSTS_VALU_MFMA_MOPS_F32``), their ratio to the algorithmic flops (tile
padding), ``MfmaUtil`` (matrix-core busy cycles over active GPU cycles times
SIMDs, in percent, as rocprofv3 derives it), the average duration, and the
executed and algorithmic rates as fractions of the fp32 matrix-core peak.

    python -m paper_1911_09287_amd.mfmastats counters.csv trace.csv [--bench bench.json]
"""
from __future__ import annotations

import argparse
import csv
import json
import re
from collections import defaultdict

from .kstats import LIBRARY_NAMES, MARKER, short

MFMA_F32_PEAK_TF = 157.3


def counters(path):
    """{dispatch id: (symbol, {counter: value})}."""
    out = {}
    for r in csv.DictReader(open(path)):
        d = out.setdefault(r["Dispatch_Id"], (r["Kernel_Name"], {}))
        d[1][r["Counter_Name"]] = d[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def durations(path):
    """Kernel durations (us) between the first two marker dispatches."""
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    marks = [i for i, r in enumerate(rows) if MARKER in r["Kernel_Name"]]
    if len(marks) < 2:
        raise SystemExit("the kernel trace holds fewer than two marker dispatches")
    return [(r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
            for r in rows[marks[0] + 1:marks[1]]]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("counters")
    ap.add_argument("trace")
    ap.add_argument("--bench", default=None, help="the benchmark's JSON output (last line is used)")
    a = ap.parse_args()
    cnt = counters(a.counters)
    dur = durations(a.trace)
    algo = {}
    if a.bench:
        line = [s for s in open(a.bench).read().splitlines() if s.startswith("{")][-1]
        for k, v in json.loads(line).get("kernels", {}).items():
            if v.get("flops_per_launch"):
                algo[k] = v["flops_per_launch"]
    names = [n for n in LIBRARY_NAMES if n.startswith("contract") and n != "contract_reduce"]
    print("| pass | dispatches (counters / trace) | executed MFMA GFLOP per dispatch | executed / algorithmic | "
          "MfmaUtil % | avg us (trace) | executed TFLOP/s | algorithmic TFLOP/s | algorithmic / 157.3 |")
    print("|---|---|---|---|---|---|---|---|---|")
    for n in names:
        pat = LIBRARY_NAMES[n]
        cs = [c for s, c in cnt.values() if re.search(pat, s)]
        ds = [t for s, t in dur if re.search(pat, s)]
        if not cs or not ds:
            continue
        fl = sum(c.get("MfmaFlopsF32", 0.0) for c in cs) / len(cs)
        ut = sum(c.get("MfmaUtil", 0.0) for c in cs) / len(cs)
        us = sum(ds) / len(ds)
        ex_tf = fl / (us * 1e-6) / 1e12
        al = algo.get(n)
        ratio = f"{fl / al:.3f}" if al else "-"
        al_tf = f"{al / (us * 1e-6) / 1e12:.1f}" if al else "-"
        al_fr = f"{al / (us * 1e-6) / 1e12 / MFMA_F32_PEAK_TF:.3f}" if al else "-"
        print(f"| {n} | {len(cs)} / {len(ds)} | {fl / 1e9:.3f} | {ratio} | {ut:.1f} | {us:.2f} | {ex_tf:.1f} | "
              f"{al_tf} | {al_fr} |")
    print("\n| kernel symbol | dispatches | executed MFMA GFLOP per dispatch | MfmaUtil % |")
    print("|---|---|---|---|")
    per = defaultdict(list)
    for s, c in cnt.values():
        if "MfmaFlopsF32" in c and c["MfmaFlopsF32"] > 0:
            per[short(s)].append(c)
    for s, cs in sorted(per.items()):
        print(f"| {s} | {len(cs)} | {sum(c['MfmaFlopsF32'] for c in cs) / len(cs) / 1e9:.3f} | "
              f"{sum(c.get('MfmaUtil', 0.0) for c in cs) / len(cs):.1f} |")


if __name__ == "__main__":
    main()
