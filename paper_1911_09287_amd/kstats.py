"""Kernel statistics of a benchmark's timed steps from a rocprofv3 kernel trace.

Measurement tool (not used by the library).  Input: the ``*_kernel_trace.csv``
of ``rocprofv3 --kernel-trace`` run on ``bench.py``.  The benchmark launches a
short spin kernel just before and just after each group of timed steps and
each pass with per-kernel events; this tool keeps the dispatches between the
markers of one such group (segment 0: the headline workload's timed steps;
segment 1: its pass with per-kernel events, from which the benchmark's
roofline durations come) and prints, per library kernel name (the names the
library's per-kernel timing reports, each covering one or more template
instantiations), the dispatch count and the average, minimum and maximum
duration, then the same per kernel symbol.  The output is a Markdown table.

    python -m paper_1911_09287_amd.kstats run_kernel_trace.csv [--segment 0]
"""
from __future__ import annotations

import argparse
import csv
import re
from collections import OrderedDict

# library kernel name -> pattern of the kernel symbols launched under it
LIBRARY_NAMES = OrderedDict([
    ("spec_fwd_2d", r"k_fft2_fwd<"),
    ("spec_fwd_filt_2d", r"k_fft2_fwd_filt<"),
    ("spec_inv_2d", r"k_fft2_inv<"),
    ("spec_inv_wgrad_2d", r"k_fft2_inv_wgrad(_wide)?<"),
    ("spec_fwd_1d", r"k_bluestein1k<[02],"),
    ("spec_inv_1d", r"k_bluestein1k<[13],"),
    ("spec_fwd_direct", r"k_spec_fwd<"),
    ("spec_inv_direct", r"k_spec_inv\b"),
    ("spec_filt", r"k_spec_filt<"),
    ("contract_fwd", r"k_cgemm\w*<\d+, \d+, true, true, true, (false|true)(, \d+)?>"),
    ("contract_dgrad", r"k_cgemm\w*<\d+, \d+, true, false, false, (false|true)(, \d+)?>"),
    ("contract_wgrad", r"k_cgemm\w*<\d+, \d+, false, true, true, (false|true)(, \d+)?>"),
    ("contract_bwd", r"k_cgemm_bwd<"),
    ("contract (thin, any pass)", r"k_thin_"),
    ("contract_reduce", r"k_split_reduce"),
    ("wgrad_idft", r"k_wgrad_wide<|k_wgrad_idft<|k_wgrad_tile<"),
    ("wgrad_reduce", r"k_wgrad_reduce"),
])
MARKER = "spin_kernel"


def short(sym):
    s = re.sub(r"^void ", "", sym)
    s = re.sub(r"blc::\(anonymous namespace\)::", "", s)
    s = s.replace("HIP_vector_type<float, 2u>", "float2")
    return re.sub(r"\(.*$", "", s)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace")
    ap.add_argument("--segment", type=int, default=0,
                    help="which marked group (0: the headline's timed steps; 1: its pass with kernel events)")
    a = ap.parse_args()
    rows = sorted(csv.DictReader(open(a.trace)), key=lambda r: int(r["Start_Timestamp"]))
    marks = [i for i, r in enumerate(rows) if MARKER in r["Kernel_Name"]]
    if len(marks) < 2 * (a.segment + 1):
        raise SystemExit(f"found {len(marks)} marker dispatches; need {2 * (a.segment + 1)}")
    lo, hi = marks[2 * a.segment], marks[2 * a.segment + 1]
    seg = rows[lo + 1:hi]
    dur = [(r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3) for r in seg]
    span = (int(rows[hi]["Start_Timestamp"]) - int(rows[lo]["End_Timestamp"])) * 1e-3
    total = sum(d for _, d in dur)
    print(f"{len(dur)} dispatches between markers {a.segment * 2} and {a.segment * 2 + 1}; "
          f"kernel time {total:.1f} us of {span:.1f} us between the markers\n")
    print("| library kernel | dispatches | avg us | min us | max us | total us | % of kernel time |")
    print("|---|---|---|---|---|---|---|")
    for name, pat in LIBRARY_NAMES.items():
        d = [t for s, t in dur if re.search(pat, s)]
        if d:
            print(f"| {name} | {len(d)} | {sum(d) / len(d):.2f} | {min(d):.2f} | {max(d):.2f} | {sum(d):.1f} | "
                  f"{100 * sum(d) / total:.1f} |")
    print("\n| kernel symbol | dispatches | avg us | min us | max us | total us |")
    print("|---|---|---|---|---|---|")
    per = OrderedDict()
    for s, t in dur:
        per.setdefault(short(s), []).append(t)
    for s, d in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        print(f"| {s} | {len(d)} | {sum(d) / len(d):.2f} | {min(d):.2f} | {max(d):.2f} | {sum(d):.1f} |")


if __name__ == "__main__":
    main()
