"""Turn two rocprofv3 counter runs into measured HBM traffic per launch.

Measurement tool (not used by the library).  Inputs are the counter CSVs of
two runs of the same command, one with ``--pmc FETCH_SIZE`` and one with
``--pmc WRITE_SIZE`` (kilobytes per dispatch), where the command first runs a
plain elementwise copy of known size (``bench.py --calibrate-copy-mib``).
The copy's readings give the scale from counter kilobytes to bytes for reads
and for writes; the kernel's average per-dispatch readings times those scales
are its measured traffic.  The result is written as JSON together with a hash
of the kernel's source file, so that a later run can tell whether the kernel
has changed since the counters were taken; the output file keeps one entry
per kernel name.

    python -m paper_1911_09287_amd.traffic --fetch F.csv --write W.csv \\
        --kernel k_bluestein --match "<1024, 2>" --name spec_fwd_1d \\
        --source paper_1911_09287_amd/csrc/bluestein.hip --copy-mib 256 \\
        --workload "..." --out profiles/traffic.json
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re


def read(path):
    rows = {}
    for r in csv.DictReader(open(path)):
        key = r["Dispatch_Id"]
        rows[key] = (r["Kernel_Name"], float(r["Counter_Value"]))
    return rows


def source_hash(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--kernel", required=True, help="substring of the kernel symbol")
    ap.add_argument("--match", default="", help="further substring (e.g. template arguments)")
    ap.add_argument("--regex", default="", help="or: a regular expression the kernel symbol must match "
                                                 "(several instantiations under one library name)")
    ap.add_argument("--name", required=True, help="the library's name for the kernel")
    ap.add_argument("--source", required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--copy-kernel", default="elementwise", help="substring of the copy kernel symbol")
    ap.add_argument("--workload", required=True)
    ap.add_argument("--out", required=True)
    a = ap.parse_args()

    f, w = read(a.fetch), read(a.write)
    copy_bytes = a.copy_mib * (1 << 20)

    def pick(rows, sub, extra="", rx=""):
        return [v for (n, v) in rows.values() if sub in n and extra in n and (not rx or re.search(rx, n))]

    cf, cw = pick(f, a.copy_kernel), pick(w, a.copy_kernel)
    if not cf or not cw:
        raise SystemExit("calibration copy kernel not found")
    # the largest dispatch of the copy kernel is the calibration copy
    read_scale = copy_bytes / (max(cf) * 1024.0)
    write_scale = copy_bytes / (max(cw) * 1024.0)
    kf, kw = pick(f, a.kernel, a.match, a.regex), pick(w, a.kernel, a.match, a.regex)
    if not kf or not kw:
        raise SystemExit("kernel not found")
    fetch = sum(kf) / len(kf) * 1024.0 * read_scale
    write = sum(kw) / len(kw) * 1024.0 * write_scale
    out = {"kernel": a.name, "symbol": a.regex or (a.kernel + a.match), "workload": a.workload,
           "source": a.source, "source_sha256_16": source_hash(a.source),
           "dispatches": len(kf), "copy_mib": a.copy_mib,
           "read_scale": read_scale, "write_scale": write_scale,
           "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
           "traffic_bytes_per_launch": fetch + write}
    # the file holds one entry per kernel name; other kernels' entries are kept
    os.makedirs(os.path.dirname(os.path.abspath(a.out)), exist_ok=True)
    table = json.load(open(a.out)) if os.path.exists(a.out) else {}
    # one entry per (library kernel name, workload)
    table[f"{a.name} @ {a.workload}"] = out
    json.dump(table, open(a.out, "w"), indent=1, sort_keys=True)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
