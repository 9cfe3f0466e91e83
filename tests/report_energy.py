"""Measured energy-based compression (the adaptive rate of Sec. 4.1), one JSON
line per workload layer: time of the per-bin energy reduction over the stored
input spectrum (kernels `input_energy` and, for few bins, `input_energy_sum`,
HIP events inside the library) and its share of peak HBM bandwidth, the time of the whole call including the input's
spectrum, and the band chosen for 90 %, 99 % and 99.9 % of the input's energy
(t, c_eff, preserved fraction) on the seeded inputs.

A reporting script, not a test (pytest does not collect it).  Run it on a GPU
host from the repository root:

    python tests/report_energy.py --out energy.jsonl
"""
import argparse
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from paper_1911_09287_amd import blconv, synth  # noqa: E402

HBM_PEAK_GBS = 8000.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--reps", type=int, default=20)
    args = ap.parse_args()
    import torch
    if not torch.cuda.is_available():
        sys.exit("report_energy.py needs a GPU")
    blconv.load()
    dev = torch.device("cuda:0")
    with open(args.out, "w") as fh:
        for ci in sorted(synth.WORKLOADS):
            for li, layer in enumerate(synth.WORKLOADS[ci].layers):
                x = torch.from_numpy(synth.layer_inputs(ci, li)[0]).to(dev)
                plan = blconv.plan_for_layer(layer, 0.0)
                ws = plan.workspace(dev)
                e = plan.input_energy(x, ws)
                torch.cuda.synchronize()
                def timed(flags, xin):
                    prof = blconv.Profile(capacity=8 * args.reps)
                    with prof:
                        for _ in range(args.reps):
                            plan.input_energy(xin, ws, e, flags=flags)
                        torch.cuda.synchronize()
                    recs = prof.records()
                    prof.release()
                    return recs

                red = timed(blconv.BL_REUSE_X, None)
                # per call: the reduction (and, for few bins, the pass over slice sums)
                red_us = 1e3 * sum(r[1] for r in red) / args.reps
                nbytes = next(r[2] for r in red if r[0] == "input_energy")
                full_us = 1e3 * sum(r[1] for r in timed(0, x)) / args.reps
                eh = e.cpu().numpy()
                choice = {}
                for fraction in (0.9, 0.99, 0.999):
                    t, c, kept_f = plan.rate_for_energy(eh, fraction)
                    choice[str(fraction)] = {"t": t, "c_eff": blconv.plan_for_layer(layer, c).c_eff,
                                             "preserved": kept_f}
                row = {"config": ci, "layer": layer.name, "kept": plan.kept, "reduce_us": red_us,
                       "reduce_GBps": nbytes / (red_us * 1e-6) / 1e9,
                       "reduce_hbm_frac": nbytes / (red_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                       "with_spectrum_us": full_us, "bands": choice}
                fh.write(json.dumps(row) + "\n")
                fh.flush()
                print(json.dumps(row), flush=True)
                del plan, ws


if __name__ == "__main__":
    main()
