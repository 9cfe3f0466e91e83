"""Measured table of the band-limited layer, one JSON line per config, layer
and rate: GPU time of forward + grad-input + grad-weight, TFLOP-equivalent
rate, the spectral stages' share of peak HBM bandwidth, the contraction's
share of peak fp32 MFMA (or HBM) rate, relative error of y, dx and dw against
the oracle, whether the kept-index mask equals the oracle's, and the oracle's
own CPU time for the three passes with the cores it used.

A reporting script, not a test (pytest does not collect it).  Run it on a
GPU host from the repository root:

    python tests/report_table.py --out table.jsonl [--configs 1 2 ...]

The oracle runs single-shot per row (fp64 NumPy; numpy.fft is single
threaded, the per-bin matmuls use the BLAS threads reported in the row).
"""
import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

import numpy as np  # noqa: E402

import bench  # noqa: E402
from oracle import bl_oracle as bo  # noqa: E402
from paper_1911_09287_amd import blconv, synth  # noqa: E402
from test_parity_gpu import elem, gpu_passes, oracle_passes, rel  # noqa: E402

SPECTRAL = ("spec_", "wgrad_idft", "wgrad_reduce")


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max((p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"), default=1)
    except Exception:
        return None


def stage_fracs(kernels):
    """Time-weighted HBM fraction of the spectral stages, and the contraction's
    fraction of its own roofline (MFMA when flop-bound, else HBM)."""
    fb = ft = 0.0
    cf = cb = ct = 0.0
    bound = set()
    for name, k in kernels.items():
        t = k["total_ms"] * 1e-3
        if name.startswith(SPECTRAL):
            fb += k["GBps"] * 1e9 * t
            ft += t
        elif name.startswith("contract"):
            ct += t
            cb += k["GBps"] * 1e9 * t
            if k["TFLOPs"]:
                cf += k["TFLOPs"] * 1e12 * t
            bound.add(k["bound"])
    fft_hbm = fb / ft / (bench.HBM_PEAK_GBS * 1e9) if ft else None
    if "mfma" in bound:
        con = ("mfma", cf / ct / (bench.MFMA_F32_PEAK_TF * 1e12))
    else:
        con = ("hbm", cb / ct / (bench.HBM_PEAK_GBS * 1e9)) if ct else (None, None)
    return fft_hbm, con


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    ap.add_argument("--configs", type=int, nargs="*", default=sorted(synth.WORKLOADS))
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    args = ap.parse_args()
    import torch
    if not torch.cuda.is_available():
        sys.exit("report_table.py needs a GPU")
    blconv.load()
    dev = torch.device("cuda:0")
    cores = len(os.sched_getaffinity(0))
    with open(args.out, "w") as fh:
        for ci in args.configs:
            cfg = synth.WORKLOADS[ci]
            for li, layer in enumerate(cfg.layers):
                x, w, dy = synth.layer_inputs(ci, li)
                for c in cfg.rates:
                    print(f"[table] config {ci} layer {layer.name} c={c}", flush=True)
                    L = bench.Layer(torch, blconv, layer, (x, w, dy), c, dev)
                    ms, _, _, _ = bench.time_steps(torch, [L], args.steps, args.warmup)
                    recs, _ = bench.profile_steps(torch, blconv, [L], 5)
                    _, ks = bench.kernel_table(recs)
                    fft_hbm, (cbound, cfrac) = stage_fracs(ks)
                    c_eff = L.plan.c_eff
                    del L
                    gy, gdx, gdw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
                    ref_mask = bo.mask(layer.ndim, plan.fft[0] if layer.ndim == 1 else plan.fft, c)
                    mask_ok = bool(np.array_equal(plan.mask(), np.asarray(ref_mask, dtype=np.uint8)))
                    t0 = time.perf_counter()
                    ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
                    t_cpu = time.perf_counter() - t0
                    row = {"config": ci, "layer": layer.name, "c": c, "c_eff": c_eff, "ms": ms,
                           "tflop_equiv_s": 3 * layer.direct_flops() / (ms * 1e-3) / 1e12,
                           "fft_hbm_frac": fft_hbm, "contract_bound": cbound, "contract_frac": cfrac,
                           "rel_err": [rel(gy, ry), rel(gdx, rdx), rel(gdw, rdw)],
                           "elem_err": [elem(gy, ry), elem(gdx, rdx), elem(gdw, rdw)], "mask_exact": mask_ok,
                           "oracle_cpu_ms": 1e3 * t_cpu, "oracle_cores": cores, "oracle_blas_threads": blas_threads(),
                           "kernels": ks}
                    fh.write(json.dumps(row) + "\n")
                    fh.flush()
                    print(f"    ms={ms:.3f} rel={row['rel_err']} mask={mask_ok} oracle={t_cpu:.2f}s", flush=True)
                    del plan


if __name__ == "__main__":
    main()
