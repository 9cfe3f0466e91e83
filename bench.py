"""Benchmark of the band-limited FFT convolution layer on one MI355X.

One step = forward + grad-input + grad-weight (with map reuse) of every layer
of the workload at compression rate c, on synthetic inputs already resident
in HBM.  Default workload: the ResNet-18-shaped stack of 3x3 layers at CIFAR
resolution (batch 128; 64->64 @32x32, 128->128 @16x16, 256->256 @8x8,
512->512 @4x4; padding 1), c = 0.5, plus the per-rate sweep c in
{0, 0.25, 0.5, 0.75}.  The 1-D FCN time-series stack is timed as an extra
workload beside it.

Timing: W untimed warm-up steps, then K timed steps between two device
synchronisations (HIP events on the stream the kernels run on); ms_per_step
is the mean over the K steps and the median of the per-step times is reported
beside it.  Then the same K steps run again with the library stamping every
kernel's own start and end (hipExtLaunchKernelGGL with two events on the
kernel's stream).  Those events lengthen the gaps between kernels, so they
are kept out of the headline steps; they give the per-kernel averages (which
agree with rocprofv3's kernel trace) and the roofline of the dominant kernel:
  * FFT stages (spectra of x, dy and w, the inverse transforms, the
    weight-gradient inverse DFT and the partial-sum passes): algorithmic
    bytes / time against 8 TB/s HBM;
  * channel contractions: algorithmic flops (8 per complex multiply-add) /
    time against 157.3 TFLOP/s fp32 MFMA where their intensity is above the
    ridge (19.7 flop/B), else bytes against HBM.

Prints ONE JSON line: value = TFLOP-equiv/s, where the equivalent work of a
layer is that of the direct convolution, 3 passes x 2 N C_in C_out Ho Wo K^d
flops.  `cpu_baseline` is the fp64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, GB/s
MFMA_F32_PEAK_TF = 157.3   # MI355X dense fp32 matrix, TFLOP/s
RIDGE = MFMA_F32_PEAK_TF * 1e12 / (HBM_PEAK_GBS * 1e9)


def bound_of(name, nbytes, nflops):
    """Roofline of a kernel: fp32 MFMA for a channel contraction whose
    algorithmic intensity is above the ridge, else HBM (every transform,
    inverse DFT and partial-sum pass is a memory-bound stage)."""
    if nflops and name.startswith("contract") and nflops / nbytes > RIDGE:
        return "mfma", MFMA_F32_PEAK_TF
    return "hbm", HBM_PEAK_GBS


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=3, help="workload index (1..5)")
    ap.add_argument("--c", type=float, default=0.5, help="compression rate of the headline value")
    ap.add_argument("--extra-config", type=int, default=2,
                    help="a second workload timed at the same rate beside the headline (0: none)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the per-c sweep")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the bfloat16-spectra variant of the headline workload")
    ap.add_argument("--graph", action="store_true",
                    help="replay per-layer HIP graphs instead of launching every kernel from the host")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--separate-backward", action="store_true",
                    help="backward as the two calls (grad-input, grad-weight) instead of the combined one")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--table", default=None, help="also write a per-config/per-c table (JSON lines) here")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first run a plain elementwise copy of this many MiB (fp32), the reference kernel "
                         "for scaling hardware traffic counters")
    return ap.parse_args()


class Layer:
    """Device state of one layer: plan, inputs, outputs and workspace."""

    def __init__(self, torch, blconv, layer, arrays, c, dev, desc_flags=0, separate_backward=False):
        self.layer = layer
        self.separate_backward = separate_backward
        self.plan = blconv.plan_for_layer(layer, c, None, desc_flags)
        x, w, dy = arrays
        self.x, self.w, self.dy = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        self.y = torch.empty(self.plan.y_shape(), device=dev)
        self.dx = torch.empty(self.plan.x_shape(), device=dev)
        self.dw = torch.empty(self.plan.w_shape(), device=dev)
        self.ws = self.plan.workspace(dev)
        self.blconv = blconv

    def step(self):
        b = self.blconv
        self.plan.forward(self.x, self.w, self.y, self.ws)
        if self.separate_backward:
            self.plan.backward_input(self.dy, self.w, self.dx, self.ws, flags=b.BL_REUSE_W)
            self.plan.backward_weight(self.x, self.dy, self.dw, self.ws, flags=b.BL_REUSE_X | b.BL_REUSE_DY)
            return
        # both gradients in one call: the grad-input and grad-weight
        # contractions share one launch where their tiles agree
        self.plan.backward(self.dy, None, None, self.dx, self.dw, self.ws, flags=b.BL_REUSE_W | b.BL_REUSE_X)


def capture(torch, layers):
    """One HIP graph per layer holding its three passes.  The layers must have
    run eagerly once (the plans' device tables are uploaded then)."""
    graphs = []
    for L in layers:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            L.step()
        graphs.append(g)
    torch.cuda.synchronize()
    return graphs


def time_steps(torch, layers, steps, warmup, graphs=None):
    """W warm-up steps, then `steps` timed steps between two synchronisations.
    Returns (mean ms per step, median ms per step, median ms per layer, wall
    seconds).  Events on the current stream bracket every step and layer."""
    run = [g.replay for g in graphs] if graphs else [L.step for L in layers]
    for _ in range(warmup):
        for r in run:
            r()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(layers) + 1)] for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    # a short spin kernel before and after the timed steps (outside the
    # events) marks them in a profiler's kernel trace
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for s in range(steps):
        for i, r in enumerate(run):
            ev[s][i].record()
            r()
        ev[s][-1].record()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    per_step = [ev[s][0].elapsed_time(ev[s][-1]) for s in range(steps)]
    per_layer = [float(np.median([ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(steps)]))
                 for i in range(len(layers))]
    return total_ms / steps, float(np.median(per_step)), per_layer, wall


def profile_steps(torch, blconv, layers, steps):
    """The same steps again with the library stamping every kernel's own start
    and end (two HIP events per launch on the stream it runs on).  The events
    add gaps between kernels (the step takes longer), not time inside them.
    Marker kernels bracket the pass, as they do the timed steps, so that a
    profiler's trace of the same pass can be compared.  Returns (all records,
    records per layer)."""
    prof = blconv.Profile(capacity=64 * steps * len(layers))
    lib = blconv.load()
    bounds = []
    torch.cuda.synchronize()
    torch.cuda._sleep(1000)  # marker kernels bracket the pass in a profiler's trace
    with prof:
        for _ in range(steps):
            for i, L in enumerate(layers):
                a = lib.bl_profile_count()
                L.step()
                bounds.append((i, a, lib.bl_profile_count()))
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    recs = prof.records()
    prof.release()
    per_layer = [[] for _ in layers]
    for i, a, b in bounds:
        per_layer[i].extend(recs[a:b])
    return recs, per_layer


def kernel_table(recs):
    """Per library kernel name: launches, average duration, algorithmic rates
    and the fraction of the roofline that applies to it."""
    agg = {}
    for name, ms, nb, nf in recs:
        a = agg.setdefault(name, [0, 0.0, 0.0, 0.0])
        a[0] += 1; a[1] += ms; a[2] += nb; a[3] += nf
    kernels = {}
    for name, (n, ms, nb, nf) in agg.items():
        s = ms * 1e-3
        bound, peak = bound_of(name, nb, nf)
        gbs = nb / s / 1e9
        contraction = name.startswith("contract") and nf > 0
        tfs = nf / s / 1e12 if contraction else None
        kernels[name] = {"launches": n, "avg_us": 1e3 * ms / n, "total_ms": ms,
                         "bytes_per_launch": nb / n, "flops_per_launch": nf / n if contraction else None,
                         "GBps": gbs, "TFLOPs": tfs, "ai": (nf / nb) if contraction else None, "bound": bound,
                         "frac": (tfs if bound == "mfma" else gbs) / peak}
    return agg, kernels


def roofline(agg):
    """Roofline object of the dominant kernel (largest total time)."""
    dom = max(agg, key=lambda k: agg[k][1])
    n, ms, nb, nf = agg[dom]
    s = ms * 1e-3
    bound, peak = bound_of(dom, nb, nf)
    if bound == "hbm":
        return {"kernel": dom, "bound": "hbm", "achieved": nb / s / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": nb / s / 1e9 / HBM_PEAK_GBS, "traffic": None,
                "avg_launch_us": 1e3 * ms / n, "launches": n, "per_launch_bytes": nb / n}
    return {"kernel": dom, "bound": "mfma", "achieved": nf / s / 1e12, "peak": MFMA_F32_PEAK_TF,
            "unit": "TFLOP/s", "frac": nf / s / 1e12 / MFMA_F32_PEAK_TF, "traffic": None,
            "avg_launch_us": 1e3 * ms / n, "launches": n, "per_launch_flops": nf / n,
            "per_launch_bytes": nb / n, "hbm_GBps": nb / s / 1e9,
            "flop_count": "algorithmic: 8 real flops per complex multiply-add"}


KERNEL_SOURCES = {"spec_fwd_1d": "bluestein.hip", "spec_inv_1d": "bluestein.hip", "spec_fwd_2d": "fft2d.hip",
                  "spec_fwd_filt_2d": "fft2d.hip", "spec_inv_wgrad_2d": "fft2d.hip",
                  "spec_inv_2d": "fft2d.hip", "contract_fwd": "contract.hip", "contract_dgrad": "contract.hip",
                  "contract_wgrad": "contract.hip", "contract_bwd": "contract.hip", "wgrad_idft": "direct.hip",
                  "spec_filt": "direct.hip"}


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter measurement, or None if
    there is none for this kernel and workload or the kernel source changed."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    t = json.load(open(path)).get(f"{kernel} @ {workload}", {})
    src = os.path.join(ROOT, "paper_1911_09287_amd", "csrc", KERNEL_SOURCES[kernel])
    if t.get("kernel") != kernel or t.get("workload") != workload or not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] != t.get("source_sha256_16"):
        return None
    return t["traffic_bytes_per_launch"]


def cpu_baseline(cfg, c, target_s):
    """The fp64 oracle on a bounded sample: the first n samples of the batch."""
    from oracle import bl_oracle as bo
    from paper_1911_09287_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    layers = synth.WORKLOADS[cfg].layers
    arrays = [synth.layer_inputs(cfg, i) for i in range(len(layers))]

    def run(n):
        t = time.perf_counter()
        flops = 0.0
        for L, (x, w, dy) in zip(layers, arrays):
            xs, dys = x[:n], dy[:n]
            spatial = (L.H,) if L.ndim == 1 else (L.H, L.W)
            bo.forward(xs, w, L.pad, c)
            bo.backward_input(dys, w, spatial, L.pad, c)
            bo.backward_weight(xs, dys, L.K, L.pad, c)
            flops += 3 * L.direct_flops() * n / L.N
        return time.perf_counter() - t, flops

    N = layers[0].N
    n = 1
    dt, _ = run(n)  # also warms up
    while n < N and dt * (2 if n * 2 <= N else N / n) < target_s:
        n = min(N, n * 2)
        dt, _ = run(n)
    reps, total, flops = 0, 0.0, 0.0
    while total < target_s or reps == 0:
        dt, f = run(n)
        total += dt; flops += f; reps += 1
    return {"value": flops / total / 1e12, "unit": "TFLOP-equiv/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 NumPy oracle, fwd+grad-input+grad-weight of all {len(layers)} layers at c={c} on the "
                      f"first {n} of {N} samples, {reps} repetition(s), {total:.1f} s; numpy.fft single-threaded, "
                      f"BLAS threads={threads}, host CPUs={len(os.sched_getaffinity(0))}"}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the band-limited layer is built and measured on a single "
              "MI355X; run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_1911_09287_amd import blconv, synth
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    blconv.load()
    dev = torch.device("cuda:0")
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib * (1 << 20) // 4
        src = torch.ones(n, device=dev)
        dst = torch.empty(n, device=dev)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)  # reads 4n bytes, writes 4n bytes
        torch.cuda.synchronize()
        del src, dst

    def workload(ci):
        cf = synth.WORKLOADS[ci]
        arr = [synth.layer_inputs(ci, i) for i in range(len(cf.layers))]
        return cf, arr, sum(3 * L.direct_flops() for L in cf.layers)

    def build(cf, arr, c, desc_flags=0):
        return [Layer(torch, blconv, L, a, c, dev, desc_flags, args.separate_backward) for L, a in zip(cf.layers, arr)]

    def graphs_for(Ls):
        if not args.graph:
            return None
        for L in Ls:  # eager once: uploads the plans' device tables before capture
            L.step()
        torch.cuda.synchronize()
        return capture(torch, Ls)

    cfg, arrays, eq_flops = workload(args.config)
    layers = build(cfg, arrays, args.c)
    graphs = graphs_for(layers)
    ms, med, per_layer, wall = time_steps(torch, layers, args.steps, args.warmup, graphs)
    value = eq_flops / (ms * 1e-3) / 1e12
    # per-kernel durations: the same K steps again with kernel events
    recs, recs_by_layer = profile_steps(torch, blconv, layers, args.steps)
    agg, kernels = kernel_table(recs)
    roof = roofline(agg)
    workload_key = f"config {args.config} c={args.c}"
    roof["traffic"] = measured_traffic(roof["kernel"], workload_key)
    if roof["traffic"] is not None:
        roof["traffic_over_algorithmic"] = roof["traffic"] / roof["per_launch_bytes"]
    by_layer = {}
    for L, rl in zip(layers, recs_by_layer):
        _, ks = kernel_table(rl)
        by_layer[L.layer.name] = {k: {"avg_us": round(v["avg_us"], 3), "frac": round(v["frac"], 4),
                                      "bound": v["bound"]} for k, v in ks.items()}

    per_c = []
    if not args.no_sweep:
        for c in cfg.rates:
            Ls = layers if c == args.c else build(cfg, arrays, c)
            m, md, pl, _ = time_steps(torch, Ls, args.steps, args.warmup,
                                      graphs if c == args.c else graphs_for(Ls))
            entry = {"c": c, "c_eff": [L.plan.c_eff for L in Ls], "ms_per_step": m, "ms_per_step_median": md,
                     "ms_per_layer": pl, "tflop_equiv_s": eq_flops / (m * 1e-3) / 1e12}
            rc, _ = profile_steps(torch, blconv, Ls, min(args.steps, 10))
            _, ks = kernel_table(rc)
            entry["kernel_frac"] = {k: round(v["frac"], 4) for k, v in ks.items()}
            per_c.append(entry)
            del Ls

    # the same workload with the saved spectra in bfloat16 (reduced precision
    # combined with band-limiting); reported beside the fp32 headline, not as it
    variants = {}
    if not args.no_variants:
        Ls = build(cfg, arrays, args.c, blconv.BL_DESC_BF16_SPECTRA)
        m, md, pl, _ = time_steps(torch, Ls, args.steps, args.warmup, graphs_for(Ls))
        variants["bf16_spectra"] = {"dtype": "bf16 spectra, fp32 accumulation", "c": args.c, "ms_per_step": m,
                                    "ms_per_layer": pl, "tflop_equiv_s": eq_flops / (m * 1e-3) / 1e12,
                                    "speedup_vs_f32": ms / m}
        del Ls

    extra = None
    if args.extra_config and args.extra_config != args.config:
        ecf, earr, eflops = workload(args.extra_config)
        Ls = build(ecf, earr, args.c)
        m, md, pl, _ = time_steps(torch, Ls, args.steps, args.warmup, graphs_for(Ls))
        extra = {"workload": ecf.name, "config_index": args.extra_config, "c": args.c, "ms_per_step": m,
                 "ms_per_step_median": md, "ms_per_layer": pl, "tflop_equiv_s": eflops / (m * 1e-3) / 1e12}
        rc, _ = profile_steps(torch, blconv, Ls, args.steps)
        eagg, eks = kernel_table(rc)
        extra["roofline"] = roofline(eagg)
        et = measured_traffic(extra["roofline"]["kernel"], f"config {args.extra_config} c={args.c}")
        extra["roofline"]["traffic"] = et
        if et is not None:
            extra["roofline"]["traffic_over_algorithmic"] = et / extra["roofline"]["per_launch_bytes"]
        extra["kernels"] = eks
        del Ls

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config, args.c, args.cpu_seconds)

    out = {
        "metric": "band-limited conv fwd+bwd TFLOP-equiv/s (ms/layer vs c; %HBM / %MFMA peak)",
        "value": value,
        "unit": "TFLOP-equiv/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_median": med,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "config_index": args.config, "c": args.c,
                   "layers": [L.name for L in cfg.layers], "batch": cfg.layers[0].N,
                   "c_eff": [L.plan.c_eff for L in layers], "ms_per_layer": per_layer,
                   "equiv_gflop_per_step": eq_flops / 1e9},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "kernels_by_layer": by_layer,
        "per_c": per_c,
        "variants": variants,
        "extra_workload": extra,
        "wall_s_timed": wall,
        "launch": "hip_graph per layer" if args.graph else "eager",
        "backward": "two calls (grad-input, grad-weight)" if args.separate_backward else "one call (both gradients)",
    }
    print(json.dumps(out), flush=True)

    if args.table:
        with open(args.table, "w") as fh:
            for ci in sorted(synth.WORKLOADS):
                cf, arr, _ = workload(ci)
                for c in cf.rates:
                    for L, a in zip(cf.layers, arr):
                        Ls = [Layer(torch, blconv, L, a, c, dev)]
                        m, md, _, _ = time_steps(torch, Ls, args.steps, args.warmup)
                        rc, _ = profile_steps(torch, blconv, Ls, min(args.steps, 10))
                        _, ks = kernel_table(rc)
                        fh.write(json.dumps({"config": ci, "layer": L.name, "c": c, "c_eff": Ls[0].plan.c_eff,
                                             "ms": m, "ms_median": md,
                                             "tflop_equiv_s": 3 * L.direct_flops() / (m * 1e-3) / 1e12,
                                             "kernels": ks}) + "\n")
                        fh.flush()
                        del Ls


if __name__ == "__main__":
    main()
