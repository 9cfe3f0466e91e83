"""Host logic of the measurement path (CPU only, no GPU calls).

The benchmark's per-kernel table and roofline object, the lookup of measured
HBM traffic (and its refusal once the kernel source has changed), and the
three tools that turn rocprofv3 output into the committed summaries (kernel
statistics between marker dispatches, matrix-core counters against the
algorithmic flops, counter bytes scaled by a copy of known size), each run on
small synthetic inputs whose answers are known by construction.
"""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def run_tool(mod, *args):
    out = subprocess.run([sys.executable, "-m", f"paper_1911_09287_amd.{mod}", *map(str, args)], cwd=ROOT,
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    return out.stdout


def write_csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=list(rows[0]))
        w.writeheader()
        w.writerows(rows)


def table_row(text, first):
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if cells and cells[0] == first:
            return cells
    raise AssertionError(f"no row {first!r} in:\n{text}")


def test_kernel_table_and_roofline():
    # (name, ms, bytes, flops) per launch: a contraction above the ridge, a transform,
    # and a contraction below the ridge (memory-bound by its intensity)
    recs = [("contract_bwd", 0.030, 60e6, 2.88e9)] * 3 + [("spec_fwd_2d", 0.010, 25e6, 1e6)] * 2 + \
           [("contract_fwd", 0.004, 40e6, 1e8)]
    agg, ks = bench.kernel_table(recs)
    k = ks["contract_bwd"]
    assert k["launches"] == 3 and k["avg_us"] == pytest.approx(30.0)
    assert k["bound"] == "mfma"
    assert k["TFLOPs"] == pytest.approx(2.88e9 / 30e-6 / 1e12)
    assert k["frac"] == pytest.approx(k["TFLOPs"] / 157.3)
    t = ks["spec_fwd_2d"]
    assert t["bound"] == "hbm" and t["flops_per_launch"] is None
    assert t["frac"] == pytest.approx(25e6 / 10e-6 / 1e9 / 8000.0)
    assert ks["contract_fwd"]["bound"] == "hbm"  # 2.5 flop/B, below the ridge
    r = bench.roofline(agg)
    assert r["kernel"] == "contract_bwd" and r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert r["achieved"] == pytest.approx(2.88e9 / 30e-6 / 1e12)
    assert r["frac"] == pytest.approx(r["achieved"] / 157.3)
    assert r["per_launch_flops"] == pytest.approx(2.88e9) and r["avg_launch_us"] == pytest.approx(30.0)


def test_measured_traffic_follows_the_source(tmp_path, monkeypatch):
    src = os.path.join(ROOT, "paper_1911_09287_amd", "csrc", "contract.hip")
    key = "contract_bwd @ config 3 c=0.5"
    table = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    assert key in table
    got = bench.measured_traffic("contract_bwd", "config 3 c=0.5")
    expect = table[key]["traffic_bytes_per_launch"]
    import hashlib
    if hashlib.sha256(open(src, "rb").read()).hexdigest()[:16] == table[key]["source_sha256_16"]:
        assert got == expect
    else:
        assert got is None
    assert bench.measured_traffic("contract_bwd", "no such workload") is None
    assert bench.measured_traffic("no_such_kernel", "config 3 c=0.5") is None
    # a tree whose kernel source differs from the measured one gets no traffic figure
    (tmp_path / "profiles").mkdir()
    (tmp_path / "paper_1911_09287_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps({key: table[key]}))
    (tmp_path / "paper_1911_09287_amd" / "csrc" / "contract.hip").write_text(open(src).read() + "\n// edited\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("contract_bwd", "config 3 c=0.5") is None


def _trace_rows():
    """A kernel trace: marker, 3 timed dispatches, marker, marker, 2 dispatches, marker."""
    t = [0]

    def disp(name, us):
        start = t[0]
        t[0] += int(us * 1000) + 500
        return {"Kernel_Name": name, "Start_Timestamp": str(start), "End_Timestamp": str(start + int(us * 1000))}

    bwd = "void blc::(anonymous namespace)::k_cgemm_bwd<64, 32, false>(float const*)"
    fwd = "void blc::(anonymous namespace)::k_fft2_fwd<17, 17, HIP_vector_type<float, 2u>, true>(float const*)"
    return [disp("spin_kernel", 1), disp(bwd, 30), disp(bwd, 34), disp(fwd, 10), disp("spin_kernel", 1),
            disp("spin_kernel", 1), disp(bwd, 40), disp(fwd, 12), disp("spin_kernel", 1)]


def test_kstats_segments(tmp_path):
    path = tmp_path / "trace.csv"
    write_csv(path, _trace_rows())
    out0 = run_tool("kstats", path)
    assert "3 dispatches between markers 0 and 1" in out0
    row = table_row(out0, "contract_bwd")
    assert row[1] == "2" and float(row[2]) == pytest.approx(32.0) and float(row[3]) == pytest.approx(30.0)
    row = table_row(out0, "spec_fwd_2d")
    assert row[1] == "1" and float(row[2]) == pytest.approx(10.0)
    assert float(table_row(out0, "contract_bwd")[6]) == pytest.approx(100 * 64 / 74, abs=0.1)
    out1 = run_tool("kstats", path, "--segment", 1)
    assert float(table_row(out1, "contract_bwd")[2]) == pytest.approx(40.0)
    assert float(table_row(out1, "spec_fwd_2d")[2]) == pytest.approx(12.0)


def test_mfmastats_against_algorithmic_flops(tmp_path):
    trace = tmp_path / "trace.csv"
    write_csv(trace, _trace_rows())
    bwd = "void blc::(anonymous namespace)::k_cgemm_bwd<64, 32, false>(float const*)"
    rows = []
    for d in (1, 2):
        rows.append({"Dispatch_Id": str(d), "Kernel_Name": bwd, "Counter_Name": "MfmaFlopsF32",
                     "Counter_Value": str(2.0e9 + 0.2e9 * d)})
        rows.append({"Dispatch_Id": str(d), "Kernel_Name": bwd, "Counter_Name": "MfmaUtil",
                     "Counter_Value": str(40.0 + d)})
    counters = tmp_path / "counters.csv"
    write_csv(counters, rows)
    bench_json = tmp_path / "bench.json"
    bench_json.write_text("noise\n" + json.dumps({"kernels": {"contract_bwd": {"flops_per_launch": 2.3e9}}}) + "\n")
    out = run_tool("mfmastats", counters, trace, "--bench", bench_json)
    row = table_row(out, "contract_bwd")
    # executed 2.3 GFLOP per dispatch on average, equal to the algorithmic count,
    # over 32 us average trace time: 71.9 TFLOP/s, 0.457 of 157.3
    assert row[1] == "2 / 2"
    assert float(row[2]) == pytest.approx(2.3)
    assert float(row[3]) == pytest.approx(1.0)
    assert float(row[4]) == pytest.approx(41.5)
    assert float(row[5]) == pytest.approx(32.0)
    assert float(row[7]) == pytest.approx(2.3e9 / 32e-6 / 1e12, abs=0.06)
    assert float(row[8]) == pytest.approx(2.3e9 / 32e-6 / 1e12 / 157.3, abs=0.001)


def test_traffic_scaled_by_copy(tmp_path):
    copy = "void at::native::elementwise_kernel<128, 4>(int)"
    kern = "void blc::(anonymous namespace)::k_cgemm_bwd<64, 32, false>(float const*)"
    mib = 256
    # the copy of 256 MiB reads as half its bytes and writes as all of them
    fetch = [{"Dispatch_Id": "1", "Kernel_Name": copy, "Counter_Name": "FETCH_SIZE", "Counter_Value": str(mib * 512)},
             {"Dispatch_Id": "2", "Kernel_Name": copy, "Counter_Name": "FETCH_SIZE", "Counter_Value": "3"},
             {"Dispatch_Id": "3", "Kernel_Name": kern, "Counter_Name": "FETCH_SIZE", "Counter_Value": "1000"},
             {"Dispatch_Id": "4", "Kernel_Name": kern, "Counter_Name": "FETCH_SIZE", "Counter_Value": "3000"}]
    write = [dict(r, Counter_Name="WRITE_SIZE") for r in fetch]
    write[0]["Counter_Value"] = str(mib * 1024)
    write[2]["Counter_Value"], write[3]["Counter_Value"] = "500", "700"
    fp, wp, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "t.json"
    write_csv(fp, fetch)
    write_csv(wp, write)
    src = os.path.join(ROOT, "paper_1911_09287_amd", "csrc", "contract.hip")
    run_tool("traffic", "--fetch", fp, "--write", wp, "--kernel", "k_cgemm_bwd", "--regex", "k_cgemm_bwd<",
             "--name", "contract_bwd", "--source", src, "--copy-mib", mib, "--workload", "w", "--out", out)
    e = json.load(open(out))["contract_bwd @ w"]
    assert e["read_scale"] == pytest.approx(2.0) and e["write_scale"] == pytest.approx(1.0)
    assert e["dispatches"] == 2
    assert e["fetch_bytes_per_launch"] == pytest.approx(2000 * 1024 * 2.0)
    assert e["write_bytes_per_launch"] == pytest.approx(600 * 1024)
    assert e["traffic_bytes_per_launch"] == pytest.approx(2000 * 2048 + 600 * 1024)


def test_bench_refuses_more_than_one_gpu():
    out = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 2
    assert "one GPU" in (out.stdout + out.stderr)
