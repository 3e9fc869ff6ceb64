"""Host logic of bench.py: the trace summary pairs the library's main kernel
launches of a rocprofv3 kernel trace with the run's logged calls in dispatch
order, attributes the auxiliary launches to the call before them, and keeps
only the timed calls."""
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _write(tmp_path, kernels, calls, line):
    path = tmp_path / "kernel_trace.csv"
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kind", "Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        t = 1000
        for i, (name, ns) in enumerate(kernels):
            w.writerow(["KERNEL_DISPATCH", i + 1, name, t, t + ns])
            t += ns + 10
    log = tmp_path / "log.json"
    log.write_text(json.dumps({"calls": calls, "bench_line": line}))
    return str(path), str(log)


def _line():
    lay = lambda name, g, ms, tf, fr: dict(layer=name, gflop=g, ms_mean=ms, ms_median=ms,
                                           tflops=tf, frac_peak=fr)
    return {"value": 1.0, "ms_per_step": 2.0,
            "config": {"workload": "stack: a, b"},
            "layers": [lay("a", 2.0, 1.0, 2.0, 0.0008), lay("b", 1.0, 0.5, 2.0, 0.0008)],
            "roofline": {"kernel": "conv3d_bf16 (fast route), layer a", "peak": 2500.0,
                         "frac": 0.0008, "achieved": 2.0},
            "configs": {"C1": {"layers": [lay("t", 0.1, 0.1, 1.0, 1.0 / 157.3)]}}}


def _run(csv_path, log_path):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--trace-summary",
                           csv_path, log_path], capture_output=True, text=True, timeout=120)


def test_trace_summary_pairs_launches_with_calls(tmp_path):
    k = "void conv3d_bf16<5, 2, 5, 2, 2, 2, true, false, 0>(Args)"
    calls = [dict(workload="stack", layer="a", phase="warmup", kernel="conv3d_bf16"),
             dict(workload="stack", layer="b", phase="warmup", kernel="pointwise"),
             dict(workload="stack", layer="a", phase="timed", kernel="conv3d_bf16"),
             dict(workload="stack", layer="b", phase="timed", kernel="pointwise"),
             dict(workload="C1", layer="t", phase="timed", kernel="fast_f32")]
    kernels = [(k, 5_000_000), ("void pointwise_conv<false>(PwArgs)", 9_000_000),
               ("at::native::fill_kernel", 777), (k, 1_000_000),
               ("void splitk_reduce<true>(...)", 250_000),
               ("void pointwise_conv<false>(PwArgs)", 500_000),
               ("void fast_conv3d<float>(FArgs)", 100_000),
               ("void cache_copy<2>(...)", 20_000), ("void mfma_probe(float*, int)", 10 ** 9)]
    r = _run(*_write(tmp_path, kernels, calls, _line()))
    assert r.returncode == 0, r.stderr
    rows = {l.split("|")[2].strip(): l for l in r.stdout.splitlines() if l.startswith("| stack")
            or l.startswith("| C1")}
    a = [c.strip() for c in rows["a"].split("|")]
    # timed launch only (1.0 ms), its split-K reduction as auxiliary time
    assert a[4] == "1" and a[5] == "1.0000" and a[7] == "0.2500"
    b = [c.strip() for c in rows["b"].split("|")]
    assert b[5] == "0.5000" and b[7] == "0.0000"
    t = [c.strip() for c in rows["t"].split("|")]
    assert t[5] == "0.1000" and t[7] == "0.0200"
    # fp32 layer priced against its own peak: 0.1 GFLOP in 0.12 ms
    assert abs(float(t[9]) - 100 * (0.1e9 / 0.12e-3 / 1e12) / 157.3) < 0.1
    assert "trace mean 1.0000 ms over 1 timed launches" in r.stdout


def test_trace_summary_refuses_a_count_mismatch(tmp_path):
    calls = [dict(workload="stack", layer="a", phase="timed", kernel="conv3d_bf16")] * 2
    kernels = [("void conv3d_bf16<1>(Args)", 1000)]
    r = _run(*_write(tmp_path, kernels, calls, _line()))
    assert r.returncode != 0 and "1 main kernel launches" in r.stderr


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
