#!/usr/bin/env python3
"""Benchmark of the cached causal Conv3D on one MI355X.

Workload (default): the 720p wide-channel decode stack -- causal Conv3D
layers Ci=Co=640 at 44x80, Ci=Co=320 at 176x320, Ci=320->Co=160 at 352x640,
Ci=Co=160 at 704x1280 (3x3x3, stride 1, spatial pad 1, 4 new frames + a
2-frame cache that starts at zeros), then a 1x1x1 shortcut conv
Ci=320->Co=160 at 352x640 that takes the fallback route; bf16 storage, fp32
accumulation.  One STEP is one chunk through all five layers: route
decisions, the fast implicit-GEMM kernel with its fused bias and cache update,
and the fallback kernel.  Caches are carried between steps.  Weights are
repacked once per layer before timing (the paper caches the derived weight
slices across calls).  Inputs are seeded synthetic tensors already resident
in device memory.

Prints ONE JSON line: whole-chunk TFLOP/s (algorithmic FLOP: only valid
temporal taps, padded spatial positions counted), chunk latency, per-layer
TFLOP/s and fraction of the 2.5 PFLOP/s bf16 matrix peak, the dominant
kernel's roofline, and the oracle's CPU rate on a bounded sample.  The same
line carries the other layer configurations, each streamed once untimed and
once timed from a zero cache ("configs": the tiny fp32 layer against the
157.3 TFLOP/s fp32 matrix peak, the 384-channel 60x104 one-frame layer with
and without the split-K workspace, the two 240x416 layers, the 96-channel
480x832 layer), and the run's provenance (host CPU, thread counts, ROCm,
hipcc and torch versions, library and kernel-source hashes, SHA-256 of every
input buffer).
"""
import argparse
import gc
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("causal Conv3D TFLOP/s and % of bf16 MFMA peak per layer shape; "
          "chunk latency (ms)")
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak (published)
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix peak (published)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E peak (published)


# The library's compute kernels, by the plan query's name for them (the
# kernel a call's plan names is its one main launch, one of the listed
# symbols); the auxiliary kernels a call may add after it (split-K reduction,
# cache copy, prologue pass).
MAIN_KERNELS = {"conv3d_bf16": ("conv3d_bf16",), "head": ("conv_head",),
                "tap1x1": ("conv_tap1x1", "conv_tap1x1_chunk"),
                "pointwise": ("pointwise_conv", "pointwise_resident"),
                "fast_f32": ("fast_conv3d",), "fallback_direct": ("fallback_conv3d",)}
MAIN_SYMBOLS = tuple(n for names in MAIN_KERNELS.values() for n in names)
AUX_KERNELS = ("splitk_reduce", "cache_copy", "cache_copy_pro", "prologue_pass")

# Further configurations timed by a default run, after the headline one:
# (label, workload, with the split-K workspace attached).
EXTRA_CONFIGS = (("C1", "tiny_f32", False), ("C2", "low_res", False),
                 ("C2+workspace", "low_res", True), ("C3", "mid_res", False),
                 ("C4", "full_res", False))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="stack_720p")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-configs", action="store_true",
                    help="time the headline workload only (skip the other configurations)")
    ap.add_argument("--no-hash", action="store_true",
                    help="skip the SHA-256 of the inputs (provenance)")
    ap.add_argument("--launch-log", default=None,
                    help="write every library call of the run (workload, layer, phase, "
                         "planned kernel) and the printed line to this JSON file, for "
                         "--trace-summary")
    ap.add_argument("--trace-summary", nargs=2, metavar=("KERNEL_TRACE_CSV", "LAUNCH_LOG"),
                    default=None,
                    help="print the per-layer kernel times of a rocprofv3 --kernel-trace "
                         "run of this script (matched to its --launch-log) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 512 MiB device copy (the reference kernel "
                         "for scaling FETCH_SIZE / WRITE_SIZE counters) and exit")
    ap.add_argument("--layer", default=None,
                    help="time only this layer of the workload (for per-layer profiles); "
                         "the JSON line then covers that layer alone")
    ap.add_argument("--fused-block", action="store_true",
                    help="time the fused residual-block form on each layer of the workload "
                         "against the plain call and against the unfused pipeline (prologue "
                         "and residual add as separate torch ops) and exit")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="time the vendor bf16 GEMM (torch.matmul) on square and "
                         "conv-shaped problems and exit: what the matrix cores reach "
                         "on this device outside this library")
    args = ap.parse_args()
    if args.trace_summary:
        trace_summary(*args.trace_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_31938_amd import c3c, inputs

    if args.copy_calibration:
        copy_calibration()
        return
    if args.gemm_reference:
        gemm_reference()
        return
    if args.fused_block:
        fused_block(args.workload, args.steps)
        return

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log = [] if args.launch_log else None
    digests = {}

    # ------------------------------------------------------------ headline
    head = Workload(args.workload, dev, layer=args.layer, log=log)
    wl = head.wl
    dtype = wl["dtype"]
    total_ms, per_layer, t_wall, counters = head.time_steps(args.steps, args.warmup)
    total_flops = sum(L_["flops"] for L_ in head.layers) * args.steps
    value = total_flops / (total_ms * 1e-3) / 1e12

    # dominant kernel: the fast conv on the largest layer
    fast_layers = [p for p in per_layer if p["route"] == "fast"] or per_layer
    dom = max(fast_layers, key=lambda p: p["gflop"])
    dom_i = [p["layer"] for p in per_layer].index(dom["layer"])
    dom_L = head.layers[dom_i]
    dom_mean_ms = dom["ms_mean"]
    achieved = dom["gflop"] * 1e9 / (dom_mean_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
    if dom["route"] == "fast":
        kname = dom["kernel"]
        roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                    "traffic": measured_traffic(dom["layer"]) if kname == "conv3d_bf16" else None,
                    "kernel": f"{kname} (fast route), layer {dom['layer']}",
                    "timing": f"mean of {args.steps} HIP-event-bracketed launches "
                              "on the launch stream"}
    else:
        # a fallback layer timed alone (--layer): HBM-bound, algorithmic bytes
        gbs = algorithmic_bytes(dom_L["sp"], dtype) / (dom_mean_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None,
                    "kernel": f"fallback route, layer {dom['layer']}"}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(dom_L, dtype, args.cpu_seconds)
    if not args.no_hash:
        digests[args.workload] = head.input_sha256()
    shapes = sorted({(L_["sp"]["T"], L_["sp"]["Tc"]) for L_ in head.layers})
    frames = ", ".join(f"T={t} new + {tc} cached frames" for t, tc in shapes)
    chunks = wl["chunks"]
    layer_names = ", ".join(L_["name"] for L_ in head.layers)
    dom_L = None
    head.free()

    # ----------------------------------------------- the other configurations
    configs = {}
    if not args.no_configs and args.layer is None and args.workload == "stack_720p":
        for label, name, ws in EXTRA_CONFIGS:
            w_ = Workload(name, dev, use_ws=ws, log=log, label=label)
            configs[label] = w_.time_stream()
            if not args.no_hash and name not in digests:
                digests[name] = w_.input_sha256()
            w_.free()

    # the matrix cores' sustained rate on this machine (outside the timed regions):
    # back-to-back bf16 products, four workgroups per compute unit
    probe = mfma_probe_rate()
    hbm = hbm_reference()
    if roofline["bound"] == "mfma" and dtype == "bf16":
        roofline["frac_of_probe"] = round(achieved / probe["tflops"], 4)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {layer_names}; N=1, {frames}, "
            f"{chunks}-chunk cache carry; step = one chunk through every layer",
            "global_batch": 1, "chunks_per_stream": chunks},
        "chunk_latency_ms": round(total_ms / args.steps, 4),
        "layers": per_layer,
        "roofline": roofline,
        "configs": configs,
        "mfma_probe": probe,
        "hbm_reference": hbm,
        "counters": counters,
        "wall_s": round(t_wall, 4),
        "provenance": provenance(digests),
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    line = json.dumps(out)
    print(line, flush=True)
    if log is not None:
        with open(args.launch_log, "w") as f:
            json.dump({"calls": log, "bench_line": out}, f)


class Workload:
    """One workload's device tensors (weights repacked once, every chunk's
    input resident in device memory, two cache buffers per layer that swap
    roles between chunks) and its timed runs."""

    def __init__(self, name, dev, use_ws=False, layer=None, log=None, label=None):
        import torch
        from paper_2609_31938_amd import c3c, inputs
        self.name, self.label, self.log = name, label or name, log
        self.wl = wl = inputs.WORKLOADS[name]
        self.dtype = dtype = wl["dtype"]
        self.chunks = wl["chunks"]
        self.ctx = c3c.Context()
        self.ws = None
        names = [lname for lname, _ in wl["layers"]]
        if layer is not None and layer not in names:
            print(f"unknown layer {layer!r}; the workload has {names}", file=sys.stderr)
            sys.exit(2)
        self.layers = []
        need = 0
        for lid, (lname, sp) in enumerate(wl["layers"]):
            if layer is not None and lname != layer:
                continue
            w, b = inputs.layer_tensors(sp, dtype, wl["id"], lid, dev)
            route, why = c3c.route_query(None, sp, dtype)
            wpack, repack_ms = None, None
            if route == "fast":
                # the second repack is timed (the first one also loads the
                # kernel's code object)
                wpack = c3c.weight_repack(self.ctx, sp, w)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                c3c.weight_repack(self.ctx, sp, w, wpack)
                e1.record()
                torch.cuda.synchronize()
                repack_ms = e0.elapsed_time(e1)
            To, Ho, Wo, L = c3c.output_dims(sp, dtype)
            xs = [inputs.chunk_input(sp, dtype, wl["id"], lid, c, dev) for c in range(self.chunks)]
            y = torch.empty((sp["N"], sp["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
            cbuf = [torch.zeros((sp["N"], sp["Ci"], sp["Tc"], sp["H"], sp["W"]), dtype=w.dtype,
                                device=dev) for _ in range(2)]
            if use_ws:
                need = max(need, c3c.workspace_bytes(sp, dtype))
            self.layers.append(dict(name=lname, sp=sp, w=w, b=b, wpack=wpack, xs=xs, y=y,
                                    cbuf=cbuf, route=route, reason=why,
                                    flops=c3c.flops(sp, dtype), repack_ms=repack_ms))
        if need:
            self.ws = torch.empty((need + 3) // 4, dtype=torch.float32, device=dev)
            self.ctx.set_workspace(self.ws)
        for L_ in self.layers:
            L_["plan"] = c3c.plan_query(self.ctx, L_["sp"], dtype,
                                        self.ws.numel() * 4 if self.ws is not None else 0)
        torch.cuda.synchronize()

    def reset_caches(self):
        for L_ in self.layers:
            for cb in L_["cbuf"]:
                cb.zero_()
            L_["cur"] = 0

    def chunk(self, c, phase, evs=None):
        """Chunk c through every layer, caches carried; evs[i] = (start, end)
        events recorded around layer i's call."""
        from paper_2609_31938_amd import c3c
        for i, L_ in enumerate(self.layers):
            sp = L_["sp"]
            cin = L_["cbuf"][L_["cur"]] if sp["Tc"] else None
            cout = L_["cbuf"][1 - L_["cur"]] if sp["Tc"] else None
            if self.log is not None:
                p = L_["plan"]
                self.log.append(dict(workload=self.label, layer=L_["name"], phase=phase,
                                     kernel=p["kernel"], splits=p["splits"],
                                     workgroups=p["workgroups"]))
            if evs is not None:
                evs[i][0].record()
            c3c.conv3d_causal_cached(self.ctx, sp, L_["xs"][c], cin, L_["w"], L_["wpack"],
                                     L_["b"], L_["y"], cout)
            if evs is not None:
                evs[i][1].record()
            if sp["Tc"]:
                L_["cur"] = 1 - L_["cur"]

    def _events(self, n):
        import torch
        return [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in self.layers]
                for _ in range(n)]

    def _per_layer(self, ev):
        peak = PEAK_BF16_TFLOPS if self.dtype == "bf16" else PEAK_F32_TFLOPS
        rows = []
        for i, L_ in enumerate(self.layers):
            times = [e[i][0].elapsed_time(e[i][1]) for e in ev]
            fl = L_["flops"]
            med = statistics.median(times)
            tf = fl / (med * 1e-3) / 1e12
            p = L_["plan"]
            rows.append(dict(layer=L_["name"], route=L_["route"], reason=L_["reason"],
                             kernel=p["kernel"], splits=p["splits"], workgroups=p["workgroups"],
                             gflop=round(fl / 1e9, 3), ms_median=round(med, 4),
                             ms_mean=round(sum(times) / len(times), 4),
                             tflops=round(tf, 2), frac_peak=round(tf / peak, 4),
                             repack_ms=(round(L_["repack_ms"], 3)
                                        if L_["repack_ms"] is not None else None)))
        return rows

    def time_steps(self, steps, warmup):
        """Headline timing: `warmup` untimed chunks, then `steps` timed chunks
        (the chunk index wraps around the stream; caches keep carrying),
        bracketed by synchronisations."""
        import torch
        # Python's cyclic collector can stall the host for tens of
        # milliseconds between two launches: it runs before the warm-up and
        # is held off until the timed region ends.  Not between the two: an
        # idle gap there lets the clocks fall before the timed steps.
        gc.collect()
        gc.disable()
        self.reset_caches()
        for s in range(warmup):
            self.chunk(s % self.chunks, "warmup")
        torch.cuda.synchronize()
        self.ctx.reset()
        self.reset_caches()
        torch.cuda.synchronize()
        ev = self._events(steps)
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_wall = time.perf_counter()
        start.record()
        for s in range(steps):
            self.chunk(s % self.chunks, "timed", ev[s])
        stop.record()
        torch.cuda.synchronize()
        t_wall = time.perf_counter() - t_wall
        gc.enable()
        return start.elapsed_time(stop), self._per_layer(ev), t_wall, self.ctx.counters()

    def time_stream(self):
        """One untimed pass over the whole stream (every chunk, caches carried
        from a zero cache), then one timed pass from a zero cache again:
        per-layer call times (median over the chunks), the chunk latency
        (first layer's start to last layer's end, median over the chunks) and
        the stream's whole time."""
        import torch
        gc.collect()
        gc.disable()
        self.reset_caches()
        for c in range(self.chunks):
            self.chunk(c, "warmup")
        torch.cuda.synchronize()
        self.ctx.reset()
        self.reset_caches()
        torch.cuda.synchronize()
        ev = self._events(self.chunks)
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for c in range(self.chunks):
            self.chunk(c, "timed", ev[c])
        stop.record()
        torch.cuda.synchronize()
        gc.enable()
        lat = [e[0][0].elapsed_time(e[-1][1]) for e in ev]
        stream_ms = start.elapsed_time(stop)
        flops = sum(L_["flops"] for L_ in self.layers) * self.chunks
        return {"workload": self.name, "dtype": self.dtype, "chunks": self.chunks,
                "split_k_workspace_bytes": self.ws.numel() * 4 if self.ws is not None else 0,
                "chunk_latency_ms_median": round(statistics.median(lat), 4),
                "stream_ms": round(stream_ms, 4),
                "stream_tflops": round(flops / (stream_ms * 1e-3) / 1e12, 2),
                "layers": self._per_layer(ev), "counters": self.ctx.counters()}

    def input_sha256(self):
        """SHA-256 over every input buffer of the workload (per layer: w, b,
        then each chunk's x; the first cache is zeros): the digest of the
        concatenated per-buffer digests."""
        import hashlib
        from concurrent.futures import ThreadPoolExecutor
        from paper_2609_31938_amd import inputs
        bufs = []
        for L_ in self.layers:
            bufs += [L_["w"], L_["b"]] + list(L_["xs"])
        with ThreadPoolExecutor(8) as ex:
            parts = list(ex.map(inputs.sha256, bufs))
        return {"sha256": hashlib.sha256("".join(parts).encode()).hexdigest(),
                "buffers": len(parts)}

    def free(self):
        import torch
        self.ctx.set_workspace(None)
        self.layers = []
        self.ws = None
        gc.collect()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def provenance(digests):
    """Host, toolchain and input records of the run."""
    import platform
    import torch
    cpu_model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    rocm = None
    try:
        rocm = open("/opt/rocm/.info/version").read().strip()
    except OSError:
        pass
    # the compiler that built the library, as the build recorded it (no
    # compiler is started here: under a profiler a child process would
    # inherit the profiler's GPU-initialising preload)
    hipcc = None
    try:
        bi = json.load(open(os.path.join(ROOT, "paper_2609_31938_amd", "libc3c.buildinfo.json")))
        hipcc = " | ".join(bi.get("hipcc", []))[:200] or None
    except (OSError, ValueError):
        pass
    import oracle
    props = torch.cuda.get_device_properties(0)
    import hashlib
    so = os.path.join(ROOT, "paper_2609_31938_amd", "libc3c.so")
    return {"cpu_model": cpu_model, "host_threads_available": len(os.sched_getaffinity(0)),
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS"),
            "oracle_threads": oracle.num_threads(), "python": platform.python_version(),
            "torch": torch.__version__, "torch_hip": torch.version.hip, "rocm": rocm,
            "hipcc": hipcc, "gpu": props.name, "gpu_arch": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count,
            "libc3c_sha256": hashlib.sha256(open(so, "rb").read()).hexdigest(),
            "conv_bf16_source_sha256": kernel_source_sha256(),
            "inputs": digests}


def trace_summary(csv_path, log_path):
    """Per-layer kernel times from a rocprofv3 kernel trace of this script,
    matched to the run's launch log: the library's main kernel launches in
    dispatch order pair one to one with the logged calls; split-K reductions
    and cache copies that follow a main launch belong to its call.  Prints
    markdown."""
    import csv
    import re
    rows = list(csv.DictReader(open(csv_path)))
    if not rows:
        sys.exit("empty kernel trace")
    key = lambda *names: next(k for k in rows[0] if any(n == k for n in names))
    kn, ks, ke = key("Kernel_Name"), key("Start_Timestamp"), key("End_Timestamp")
    kd = next((k for k in rows[0] if k in ("Dispatch_Id", "Correlation_Id")), None)
    rows.sort(key=lambda r: int(r[kd]) if kd else int(r[ks]))
    main_re = re.compile(r"\b(" + "|".join(MAIN_SYMBOLS) + r")\b")
    aux_re = re.compile(r"\b(" + "|".join(AUX_KERNELS) + r")\b")
    log = json.load(open(log_path))
    calls, line = log["calls"], log["bench_line"]
    launches = []  # [name, main ms, aux ms]
    for r in rows:
        name = r[kn]
        ms = (int(r[ke]) - int(r[ks])) * 1e-6
        m = main_re.search(name)
        if m:
            launches.append([name, ms, 0.0])
        elif aux_re.search(name) and launches:
            launches[-1][2] += ms
    if len(launches) != len(calls):
        sys.exit(f"{len(launches)} main kernel launches in the trace, {len(calls)} calls logged")
    groups = {}
    for c, (name, ms, aux) in zip(calls, launches):
        if main_re.search(name).group(1) not in MAIN_KERNELS[c["kernel"]]:
            sys.exit(f"call {c} matched to launch {name}")
        if c["phase"] != "timed":
            continue
        g = groups.setdefault((c["workload"], c["layer"]), dict(kernel=name, ms=[], aux=[]))
        g["ms"].append(ms)
        g["aux"].append(aux)
    ev = {(line["config"]["workload"].split(":")[0], p["layer"]): p for p in line["layers"]}
    for label, cfg in line.get("configs", {}).items():
        for p in cfg["layers"]:
            ev[(label, p["layer"])] = p
    head = line["config"]["workload"].split(":")[0]
    print("| workload | layer | kernel | launches | trace mean ms | trace median ms | "
          "aux ms | TFLOP/s (trace mean) | % of peak (trace) | event mean ms | % of peak (events) |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for (wl, layer), g in groups.items():
        wl_name = head if wl == head else wl
        p = ev.get((wl_name, layer))
        mean = sum(g["ms"]) / len(g["ms"])
        med = statistics.median(g["ms"])
        aux = sum(g["aux"]) / len(g["aux"])
        km = re.search(r"\b(" + "|".join(MAIN_SYMBOLS) + r")\b(<[^()]*>)?", g["kernel"])
        kname = km.group(0) if km else g["kernel"]
        if p is not None:
            peak = p["tflops"] / p["frac_peak"] if p["frac_peak"] else PEAK_BF16_TFLOPS
            tf = p["gflop"] * 1e9 / ((mean + aux) * 1e-3) / 1e12
            print(f"| {wl} | {layer} | `{kname}` | {len(g['ms'])} | {mean:.4f} | {med:.4f} | "
                  f"{aux:.4f} | {tf:.1f} | {100 * tf / peak:.1f} | {p['ms_mean']:.4f} | "
                  f"{100 * p['frac_peak']:.1f} (median) |")
    rf = line["roofline"]
    dom = rf["kernel"].split("layer ")[-1]
    g = groups.get((head, dom))
    if g is not None:
        mean = sum(g["ms"]) / len(g["ms"])
        gflop = ev[(head, dom)]["gflop"]
        tf = gflop * 1e9 / (mean * 1e-3) / 1e12
        print(f"\nDominant kernel ({rf['kernel']}): trace mean {mean:.4f} ms over "
              f"{len(g['ms'])} timed launches = {tf:.1f} TFLOP/s = frac {tf / rf['peak']:.4f} "
              f"of {rf['peak']}; the line's event-based frac is {rf['frac']} "
              f"(achieved {rf['achieved']}).")
    print(f"\nBench line of the same run: value {line['value']} TFLOP/s, "
          f"{line['ms_per_step']} ms per chunk.")


def algorithmic_bytes(sp, dtype):
    """Bytes one call must move at least: read x, cache, w and bias once,
    write y and the new cache once."""
    es = 4 if dtype == "f32" else 2
    hw = sp["H"] * sp["W"]
    Z = sp["Tc"] + sp["T"]
    L = min(sp["p_base"], Z)
    p_l = sp["p_base"] - sp["Tc"]
    To = (Z + p_l + sp["p_r"] - sp["d_t"] * (sp["Kt"] - 1) - 1) // sp["s_t"] + 1
    Ho = (sp["H"] + 2 * sp["p_h"] - sp["d_h"] * (sp["Kh"] - 1) - 1) // sp["s_h"] + 1
    Wo = (sp["W"] + 2 * sp["p_w"] - sp["d_w"] * (sp["Kw"] - 1) - 1) // sp["s_w"] + 1
    n_in = sp["N"] * sp["Ci"] * Z * hw
    n_w = sp["Co"] * (sp["Ci"] // sp["groups"]) * sp["Kt"] * sp["Kh"] * sp["Kw"]
    n_out = sp["N"] * sp["Co"] * To * Ho * Wo + sp["N"] * sp["Ci"] * L * hw
    return es * (n_in + n_w + sp["Co"] * sp["has_bias"] + n_out)


def mfma_probe_rate(iters=50000):
    """TFLOP/s of the library's matrix-core probe (c3c_mfma_probe): 8
    independent bf16 16x16x32 products back to back per wave, no memory
    traffic, at four workgroups of 4 waves per compute unit (4 waves per
    SIMD) and at one (one wave per SIMD, as the convolution kernels run).  The
    published peak times the clock the device holds under matrix-core load;
    the implied clock is reported with it."""
    import torch
    from paper_2609_31938_amd import c3c
    cus = torch.cuda.get_device_properties(0).multi_processor_count

    def rate(blocks, n):
        c3c.mfma_probe(blocks, n // 10)  # warm-up
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        out, fl = c3c.mfma_probe(blocks, n)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        return fl / (ms * 1e-3) / 1e12, ms, bool(torch.isfinite(out).all().item())

    tf, ms, fin = rate(4 * cus, iters)
    tf1, _, fin1 = rate(cus, 4 * iters)
    return {"tflops": round(tf, 1), "frac_of_published_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "implied_clock_ghz": round(2.4 * tf / PEAK_BF16_TFLOPS, 3), "ms": round(ms, 3),
            "launch": f"{4 * cus} workgroups x 4 waves, 8 chains, {iters} iterations",
            "tflops_one_wave_per_simd": round(tf1, 1),
            "finite": fin and fin1}


def hbm_reference():
    """What plain device streams reach on this machine (outside the timed
    regions): torch's copy of 1 GiB (read + write) and fill of 1 GiB (write),
    the practical ceiling for the HBM-bound kernels next to the published
    8 TB/s."""
    import torch
    n = 512 * 1024 * 1024
    a = torch.ones(n, device="cuda", dtype=torch.bfloat16)
    b = torch.empty_like(a)

    def rate(fn, nbytes, k=10):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return round(nbytes / (e0.elapsed_time(e1) / k * 1e-3) / 1e9, 1)

    out = {"copy_GBps": rate(lambda: b.copy_(a), 2 * a.numel() * 2),
           "fill_GBps": rate(lambda: b.fill_(0.5), a.numel() * 2), "bytes": a.numel() * 2}
    del a, b
    torch.cuda.empty_cache()
    return out


def fused_block(workload, iters):
    """Per layer: the plain call, the fused form (prologue + residual, and each
    alone; and with the prologue-pass workspace attached), and the unfused
    pipeline a PyTorch user would run (the prologue as torch ops into a new
    tensor, the plain call, then y += residual), with the HBM-bound floor of
    the two separate passes (read x, write u; read y and the residual, write
    y) and the extra device memory each path allocates."""
    import torch
    from paper_2609_31938_amd import c3c, inputs
    wl = inputs.WORKLOADS[workload]
    dtype = wl["dtype"]
    dev = torch.device("cuda", 0)
    ctx = c3c.Context()
    out = []

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for lid, (lname, sp) in enumerate(wl["layers"]):
        # the collector runs here, before the layer's inputs are made, and
        # is held off through its measurements (no pause between launches,
        # no idle gap that lets the clocks fall before a timed call)
        gc.collect()
        gc.disable()
        w, b = inputs.layer_tensors(sp, dtype, wl["id"], lid, dev)
        route, _ = c3c.route_query(None, sp, dtype)
        wpack = c3c.weight_repack(ctx, sp, w) if route == "fast" else None
        To, Ho, Wo, L = c3c.output_dims(sp, dtype)
        x = inputs.chunk_input(sp, dtype, wl["id"], lid, 0, dev)
        cin = torch.zeros((sp["N"], sp["Ci"], sp["Tc"], sp["H"], sp["W"]), dtype=w.dtype,
                          device=dev) if sp["Tc"] else None
        cout = torch.empty((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), dtype=w.dtype,
                           device=dev) if L else None
        y = torch.empty((sp["N"], sp["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
        scale, shift = inputs.affine_inputs(sp, wl["id"], lid, 0, dev)
        r = inputs.residual_input(tuple(y.shape), dtype, wl["id"], lid, 0, dev)
        s5, t5 = scale[:, :, None, None, None], shift[:, :, None, None, None]

        def plain():
            c3c.conv3d_causal_cached(ctx, sp, x, cin, w, wpack, b, y, cout)

        def fused(pro=True, res=True, c=ctx):
            c3c.conv3d_causal_cached_fused(c, sp, x, cin, w, wpack, b,
                                           scale if pro else None, shift if pro else None,
                                           r if res else None, y, cout)

        # the same fused call with the prologue-pass workspace attached
        need = c3c.fused_workspace_bytes(sp, dtype)
        ctx_ws = c3c.Context()
        ws = torch.empty(max(need, 16) // 4, dtype=torch.float32, device=dev) if need else None
        ctx_ws.set_workspace(ws)

        def unfused():
            u = torch.nn.functional.silu(x.float() * s5 + t5).to(w.dtype)
            c3c.conv3d_causal_cached(ctx, sp, u, cin, w, wpack, b, y, cout)
            y.add_(r)

        # the normalised block form (per-pixel RMS over the channels, gain,
        # bias, SiLU in one pass into the workspace; residual fused) against
        # the same steps as torch ops around the plain call
        ctx_b = c3c.Context()
        need_b = c3c.block_workspace_bytes(sp, dtype)
        ws_b = torch.empty((need_b + 3) // 4, dtype=torch.float32, device=dev)
        ctx_b.set_workspace(ws_b)
        gamma, beta = inputs.norm_inputs(sp, wl["id"], lid, dev)
        g5, b5 = gamma[None, :, None, None, None], beta[None, :, None, None, None]

        def block():
            c3c.conv3d_causal_cached_block(ctx_b, sp, x, cin, w, wpack, b, gamma, beta, 1e-6, r,
                                           y, cout)

        def unfused_norm():
            xf = x.float()
            rr = torch.rsqrt(xf.square().mean(dim=1, keepdim=True) + 1e-6)
            u = torch.nn.functional.silu(xf * rr * g5 + b5).to(w.dtype)
            c3c.conv3d_causal_cached(ctx, sp, u, cin, w, wpack, b, y, cout)
            y.add_(r)

        torch.cuda.synchronize()
        m0 = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        unfused()
        torch.cuda.synchronize()
        extra_unfused = torch.cuda.max_memory_allocated() - m0
        torch.cuda.reset_peak_memory_stats()
        fused()
        torch.cuda.synchronize()
        extra_fused = torch.cuda.max_memory_allocated() - m0
        n = max(2, iters)
        t_plain = timed(plain, n)
        t_fused = timed(fused, n)
        t_pro = timed(lambda: fused(True, False), n)
        t_res = timed(lambda: fused(False, True), n)
        t_unf = timed(unfused, n)
        t_pass = timed(lambda: fused(c=ctx_ws), n) if need else None
        t_block = timed(block, n)
        t_unf_norm = timed(unfused_norm, n)
        xb, yb = x.numel() * 2, y.numel() * 2
        floor_ms = (2 * xb + 3 * yb) / (PEAK_HBM_GBS * 1e9) * 1e3
        out.append(dict(layer=lname, route=route, plain_ms=round(t_plain, 4),
                        fused_ms=round(t_fused, 4), prologue_only_ms=round(t_pro, 4),
                        residual_only_ms=round(t_res, 4), unfused_torch_ms=round(t_unf, 4),
                        fused_prologue_pass_ms=round(t_pass, 4) if t_pass is not None else None,
                        prologue_pass_workspace_bytes=int(need),
                        unfused_floor_ms=round(t_plain + floor_ms, 4),
                        block_norm_ms=round(t_block, 4), unfused_norm_torch_ms=round(t_unf_norm, 4),
                        block_workspace_bytes=int(need_b),
                        extra_bytes_unfused=int(extra_unfused), extra_bytes_fused=int(extra_fused)))
        print(json.dumps(out[-1]), flush=True)
        ctx_ws.set_workspace(None)
        ctx_b.set_workspace(None)
        del x, y, r, cin, cout, w, b, wpack, ws, ws_b
        gc.enable()
        torch.cuda.empty_cache()
    print(json.dumps({"fused_block": workload, "layers": out}), flush=True)


def copy_calibration():
    """A plain device-to-device copy of 512 MiB, three times: the kernel of
    known traffic against which the FETCH_SIZE / WRITE_SIZE counters are
    scaled."""
    import torch
    n = 256 * 1024 * 1024
    a = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_each_way": a.numel() * 2, "launches": 3}),
          flush=True)


def gemm_reference():
    """bf16 GEMM rates of the vendor library (torch.matmul -> hipBLASLt) on
    this device: two square problems, and the plain GEMMs with the shapes of
    the 720p layers as implicit GEMMs (M = output pixels of one frame times
    T_o, K = 27 Ci, N = Co).  A reference for what the matrix cores reach at
    this device's sustained clock; no part of this library."""
    import torch
    dev = torch.device("cuda", 0)
    out = []
    for (M, K, N) in ((8192, 8192, 8192), (16384, 16384, 16384),
                      (4 * 704 * 1280, 27 * 160, 160), (4 * 352 * 640, 27 * 320, 160),
                      (4 * 176 * 320, 27 * 320, 320), (4 * 44 * 80, 27 * 640, 640)):
        a = torch.randn(M, K, device=dev, dtype=torch.bfloat16)
        b = torch.randn(K, N, device=dev, dtype=torch.bfloat16)
        iters = 3 if M * K * N > 2 ** 42 else 10
        for _ in range(3):
            c = a @ b
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            c = a @ b
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        tf = 2.0 * M * K * N / (ms * 1e-3) / 1e12
        out.append(dict(M=M, K=K, N=N, ms=round(ms, 4), tflops=round(tf, 1),
                        frac_peak=round(tf / PEAK_BF16_TFLOPS, 4)))
        del a, b, c
    print(json.dumps({"gemm_reference": "torch.matmul bf16", "results": out}), flush=True)


def kernel_source_sha256():
    import hashlib
    src = os.path.join(ROOT, "paper_2609_31938_amd", "csrc", "conv_bf16.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()


def measured_traffic(layer):
    """HBM bytes per launch of the dominant kernel, from the committed
    rocprofv3 counter summary, or None when that summary was taken on a
    different kernel source (or does not exist)."""
    path = os.path.join(ROOT, "profiles", f"conv3d_bf16_{layer}_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            fields[k.strip("` ")] = v.strip().strip("`")
    if fields.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(L_, dtype, budget_s):
    """The oracle, as it stands, on host cores: output rows of the dominant
    layer for an output frame whose three taps are all valid, sampled until
    about `budget_s` seconds of CPU work; scaled to TFLOP/s."""
    import torch
    import oracle
    sp = dict(L_["sp"])
    x = L_["xs"][1].cpu()
    cache = L_["xs"][0][:, :, -sp["Tc"]:].contiguous().cpu() if sp["Tc"] else None
    w, b = L_["w"].cpu(), L_["b"].cpu()
    To, Ho, Wo, _ = oracle.output_dims(sp)
    t_frame = To - 1  # last output frame: every tap reads a real frame
    per_row = 2.0 * sp["Ci"] * sp["Kt"] * sp["Kh"] * sp["Kw"] * Wo
    rows_done, t_used, co = 0, 0.0, 0
    batch = 8
    while t_used < budget_s and co < sp["Co"]:
        r0 = (co * To + t_frame) * Ho + 1  # interior rows: all 3 kernel rows valid
        n = min(batch, Ho - 2)
        t0 = time.perf_counter()
        oracle.conv3d_rows(sp, dtype, x, cache, w, b, r0, r0 + n)
        dt = time.perf_counter() - t0
        t_used += dt
        rows_done += n
        co += 1
        if dt < 1.0:
            batch = min(batch * 2, Ho - 2)
    flops = per_row * rows_done
    return {"value": round(flops / t_used / 1e12, 6), "unit": "TFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"layer {L_['name']}: {rows_done} interior output rows of "
                      f"{Wo} pixels in output frame {t_frame} (all taps valid), "
                      f"{flops / 1e9:.1f} GFLOP fp64 in {t_used:.1f} s"}


if __name__ == "__main__":
    main()
