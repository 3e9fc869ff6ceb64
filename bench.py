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
kernel's roofline, and the oracle's CPU rate on a bounded sample.
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="stack_720p")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
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

    wl = inputs.WORKLOADS[args.workload]
    dtype = wl["dtype"]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ctx = c3c.Context()
    chunks = wl["chunks"]

    # ---------------------------------------------------------------- setup
    layers = []
    names = [lname for lname, _ in wl["layers"]]
    if args.layer is not None and args.layer not in names:
        print(f"unknown layer {args.layer!r}; the workload has {names}", file=sys.stderr)
        sys.exit(2)
    for lid, (lname, sp) in enumerate(wl["layers"]):
        if args.layer is not None and lname != args.layer:
            continue
        w, b = inputs.layer_tensors(sp, dtype, wl["id"], lid, dev)
        route, why = c3c.route_query(None, sp, dtype)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        wpack = c3c.weight_repack(ctx, sp, w) if route == "fast" else None
        torch.cuda.synchronize()
        repack_ms = (time.perf_counter() - t0) * 1e3 if route == "fast" else None
        To, Ho, Wo, L = c3c.output_dims(sp, dtype)
        xs = [inputs.chunk_input(sp, dtype, wl["id"], lid, c, dev) for c in range(chunks)]
        y = torch.empty((sp["N"], sp["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
        cbuf = [torch.zeros((sp["N"], sp["Ci"], sp["Tc"], sp["H"], sp["W"]), dtype=w.dtype,
                            device=dev) for _ in range(2)]
        layers.append(dict(name=lname, sp=sp, w=w, b=b, wpack=wpack, xs=xs, y=y, cbuf=cbuf,
                           route=route, reason=why, flops=c3c.flops(sp, dtype),
                           repack_ms=repack_ms))
    torch.cuda.synchronize()

    def reset_caches():
        for L_ in layers:
            for cb in L_["cbuf"]:
                cb.zero_()
            L_["cur"] = 0

    def step(s, evs=None):
        c = s % chunks
        for i, L_ in enumerate(layers):
            sp = L_["sp"]
            cin = L_["cbuf"][L_["cur"]] if sp["Tc"] else None
            cout = L_["cbuf"][1 - L_["cur"]] if sp["Tc"] else None
            if evs is not None:
                evs[i][0].record()
            c3c.conv3d_causal_cached(ctx, sp, L_["xs"][c], cin, L_["w"], L_["wpack"], L_["b"],
                                     L_["y"], cout)
            if evs is not None:
                evs[i][1].record()
            if sp["Tc"]:
                L_["cur"] = 1 - L_["cur"]

    # ---------------------------------------------------------------- warmup
    # Python's cyclic collector can stall the host for tens of milliseconds
    # between two launches (seen at fixed points of a run): it runs before
    # the warm-up and is held off until the timed region ends.  Not between
    # the two: an idle gap there lets the clocks fall before the timed steps.
    gc.collect()
    gc.disable()
    reset_caches()
    for s in range(args.warmup):
        step(s)
    torch.cuda.synchronize()
    ctx.reset()
    reset_caches()
    torch.cuda.synchronize()

    # ---------------------------------------------------------------- timed
    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in layers]
          for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record()
    for s in range(args.steps):
        step(s, ev[s])
    stop.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    gc.enable()
    total_ms = start.elapsed_time(stop)

    counters = ctx.counters()
    per_layer = []
    total_flops = 0.0
    for i, L_ in enumerate(layers):
        times = [ev[s][i][0].elapsed_time(ev[s][i][1]) for s in range(args.steps)]
        fl = L_["flops"]
        total_flops += fl * args.steps
        med = statistics.median(times)
        tf = fl / (med * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
        per_layer.append(dict(layer=L_["name"], route=L_["route"], reason=L_["reason"],
                              gflop=round(fl / 1e9, 3), ms_median=round(med, 4),
                              ms_mean=round(sum(times) / len(times), 4),
                              tflops=round(tf, 2), frac_peak=round(tf / peak, 4),
                              repack_ms=(round(L_["repack_ms"], 3)
                                         if L_["repack_ms"] is not None else None)))
    value = total_flops / (total_ms * 1e-3) / 1e12

    # dominant kernel: the fast conv on the largest layer
    fast_layers = [p for p in per_layer if p["route"] == "fast"] or per_layer
    dom = max(fast_layers, key=lambda p: p["gflop"])
    dom_i = [p["layer"] for p in per_layer].index(dom["layer"])
    dom_mean_ms = dom["ms_mean"]
    achieved = dom["gflop"] * 1e9 / (dom_mean_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
    if dom["route"] == "fast":
        kname = "conv3d_bf16" if layers[dom_i]["sp"]["Kh"] == 3 else "pointwise_conv (1x1 spatial)"
        roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                    "traffic": measured_traffic(dom["layer"]) if kname == "conv3d_bf16" else None,
                    "kernel": f"{kname} (fast route), layer {dom['layer']}"}
    else:
        # a fallback layer timed alone (--layer): HBM-bound, algorithmic bytes
        gbs = algorithmic_bytes(layers[dom_i]["sp"], dtype) / (dom_mean_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                    "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None,
                    "kernel": f"fallback route, layer {dom['layer']}"}
    # the matrix cores' sustained rate on this machine (outside the timed region):
    # back-to-back bf16 products, one workgroup per compute unit
    probe = mfma_probe_rate()
    if roofline["bound"] == "mfma" and dtype == "bf16":
        roofline["frac_of_probe"] = round(achieved / probe["tflops"], 4)
    shapes = sorted({(L_["sp"]["T"], L_["sp"]["Tc"]) for L_ in layers})
    frames = ", ".join(f"T={t} new + {tc} cached frames" for t, tc in shapes)

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
        "config": {"workload": f"{args.workload}: " + ", ".join(
            f"{L_['name']}" for L_ in layers) + f"; N=1, {frames}, "
            f"{chunks}-chunk cache carry; step = one chunk through every layer",
            "global_batch": 1, "chunks_per_stream": chunks},
        "chunk_latency_ms": round(total_ms / args.steps, 4),
        "layers": per_layer,
        "roofline": roofline,
        "mfma_probe": probe,
        "counters": counters,
        "wall_s": round(t_wall, 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layers[dom_i], dtype, args.cpu_seconds)
    print(json.dumps(out), flush=True)


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
    """TFLOP/s of the library's matrix-core probe (c3c_mfma_probe): four
    workgroups of 4 waves per compute unit, 8 independent bf16 16x16x32
    products back to back per wave, no memory traffic.  The published peak
    times the clock the device holds under matrix-core load; the implied
    clock is reported with it."""
    import torch
    from paper_2609_31938_amd import c3c
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 4 * cus
    c3c.mfma_probe(blocks, iters // 10)  # warm-up
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    out, fl = c3c.mfma_probe(blocks, iters)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    tf = fl / (ms * 1e-3) / 1e12
    return {"tflops": round(tf, 1), "frac_of_published_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "implied_clock_ghz": round(2.4 * tf / PEAK_BF16_TFLOPS, 3), "ms": round(ms, 3),
            "launch": f"{blocks} workgroups x 4 waves, 8 chains, {iters} iterations",
            "finite": bool(torch.isfinite(out).all().item())}


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
        xb, yb = x.numel() * 2, y.numel() * 2
        floor_ms = (2 * xb + 3 * yb) / (PEAK_HBM_GBS * 1e9) * 1e3
        out.append(dict(layer=lname, route=route, plain_ms=round(t_plain, 4),
                        fused_ms=round(t_fused, 4), prologue_only_ms=round(t_pro, 4),
                        residual_only_ms=round(t_res, 4), unfused_torch_ms=round(t_unf, 4),
                        fused_prologue_pass_ms=round(t_pass, 4) if t_pass is not None else None,
                        prologue_pass_workspace_bytes=int(need),
                        unfused_floor_ms=round(t_plain + floor_ms, 4),
                        extra_bytes_unfused=int(extra_unfused), extra_bytes_fused=int(extra_fused)))
        print(json.dumps(out[-1]), flush=True)
        ctx_ws.set_workspace(None)
        del x, y, r, cin, cout, w, b, wpack, ws
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
