"""GPU parity at the benchmarked layer shapes (Wan-VAE-decoder-shaped causal
Conv3D layers), streamed chunk by chunk with the cache carried on the device.

The tiny fp32 workload is compared in full; the bf16 layers, too large for a
full fp64 oracle pass, are compared on sampled outputs the oracle computes one
by one (random positions plus every tile border of several planes), on the
first chunks and the last.  The carried cache is compared bit for bit on every
checked chunk, and the route counters and the fallback-shape histogram must
equal what the route rule gives for the whole call sequence.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs
from paper_2609_31938_amd.inputs import WORKLOADS

from gpu_util import as_f64, check, host, run, sample_indices, say

pytestmark = pytest.mark.gpu


def _bits(t, dtype):
    t = host(t)
    return t.view(torch.int16).numpy().view(np.uint16) if dtype in ("bf16", "f16") else t.numpy()


def _stream(name, check_chunks=None, full=False):
    wl = WORKLOADS[name]
    dtype = wl["dtype"]
    ctx = c3c.Context()
    expect = dict(calls=0, fast=0, fallback=0, unsupported=0)
    hist = {}
    for lid, (lname, sp0) in enumerate(wl["layers"]):
        w, b = inputs.layer_tensors(sp0, dtype, wl["id"], lid, "cuda")
        r0, _ = c3c.route_query(None, sp0, dtype)
        wpack = c3c.weight_repack(ctx, sp0, w) if r0 == "fast" else None
        cache = inputs.zero_cache(sp0, dtype, "cuda") if sp0["Tc"] else None
        last = wl["chunks"] - 1
        todo = set(range(wl["chunks"])) if check_chunks is None else {c % wl["chunks"] for c in check_chunks}
        for ci in range(wl["chunks"]):
            sp = dict(sp0, Tc=0 if cache is None else cache.shape[2])
            x = inputs.chunk_input(sp, dtype, wl["id"], lid, ci, "cuda")
            say(f"{name}/{lname} chunk {ci} {'check' if ci in todo else ''}")
            y, cache_new = run(ctx, sp, x, cache, w, wpack, b)
            route, why = oracle.route(sp, dtype)
            expect["calls"] += 1
            if route == "fast":
                expect["fast"] += 1
            else:
                expect["fallback"] += 1
                expect["unsupported"] += 1
                key = (why, lname)
                hist[key] = hist.get(key, 0) + 1
            if ci in todo:
                hx, hc = host(x), host(cache) if cache is not None else None
                hw_, hb = host(w), host(b)
                if full:
                    ref = oracle.conv3d(sp, dtype, hx, hc, hw_, hb)
                    m = check(as_f64(y), ref, dtype, f"{lname} chunk {ci}")
                else:
                    idx = sample_indices(tuple(y.shape), 2048, seed=ci)
                    ref = oracle.conv3d_points(sp, dtype, hx, hc, hw_, hb, idx)
                    got = as_f64(y.reshape(-1)[torch.from_numpy(idx).cuda()])
                    m = check(got, ref, dtype, f"{lname} chunk {ci}")
                ref_cache = oracle.cache_update(sp, dtype, hx, hc)
                assert np.array_equal(_bits(cache_new, dtype), ref_cache), f"{lname} cache {ci}"
                say(f"  rel={m['rel']:.3e} rmse={m['rmse']:.3e} cos={m['cos']:.8f}")
            cache = cache_new if cache_new.numel() else None
    c = ctx.counters()
    for k, v in expect.items():
        assert c[k] == v, (k, c, expect)
    assert c["strict_rejects"] == c["fast_error"] == c["forced"] == 0
    got_hist = {(r, None): n for r, _, n in ctx.fallback_shapes()}
    assert sum(got_hist.values()) == sum(hist.values())
    return ctx


def test_tiny_f32_stream_full_compare():
    _stream("tiny_f32", full=True)


def test_low_res_stream_21_chunks():
    _stream("low_res", check_chunks=None)


def test_mid_res_layers():
    _stream("mid_res", check_chunks=[0, 1, -1])


def test_full_res_layer():
    _stream("full_res", check_chunks=[0, 1, -1])


def test_stack_720p():
    ctx = _stream("stack_720p", check_chunks=[0, 1, -1])
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"], c["unsupported"]) == (25, 20, 5, 5)
    shapes = ctx.fallback_shapes()
    assert len(shapes) == 1 and shapes[0][0] == "kt1" and shapes[0][2] == 5
    assert shapes[0][1]["Kt"] == 1 and shapes[0][1]["Ci"] == 320 and shapes[0][1]["Co"] == 160


def test_temporal_convs():
    """Temporal convolutions (kernel 3x1x1) on the fast route: the 1x1-spatial
    kernel, unit stride with a 2-frame cache and stride 2 with a 1-frame
    cache, streamed over 5 chunks."""
    ctx = _stream("temporal", check_chunks=[0, 1, -1])
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (15, 15, 0)


def test_head_conv():
    """The decoder's output head (96 -> 3 channels at 480x832) on the
    16-channel tile, streamed over 5 chunks."""
    ctx = _stream("head", check_chunks=[0, -1])
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (5, 5, 0)
