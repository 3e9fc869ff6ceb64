"""GPU parity at the benchmarked layer shapes (Wan-VAE-decoder-shaped causal
Conv3D layers), streamed chunk by chunk with the cache carried on the device.

Every chunk of every layer writes into NaN-filled outputs bracketed by NaN
guard bands: all of y and of the new cache must come back finite (every
element written), the guard bands untouched, and the new cache must equal
the oracle's bit for bit.  On the checked chunks (the first two and the
last) the output is compared with the oracle:
  * whole output planes (n, co, t) at both edges of output-channel tiles, in
    the first and the last output frame;
  * sampled points: random ones, and the tile borders of the workgroup grid
    the call actually used (from the library's plan query);
  * and, for one chunk of the 384->192 and 96->96 layers, every output.
The tiny fp32 workload is compared in full on every chunk.  The same streams
are rerun with every call forced onto the fallback route (the paper's
baseline with zero fast hits).  Route counters and the fallback-shape
histogram must equal what the route rule gives for the whole sequence.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs
from paper_2609_31938_amd.inputs import WORKLOADS

from gpu_util import (as_f64, check, check_planes, guarded, guards_intact, host,
                      sample_indices, say)

pytestmark = pytest.mark.gpu

# (layer, chunk) pairs compared on every output element
FULL = {("c384to192_240x416", 1), ("c96_480x832", 1), ("c32_32x32", 0), ("c32_32x32", 1),
        ("c32_32x32", 2), ("c32_32x32", 3)}


def _bits(t, dtype):
    t = host(t)
    return t.view(torch.int16).numpy().view(np.uint16) if dtype in ("bf16", "f16") else t.numpy()


def _planes(shape, plan):
    """(n, co, t) planes compared whole: both edges of the first and last
    output-channel tiles, in the first and the last output frame."""
    N, Co, To, _, _ = shape
    tco = plan["tile_co"] or Co
    edges = sorted({0, min(tco - 1, Co - 1), min(tco, Co - 1), Co - 1})
    return sorted({(n, co, t) for n in {0, N - 1} for co in edges for t in {0, To - 1}})


def _stream(name, check_chunks=(0, 1, -1), mode=0):
    wl = WORKLOADS[name]
    dtype = wl["dtype"]
    ctx = c3c.Context(mode)
    forced = bool(mode & c3c.MODE_FORCE_FALLBACK)
    expect = dict(calls=0, fast=0, fallback=0, unsupported=0, forced=0)
    hist = {}
    for lid, (lname, sp0) in enumerate(wl["layers"]):
        w, b = inputs.layer_tensors(sp0, dtype, wl["id"], lid, "cuda")
        r0, _ = c3c.route_query(None, sp0, dtype)
        wpack = c3c.weight_repack(ctx, sp0, w) if r0 == "fast" else None
        cache = inputs.zero_cache(sp0, dtype, "cuda") if sp0["Tc"] else None
        todo = {c % wl["chunks"] for c in check_chunks}
        for ci in range(wl["chunks"]):
            sp = dict(sp0, Tc=0 if cache is None else cache.shape[2])
            plan = c3c.plan_query(ctx, sp, dtype)
            x = inputs.chunk_input(sp, dtype, wl["id"], lid, ci, "cuda")
            To, Ho, Wo, L = c3c.output_dims(sp, dtype)
            y, ybuf = guarded((sp["N"], sp["Co"], To, Ho, Wo), dtype)
            cache_new, cbuf = guarded((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), dtype)
            say(f"{name}/{lname} chunk {ci} mode={mode} kernel={plan['kernel']} "
                f"tile={plan['tile_co']}x{plan['tile_h']}x{plan['tile_w']} "
                f"{'check' if ci in todo else ''}")
            c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b, y, cache_new)
            torch.cuda.synchronize()
            assert bool(torch.isfinite(y).all().item()), f"{lname} chunk {ci}: y not fully written"
            assert bool(torch.isfinite(cache_new).all().item()), f"{lname} chunk {ci}: cache'"
            assert guards_intact(ybuf) and guards_intact(cbuf), f"{lname} chunk {ci}: guard band"
            route, why = oracle.route(sp, dtype, forced)
            expect["calls"] += 1
            if route == "fast":
                expect["fast"] += 1
            else:
                expect["fallback"] += 1
                expect["forced" if forced else "unsupported"] += 1
                hist[(why, lname)] = hist.get((why, lname), 0) + 1
            assert (plan["route"], plan["reason"]) == (route, why)
            hx, hc = host(x), host(cache) if cache is not None else None
            ref_cache = oracle.cache_update(sp, dtype, hx, hc)
            assert np.array_equal(_bits(cache_new, dtype), ref_cache), f"{lname} cache {ci}"
            if ci in todo or (lname, ci) in FULL:
                oin = (hx, hc, host(w), host(b))
                if (lname, ci) in FULL:
                    say(f"  full compare ({y.numel()} outputs)")
                    ref = oracle.conv3d(sp, dtype, *oin)
                    m = check(as_f64(y), ref, dtype, f"{lname} chunk {ci}")
                    del ref
                    say(f"  full: rel={m['rel']:.3e} rmse={m['rmse']:.3e} cos={m['cos']:.8f}")
                pl = _planes(tuple(y.shape), plan)
                worst = check_planes(y, sp, dtype, pl, oin, f"{lname} chunk {ci}")
                idx = sample_indices(tuple(y.shape), plan, 2048, seed=ci)
                ref = oracle.conv3d_points(sp, dtype, *oin, idx)
                got = as_f64(y.reshape(-1)[torch.from_numpy(idx).cuda()])
                m = check(got, ref, dtype, f"{lname} chunk {ci}")
                say(f"  {len(pl)} planes: worst rel={worst:.3e}; {idx.size} points "
                    f"(tile borders {plan['tile_h']}x{plan['tile_w']}): rel={m['rel']:.3e} "
                    f"cos={m['cos']:.8f}")
            cache = cache_new if cache_new.numel() else None
            del y, ybuf
    c = ctx.counters()
    for k, v in expect.items():
        assert c[k] == v, (k, c, expect)
    assert c["strict_rejects"] == c["fast_error"] == c["failed"] == 0
    got_hist = {}
    for r, desc, n in ctx.fallback_shapes():
        got_hist[r] = got_hist.get(r, 0) + n
    want_hist = {}
    for (r, _), n in hist.items():
        want_hist[r] = want_hist.get(r, 0) + n
    assert got_hist == want_hist, (got_hist, want_hist)
    return ctx


def test_tiny_f32_stream_full_compare():
    _stream("tiny_f32")


def test_low_res_stream_21_chunks():
    _stream("low_res", check_chunks=range(21))


def test_mid_res_layers():
    _stream("mid_res")


def test_full_res_layer():
    _stream("full_res")


def test_stack_720p():
    ctx = _stream("stack_720p")
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"], c["unsupported"]) == (25, 20, 5, 5)
    shapes = ctx.fallback_shapes()
    assert len(shapes) == 1 and shapes[0][0] == "kt1" and shapes[0][2] == 5
    assert shapes[0][1]["Kt"] == 1 and shapes[0][1]["Ci"] == 320 and shapes[0][1]["Co"] == 160


def test_temporal_convs():
    """Temporal convolutions (kernel 3x1x1) on the fast route: the 1x1-spatial
    kernel, unit stride with a 2-frame cache and stride 2 with a 1-frame
    cache, streamed over 5 chunks."""
    ctx = _stream("temporal")
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (15, 15, 0)


def test_head_conv():
    """The decoder's output head (96 -> 3 channels at 480x832) on the head
    kernel, streamed over 5 chunks."""
    ctx = _stream("head", check_chunks=(0, -1))
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (5, 5, 0)


# ---------------------------------------------------------------- the baseline
# Every call of every workload forced onto the fallback route at full size:
# zero fast hits, every call counted as forced, the same outputs (first and
# last chunk checked) and bit-exact caches on every chunk.

@pytest.mark.parametrize("name", ["tiny_f32", "low_res", "mid_res", "full_res", "stack_720p"])
def test_forced_fallback_full_size(name):
    ctx = _stream(name, check_chunks=(0, -1), mode=c3c.MODE_FORCE_FALLBACK)
    c = ctx.counters()
    assert c["fast"] == 0 and c["forced"] == c["fallback"] == c["calls"]
    assert all(r == "forced" for r, _, _ in ctx.fallback_shapes())

