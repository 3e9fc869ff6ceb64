"""GPU parity: the HIP library (called through its C ABI) against the CPU
oracle, element by element on the same seeded inputs.

Bar: max|err| / max|ref| <= 1e-5 (fp32) and <= 2e-2 (bf16) per output tensor
per call; cache contents, route counters and output shapes bit-exact; no
NaN/Inf; every output element written (poisoned buffers).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs
from paper_2609_31938_amd.inputs import spec

from gpu_util import (TOL, as_f64, check, chunk, guarded, guards_intact, host, layer, metrics,
                      oracle_args, run, say)

pytestmark = pytest.mark.gpu


def _case(sp, dtype, mode=0, seed=0, ws=False, kernel=None):
    """One call on fresh inputs, compared in full with the oracle.  The
    outputs are NaN-filled and sit inside NaN guard bands that must stay
    untouched.  ws: attach a split-K workspace of the size the call asks
    for.  kernel: the kernel the plan must name."""
    ctx = c3c.Context(mode)
    w, b = layer(sp, dtype, 901, seed)
    x = chunk(sp, dtype, 901, seed, 0)
    cache = chunk(dict(sp, T=sp["Tc"]), dtype, 901, seed, 1)
    wpack = None
    if c3c.route_query(None, sp, dtype)[0] == "fast":
        wpack = c3c.weight_repack(ctx, sp, w)
    need = c3c.workspace_bytes(sp, dtype) if ws else 0
    wsb = None
    if need:
        wsb = torch.empty(need // 4, dtype=torch.float32, device="cuda")
        ctx.set_workspace(wsb)
    plan = c3c.plan_query(ctx, sp, dtype, need)
    say(f"case {dtype} {sp} mode={mode} plan={plan}")
    if kernel is not None:
        assert plan["kernel"] == kernel, plan
    To, Ho, Wo, L = c3c.output_dims(sp, dtype)
    y, ybuf = guarded((sp["N"], sp["Co"], To, Ho, Wo), dtype)
    co, cbuf = guarded((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), dtype)
    y, co = c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b, y, co)
    torch.cuda.synchronize()
    assert guards_intact(ybuf) and guards_intact(cbuf), "a write outside the outputs"
    args = oracle_args(sp, x, cache, w, b)
    ref = oracle.conv3d(sp, dtype, *args)
    assert tuple(y.shape) == ref.shape
    m = check(as_f64(y), ref, dtype, str(sp))
    ref_cache = oracle.cache_update(sp, dtype, args[0], args[1])
    got_cache = host(co)
    if dtype == "bf16":
        got_cache = got_cache.view(torch.int16).numpy().view(np.uint16)
    else:
        got_cache = got_cache.numpy()
    assert np.array_equal(got_cache, ref_cache)
    return ctx, y, m


# ---------------------------------------------------------------- repack

@pytest.mark.parametrize("Ci,Co,Kt,Kh", [(48, 80, 3, 3), (320, 160, 5, 3), (40, 21, 3, 1),
                                         (64, 16, 2, 3), (33, 17, 6, 3), (96, 3, 1, 3)])
def test_repack_layout_matches_its_definition(Ci, Co, Kt, Kh):
    """bf16 packed weights against the layout written out on the host: the
    16-byte slot of lane L in fragment (tap, chunk, output fragment) holds
    w[16 f + L % 16][32 chunk + 8 (L / 16) + e][tap], e = 0..7, zero past Ci
    / Co (45 and 54 taps: both sides of the block kernel's tap limit)."""
    sp = spec(N=1, Ci=Ci, Co=Co, T=2, Tc=2, H=4, W=4, Kt=Kt, Kh=Kh, Kw=Kh)
    say(f"repack layout {Ci}->{Co} Kt={Kt} K={Kh}")
    ctx = c3c.Context()
    w, _ = layer(sp, "bf16")
    wp = c3c.weight_repack(ctx, sp, w)
    torch.cuda.synchronize()
    taps = Kt * Kh * Kh
    chunks, frags = (Ci + 31) // 32, (Co + 15) // 16
    wb = w.view(torch.int16).cpu().numpy().view(np.uint16).reshape(Co, Ci, taps)
    pad = np.zeros((frags * 16, chunks * 32, taps), np.uint16)
    pad[:Co, :Ci] = wb
    # [co = 16 f + r][ci = 32 c + 8 g + e][tap] -> [tap][c][f][g][r][e]
    want = pad.reshape(frags, 16, chunks, 4, 8, taps).transpose(5, 2, 0, 3, 1, 4)
    got = wp.view(torch.int16).cpu().numpy().view(np.uint16).reshape(taps, chunks, frags, 4, 16, 8)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("Ci,Co,dtype", [(48, 80, "bf16"), (384, 384, "bf16"), (3, 5, "bf16"),
                                         (32, 32, "f32"), (7, 45, "f32")])
def test_repack_round_trip(Ci, Co, dtype):
    sp = spec(N=1, Ci=Ci, Co=Co, T=2, Tc=2, H=4, W=4)
    say(f"repack {Ci}->{Co} {dtype}")
    ctx = c3c.Context()
    w, _ = layer(sp, dtype)
    wp = c3c.weight_repack(ctx, sp, w)
    back = c3c.weight_unpack(sp, wp)
    torch.cuda.synchronize()
    assert torch.equal(back.view(torch.int16) if dtype == "bf16" else back,
                       w.view(torch.int16) if dtype == "bf16" else w)
    assert ctx.counters()["repacks"] == 1
    # the padding of partial fragments is zero: total |wpack| == total |w|
    assert torch.equal(wp.float().abs().sum(), w.float().abs().sum())


# ---------------------------------------------------------------- fast route

FAST_CASES = [
    ("bf16", dict(N=1, Ci=48, Co=80, T=3, Tc=2, H=37, W=70)),
    ("bf16", dict(N=2, Ci=32, Co=64, T=2, Tc=1, H=9, W=33)),
    ("bf16", dict(N=1, Ci=160, Co=96, T=4, Tc=2, H=20, W=100)),
    ("bf16", dict(N=1, Ci=96, Co=96, T=2, Tc=2, H=20, W=136)),         # 6 x 64 tiles, ragged both ways
    ("bf16", dict(N=1, Ci=16, Co=32, T=1, Tc=0, H=5, W=5)),
    ("bf16", dict(N=1, Ci=24, Co=40, T=2, Tc=3, H=11, W=65)),          # p_l < 0
    ("bf16", dict(N=1, Ci=64, Co=192, T=4, Tc=2, H=16, W=64)),
    # the 160-channel tiles (97..191 output channels): 4x80 ragged in both
    # directions and in the channel tile, two channel tiles, and 10x32
    ("bf16", dict(N=1, Ci=64, Co=160, T=3, Tc=2, H=22, W=170)),
    ("bf16", dict(N=1, Ci=72, Co=130, T=2, Tc=2, H=13, W=96)),
    ("bf16", dict(N=2, Ci=40, Co=181, T=2, Tc=1, H=9, W=83)),
    ("bf16", dict(N=1, Ci=48, Co=320, T=2, Tc=2, H=10, W=88)),
    ("bf16", dict(N=1, Ci=40, Co=150, T=4, Tc=2, H=333, W=30)),
    # the 128-channel 4x80 tile: two exact channel tiles, ragged rows and columns
    ("bf16", dict(N=1, Ci=40, Co=256, T=2, Tc=2, H=9, W=90)),
    ("bf16", dict(N=1, Ci=8, Co=8, T=5, Tc=4, H=6, W=40, d_t=2, p_base=4)),  # temporal dilation
    ("bf16", dict(N=1, Ci=20, Co=36, T=2, Tc=2, H=7, W=9, Kt=5, p_base=4)),  # Kt = 5
    ("bf16", dict(N=1, Ci=12, Co=20, T=3, Tc=2, H=6, W=35, p_r=1)),          # right pad
    ("f32", dict(N=1, Ci=32, Co=32, T=2, Tc=2, H=32, W=32)),
    ("f32", dict(N=2, Ci=7, Co=45, T=3, Tc=1, H=13, W=34)),
    ("f32", dict(N=1, Ci=33, Co=70, T=1, Tc=2, H=10, W=66)),
    # few output channels (a head conv to RGB): the 16-channel tile
    ("bf16", dict(N=1, Ci=96, Co=3, T=4, Tc=2, H=20, W=72)),
    ("bf16", dict(N=1, Ci=40, Co=16, T=2, Tc=2, H=9, W=35)),             # unaligned width
    ("bf16", dict(N=2, Ci=33, Co=1, T=3, Tc=0, H=17, W=64)),
    # 1x1 spatial kernels (temporal convolutions): per-frame matrix products
    ("bf16", dict(N=1, Ci=96, Co=192, T=4, Tc=2, H=16, W=40, Kh=1, Kw=1)),
    ("bf16", dict(N=2, Ci=40, Co=200, T=3, Tc=2, H=9, W=24, Kh=1, Kw=1)),    # chunk tail, 2 co tiles
    ("bf16", dict(N=1, Ci=33, Co=17, T=5, Tc=2, H=5, W=7, Kh=1, Kw=1)),      # H*W = 35: unaligned
    ("bf16", dict(N=1, Ci=64, Co=64, T=6, Tc=0, H=8, W=16, Kh=1, Kw=1, s_t=2)),  # stride 2
    ("bf16", dict(N=1, Ci=32, Co=48, T=4, Tc=4, H=8, W=8, Kh=1, Kw=1, d_t=2, p_base=4)),
    ("bf16", dict(N=1, Ci=16, Co=32, T=2, Tc=0, H=4, W=64, Kt=2, Kh=1, Kw=1)),
    ("bf16", dict(N=1, Ci=24, Co=40, T=3, Tc=2, H=6, W=20, Kh=1, Kw=1, p_r=1)),
    ("bf16", dict(N=1, Ci=300, Co=70, T=5, Tc=1, H=3, W=37, Kh=1, Kw=1, s_t=3, p_base=2)),
    ("f32", dict(N=1, Ci=20, Co=40, T=3, Tc=2, H=10, W=12, Kh=1, Kw=1)),
    ("f32", dict(N=1, Ci=8, Co=8, T=5, Tc=0, H=6, W=6, Kh=1, Kw=1, s_t=2)),
]


@pytest.mark.parametrize("dtype,over", FAST_CASES)
def test_fast_route_matches_oracle(dtype, over):
    sp = spec(**over)
    ctx, _, m = _case(sp, dtype)
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (1, 1, 0)
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")


# An unsplit call whose tiles fill less than one round of the compute units
# may take 64-channel 4x64 tiles (two output-channel fragments per wave);
# C3C_MODE_CHANNEL_TILES keeps the tile its output-channel count selects.
# These cases (above, and a few more for the smaller tile: W not a multiple
# of 8, temporal dilation, five taps) run on both tilings: each against the
# oracle, the two outputs and caches bit-identical (every output element's
# products are accumulated in the same order on every tile).
RETILED = [
    (dict(N=1, Ci=64, Co=192, T=4, Tc=2, H=16, W=64), (192, 4, 64)),
    (dict(N=1, Ci=64, Co=160, T=3, Tc=2, H=22, W=170), (160, 4, 80)),
    (dict(N=1, Ci=72, Co=130, T=2, Tc=2, H=13, W=96), (160, 4, 80)),
    (dict(N=2, Ci=40, Co=181, T=2, Tc=1, H=9, W=83), (128, 4, 80)),
    (dict(N=1, Ci=48, Co=320, T=2, Tc=2, H=10, W=88), (160, 4, 80)),
    (dict(N=1, Ci=40, Co=256, T=2, Tc=2, H=9, W=90), (128, 4, 80)),
    (dict(N=1, Ci=40, Co=128, T=2, Tc=2, H=9, W=70), (128, 4, 80)),
    (dict(N=1, Ci=24, Co=128, T=3, Tc=4, H=8, W=64, d_t=2, p_base=4), (128, 4, 80)),
    (dict(N=1, Ci=20, Co=100, T=2, Tc=2, H=7, W=72, Kt=5, p_base=4), (128, 4, 80)),
]


@pytest.mark.parametrize("over,tile", RETILED)
def test_small_tiles_match_the_channel_tiles(over, tile):
    sp = spec(**over)
    plans = [c3c.plan_query(c3c.Context(m), sp, "bf16") for m in (0, c3c.MODE_CHANNEL_TILES)]
    assert [(p["tile_co"], p["tile_h"], p["tile_w"]) for p in plans] == [(64, 4, 64), tile], plans
    outs = []
    for mode in (0, c3c.MODE_CHANNEL_TILES):
        ctx, y, m = _case(sp, "bf16", mode, kernel="conv3d_bf16")
        c = ctx.counters()
        assert (c["calls"], c["fast"], c["fallback"]) == (1, 1, 0)
        say(f"  mode={mode} rel={m['rel']:.3e} cos={m['cos']:.8f}")
        outs.append(host(y).view(torch.int16))
    assert torch.equal(outs[0], outs[1])


# No bias (has_bias = 0) on every kernel that loads the bias before its
# epilogue: the 3x3 kernel's 96-, 64- (W not a multiple of 8) and 160-channel
# tiles, both 1x1 kernels of the temporal route (several output frames, and
# one), the pointwise kernel on the fast route and, for a 1x1x1 call, on the
# fallback, and the head kernel.
NO_BIAS = [
    (dict(N=1, Ci=48, Co=80, T=3, Tc=2, H=37, W=72), "conv3d_bf16"),
    (dict(N=1, Ci=40, Co=200, T=2, Tc=2, H=9, W=37), "conv3d_bf16"),
    (dict(N=1, Ci=40, Co=160, T=4, Tc=2, H=64, W=160), "conv3d_bf16"),
    (dict(N=1, Ci=64, Co=384, T=4, Tc=2, H=32, W=64, Kh=1, Kw=1), "tap1x1"),
    (dict(N=1, Ci=64, Co=384, T=1, Tc=2, H=64, W=128, Kh=1, Kw=1), "tap1x1"),
    (dict(N=1, Ci=64, Co=96, T=3, Tc=2, H=8, W=40, Kh=1, Kw=1), "pointwise"),
    (dict(N=1, Ci=64, Co=96, T=2, Tc=0, H=16, W=64, Kt=1, Kh=1, Kw=1), "pointwise"),
    (dict(N=1, Ci=96, Co=3, T=2, Tc=2, H=12, W=48), "head"),
]


@pytest.mark.parametrize("over,kernel", NO_BIAS)
def test_no_bias_matches_oracle(over, kernel):
    sp = spec(**over, has_bias=0)
    ctx, _, m = _case(sp, "bf16", kernel=kernel)
    c = ctx.counters()
    assert c["calls"] == 1 and c["failed"] == c["fast_error"] == 0
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")


# ---------------------------------------------------------------- fallback route

FALLBACK_CASES = FAST_CASES + [
    ("bf16", dict(N=1, Ci=32, Co=16, T=4, Tc=0, H=12, W=20, Kt=1, Kh=1, Kw=1)),  # 1x1x1
    ("bf16", dict(N=2, Ci=6, Co=4, T=5, Tc=2, H=9, W=7, s_t=2)),                # stride_t 2
    ("bf16", dict(N=1, Ci=8, Co=12, T=3, Tc=2, H=10, W=11, groups=4)),
    ("f32", dict(N=1, Ci=5, Co=6, T=3, Tc=1, H=9, W=13, Kh=5, Kw=3, s_h=2, d_w=2, p_w=2)),
    ("f32", dict(N=1, Ci=4, Co=4, T=2, Tc=2, H=6, W=6, p_r=2)),
    ("f32", dict(N=1, Ci=4, Co=4, T=4, Tc=2, H=6, W=6, p_r=-1)),
    ("f16", dict(N=1, Ci=16, Co=24, T=3, Tc=2, H=10, W=18)),
    # (input channel, tap) pairs spanning several staged weight chunks
    ("f32", dict(N=1, Ci=3, Co=5, T=7, Tc=0, H=9, W=9, Kt=7, Kh=7, Kw=7, p_base=6)),
    ("bf16", dict(N=2, Ci=300, Co=70, T=2, Tc=0, H=6, W=21, Kt=1, Kh=1, Kw=1)),
    ("bf16", dict(N=1, Ci=40, Co=33, T=3, Tc=2, H=5, W=600, Kh=3, Kw=5, p_w=2)),
    # pointwise (1x1x1) calls on the matrix-core fallback kernel: ragged pixel
    # tile, channel-chunk tail, two output-channel tiles
    ("bf16", dict(N=1, Ci=40, Co=200, T=3, Tc=0, H=9, W=24, Kt=1, Kh=1, Kw=1)),
    # fp16, a cached frame read and carried (p_base = 1)
    ("f16", dict(N=2, Ci=64, Co=24, T=2, Tc=1, H=4, W=34, Kt=1, Kh=1, Kw=1, p_base=1)),
    # temporal stride 2
    ("bf16", dict(N=1, Ci=16, Co=8, T=5, Tc=0, H=8, W=16, Kt=1, Kh=1, Kw=1, s_t=2)),
    # left pad past the cache: the first output frames are the bias alone
    ("bf16", dict(N=1, Ci=24, Co=48, T=2, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1, p_base=2)),
    ("bf16", dict(N=1, Ci=24, Co=48, T=2, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1, p_base=2,
                  has_bias=0)),
    # H*W not a multiple of 8: the generic kernel
    ("bf16", dict(N=1, Ci=8, Co=16, T=2, Tc=0, H=3, W=5, Kt=1, Kh=1, Kw=1)),
    # the resident-weight pointwise kernel (Co <= 160, at most 11 channel
    # chunks): all 11 chunks and 160 channels; ragged output fragments and a
    # pixel tail; a right pad (the last output frame is the bias alone);
    # stride 2 reading a cached frame; more tiles than workgroups (each
    # workgroup walks two tiles, the ring running on across them)
    ("bf16", dict(N=1, Ci=352, Co=160, T=2, Tc=0, H=10, W=40, Kt=1, Kh=1, Kw=1)),
    ("bf16", dict(N=2, Ci=96, Co=100, T=3, Tc=0, H=9, W=24, Kt=1, Kh=1, Kw=1)),
    ("bf16", dict(N=1, Ci=40, Co=24, T=3, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1, p_r=1)),
    ("f16", dict(N=1, Ci=48, Co=40, T=4, Tc=1, H=8, W=40, Kt=1, Kh=1, Kw=1, s_t=2, p_base=1)),
    ("bf16", dict(N=1, Ci=64, Co=24, T=2, Tc=0, H=64, W=1024, Kt=1, Kh=1, Kw=1)),
]


@pytest.mark.parametrize("dtype,over", FALLBACK_CASES)
def test_fallback_route_matches_oracle(dtype, over):
    sp = spec(**over)
    forced = oracle.route(sp, dtype)[0] == "fast"
    mode = c3c.MODE_FORCE_FALLBACK if forced else 0
    ctx, _, m = _case(sp, dtype, mode)
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"]) == (1, 0, 1)
    assert c["forced"] == int(forced) and c["unsupported"] == int(not forced)
    shapes = ctx.fallback_shapes()
    assert len(shapes) == 1 and shapes[0][2] == 1
    assert shapes[0][0] == oracle.route(sp, dtype, forced)[1]


def test_injected_fast_failure_falls_back():
    sp = spec(N=1, Ci=16, Co=32, T=2, Tc=2, H=8, W=40)
    ctx, _, _ = _case(sp, "bf16", c3c.MODE_INJECT_FAST_FAILURE)
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"], c["fast_error"]) == (1, 0, 1, 1)
    assert ctx.fallback_shapes()[0][0] == "fast_error"


# ---------------------------------------------------------------- edge cases

def test_empty_chunk_keeps_the_cache():
    # T = 0: no output frame (fallback, reason no_output), cache' == cache
    sp = spec(N=1, Ci=8, Co=8, T=0, Tc=2, H=5, W=7)
    ctx, y, _ = _case(sp, "bf16")
    assert y.numel() == 0
    assert ctx.fallback_shapes()[0][0] == "no_output"


def test_first_chunk_without_cache_equals_zero_cache():
    sp0 = spec(N=1, Ci=32, Co=48, T=3, Tc=0, H=10, W=40)
    sp2 = dict(sp0, Tc=2)
    ctx = c3c.Context()
    w, b = layer(sp0, "bf16")
    x = chunk(sp0, "bf16")
    wp = c3c.weight_repack(ctx, sp0, w)
    y0, c0 = run(ctx, sp0, x, None, w, wp, b)
    zero = torch.zeros((1, 32, 2, 10, 40), dtype=torch.bfloat16, device="cuda")
    y2, c2 = run(ctx, sp2, x, zero, w, wp, b)
    assert torch.equal(y0.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(c0.view(torch.int16), c2.view(torch.int16))


def test_deterministic_bitwise():
    sp = spec(N=1, Ci=96, Co=160, T=4, Tc=2, H=24, W=72)
    ctx = c3c.Context()
    w, b = layer(sp, "bf16")
    x = chunk(sp, "bf16")
    cache = chunk(dict(sp, T=2), "bf16", ci=1)
    wp = c3c.weight_repack(ctx, sp, w)
    y1, _ = run(ctx, sp, x, cache, w, wp, b)
    y2, _ = run(ctx, sp, x, cache, w, wp, b)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_streaming_equals_whole_sequence_on_gpu(dtype):
    Ci, Co, H, W = 24, 40, 9, 45
    sizes = [2, 1, 3, 2]
    whole = spec(N=1, Ci=Ci, Co=Co, T=sum(sizes), Tc=0, H=H, W=W)
    ctx = c3c.Context()
    w, b = layer(whole, dtype)
    X = chunk(whole, dtype)
    wp = c3c.weight_repack(ctx, whole, w)
    ref = oracle.conv3d(whole, dtype, host(X), None, host(w), host(b))
    yw, _ = run(ctx, whole, X, None, w, wp, b)
    check(as_f64(yw), ref, dtype, "whole")
    cache, outs, t0 = None, [], 0
    for T in sizes:
        sp = spec(N=1, Ci=Ci, Co=Co, T=T, Tc=0 if cache is None else cache.shape[2], H=H, W=W)
        y, cache = run(ctx, sp, X[:, :, t0:t0 + T].contiguous(), cache, w, wp, b)
        outs.append(y)
        t0 += T
    ys = torch.cat(outs, dim=2)
    check(as_f64(ys), ref, dtype, "streamed")
    assert ctx.counters()["fast"] == 1 + len(sizes)


@pytest.mark.parametrize("seed", range(40))
def test_fuzz_off_grid_shapes(seed):
    rng = np.random.default_rng(4242 + seed)
    dtype = "bf16" if seed % 4 else "f32"
    d_t = int(rng.choice([1, 1, 2]))
    sp = spec(N=int(rng.integers(1, 3)), Ci=int(rng.integers(1, 70)), Co=int(rng.integers(1, 100)),
              T=int(rng.integers(1, 5)), Tc=int(rng.integers(0, 4)), H=int(rng.integers(1, 23)),
              W=int(rng.integers(1, 90)), d_t=d_t, Kt=int(rng.choice([2, 3, 3])))
    if sp["Tc"] > sp["p_base"] + 1:
        sp["Tc"] = sp["p_base"] + 1
    ctx, _, m = _case(sp, dtype, seed=seed)
    assert ctx.counters()["fast"] == 1


# ---------------------------------------------------------------- 1x1: the 4-wave kernel
# Temporal convolutions that take the 4-wave 1x1 kernel (192-channel x
# 128-pixel workgroups): it is chosen unless its padded output channels
# exceed the 160-channel pointwise kernel's by more than 10%, when there are
# at least half as many workgroups as compute units and H*W is a multiple of 8.
# Ragged output channels, a channel-chunk tail, a ragged last pixel tile,
# stride 2, dilation with partial first frames.
TAP1X1_CASES = [
    dict(N=2, Ci=64, Co=180, T=4, Tc=2, H=64, W=80),
    dict(N=1, Ci=40, Co=192, T=8, Tc=2, H=64, W=80),
    dict(N=2, Ci=72, Co=350, T=4, Tc=2, H=56, W=72, p_r=1),
    dict(N=1, Ci=64, Co=384, T=16, Tc=1, H=64, W=80, s_t=2, p_base=1),
    dict(N=1, Ci=48, Co=576, T=6, Tc=0, H=56, W=64, d_t=2, p_base=4),
    dict(N=2, Ci=48, Co=768, T=2, Tc=2, H=30, W=52),             # H*W = 1560: ragged tile
    # frame groups: the first group's taps clipped by the left pad, an odd
    # number of output frames (the last group half used)
    dict(N=1, Ci=64, Co=192, T=5, Tc=0, H=64, W=64, p_base=2),
    # stride 3 (one output frame per group), and a new cache frame that no
    # output frame reads (the copy kernel writes it)
    dict(N=1, Ci=40, Co=192, T=9, Tc=1, H=96, W=64, s_t=3, p_base=1),
    # Kt = 2 at stride 2: two-tap slots, new cache again by the copy
    dict(N=1, Ci=64, Co=180, T=8, Tc=1, H=64, W=64, Kt=2, s_t=2, p_base=1),
    # one output frame (all taps of a chunk per stage), and one with no
    # cache whose first two taps fall on the left pad (one live tap; the
    # new cache is the chunk's only frame)
    dict(N=1, Ci=96, Co=384, T=1, Tc=2, H=128, W=128),
    dict(N=2, Ci=40, Co=180, T=1, Tc=0, H=64, W=128, p_base=2),
    # Kt = 4: the one-frame-per-workgroup kernel
    dict(N=1, Ci=32, Co=192, T=4, Tc=3, H=64, W=64, Kt=4),
]


def _takes_tap1x1(sp, To):
    pad = lambda tile: -(-sp["Co"] // tile) * tile
    blocks = -(-sp["H"] * sp["W"] // 128) * -(-sp["Co"] // 192) * To * sp["N"]
    return 10 * pad(192) <= 11 * pad(160) and 2 * blocks >= 256 and (sp["H"] * sp["W"]) % 8 == 0


@pytest.mark.parametrize("over", TAP1X1_CASES)
def test_tap1x1_kernel_matches_oracle(over):
    sp = spec(Kh=1, Kw=1, **over)
    To, _, _, _ = c3c.output_dims(sp, "bf16")
    assert _takes_tap1x1(sp, To)
    ctx, _, m = _case(sp, "bf16")
    assert ctx.counters()["fast"] == 1
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")


# ---------------------------------------------------------------- few output channels
# The head kernel (Co <= 5, W a multiple of 8): the 9 spatial taps x Co as
# matrix-core columns, then a 3x3 gather-sum.  Every Co it serves, ragged
# rows (H not a multiple of the 6-row tile) and columns (W not a multiple of
# 64), a channel-chunk tail, dilation, p_l < 0, no cache, N = 2, Kt = 2,
# more output frames than one pass of the kernel takes, and weight tables
# that take the three-buffer form.
HEAD_CASES = [
    dict(N=1, Ci=96, Co=3, T=4, Tc=2, H=37, W=136),
    dict(N=1, Ci=40, Co=1, T=2, Tc=2, H=20, W=72),
    dict(N=2, Ci=64, Co=2, T=3, Tc=1, H=13, W=64),
    dict(N=1, Ci=48, Co=4, T=2, Tc=3, H=19, W=80),
    dict(N=1, Ci=32, Co=5, T=3, Tc=4, H=11, W=40, d_t=2),
    dict(N=1, Ci=72, Co=3, T=3, Tc=0, H=25, W=200),
    dict(N=1, Ci=24, Co=3, T=2, Tc=1, H=8, W=8, Kt=2),
    # more output frames than one group (4, or 2 with three column
    # fragments): the new cache written by the group that first stages it
    dict(N=1, Ci=40, Co=3, T=6, Tc=2, H=14, W=56),
    dict(N=2, Ci=36, Co=5, T=5, Tc=2, H=9, W=48),
    # weight tables too large for four stage buffers: the three-buffer form
    # (3 x 3 x 3 = 27 entries; 3 x 5 x 2 = 30 with a channel-chunk tail)
    dict(N=1, Ci=96, Co=5, T=3, Tc=2, H=13, W=48),
    dict(N=1, Ci=150, Co=3, T=4, Tc=2, H=16, W=104),
]


@pytest.mark.parametrize("over", HEAD_CASES)
def test_head_kernel_matches_oracle(over):
    sp = spec(**over)
    assert sp["Co"] <= 5 and sp["W"] % 8 == 0  # takes the head kernel
    ctx, _, m = _case(sp, "bf16")
    assert ctx.counters()["fast"] == 1
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")


# ---------------------------------------------------------------- one temporal tap
# A (1,3,3) call (a per-frame spatial convolution) routes fast: the 3x3
# kernels with a single tap, every tile configuration, the head kernel, fp32,
# and W not a multiple of 8.
KT1_CASES = [
    ("bf16", dict(N=1, Ci=64, Co=160, T=3, Tc=0, H=20, W=80)),
    ("bf16", dict(N=2, Ci=40, Co=96, T=2, Tc=0, H=13, W=37)),
    ("bf16", dict(N=1, Ci=48, Co=192, T=2, Tc=0, H=12, W=64)),
    ("bf16", dict(N=1, Ci=96, Co=3, T=2, Tc=0, H=19, W=104)),
    ("f32", dict(N=1, Ci=20, Co=36, T=2, Tc=0, H=9, W=21)),
]


@pytest.mark.parametrize("dtype,over", KT1_CASES)
def test_single_temporal_tap_routes_fast(dtype, over):
    sp = spec(Kt=1, p_base=0, **over)
    assert c3c.route_query(None, sp, dtype) == ("fast", "none")
    ctx, _, m = _case(sp, dtype)
    assert ctx.counters()["fast"] == 1
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")
