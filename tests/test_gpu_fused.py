"""GPU parity of the fused residual-block form (c3c_conv3d_causal_cached_fused)
against the oracle's fused composition, on the same seeded inputs.

Bar: y within max|err| / max|ref| <= 2e-2 (bf16); cache frames that come from
the old cache bit-exact; cache frames that come from the new chunk (the
prologue's output) within one bf16 step of the oracle's: the kernels evaluate
SiLU in fp32 with the hardware exponential and reciprocal, the oracle in
fp64, so a value within a few fp32 ulp of a bf16 rounding midpoint may round
the other way (the test also bounds how often that happens).  Every output
element written (NaN-poisoned buffers), counters as for the plain call.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs
from paper_2609_31938_amd.inputs import spec

from gpu_util import as_f64, check, chunk, host, layer, say

pytestmark = pytest.mark.gpu

WID = 907


def _bits(t):
    return host(t).contiguous().view(torch.int16).numpy().view(np.uint16)


def _check_cache(got, ref, sp):
    """Old-cache frames bit-exact, new-chunk frames within one bf16 step."""
    L = ref.shape[2]
    Z = sp["Tc"] + sp["T"]
    from_x = np.array([Z - L + j >= sp["Tc"] for j in range(L)], bool)
    if (~from_x).any():
        assert np.array_equal(got[:, :, ~from_x], ref[:, :, ~from_x])
    if from_x.any():
        g = got[:, :, from_x].astype(np.int32)
        r = ref[:, :, from_x].astype(np.int32)
        # same sign: adjacent bit patterns are adjacent values; across zero
        # only the two zeros and the smallest values may meet
        same = (g ^ r) & 0x8000 == 0
        step = np.where(same, np.abs(g - r), (g & 0x7fff) + (r & 0x7fff))
        assert step.max() <= 1, step.max()
        frac = np.count_nonzero(step) / step.size
        assert frac <= 1e-3, frac
        return frac
    return 0.0


def _run(sp, mode=0, pro=True, res=True, inplace=False, ws=False, seed=0, ctx=None,
         x=None, cache=None, expect_fast=None):
    """One fused call on fresh (or given) inputs, compared in full with the oracle."""
    say(f"fused case {sp} mode={mode} pro={pro} res={res} inplace={inplace} ws={ws}")
    ctx = ctx or c3c.Context(mode)
    w, b = layer(sp, "bf16", WID, seed)
    x = chunk(sp, "bf16", WID, seed, 0) if x is None else x
    if cache is None and sp["Tc"]:
        cache = chunk(dict(sp, T=sp["Tc"]), "bf16", WID, seed, 1)
    route = c3c.route_query(None, sp, "bf16")[0]
    wpack = c3c.weight_repack(ctx, sp, w) if route == "fast" else None
    To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
    yshape = (sp["N"], sp["Co"], To, Ho, Wo)
    scale, shift = inputs.affine_inputs(sp, WID, seed, 0, "cuda") if pro else (None, None)
    r = inputs.residual_input(yshape, "bf16", WID, seed, 0, "cuda") if res else None
    r_host = host(r) if r is not None else None
    if ws:
        need = c3c.workspace_bytes(sp, "bf16")
        assert need > 0, "this case should split"
        ctx.set_workspace(torch.empty(need // 4, dtype=torch.float32, device="cuda"))
    if inplace:
        y = r.clone()
        residual = y
    else:
        y = torch.full(yshape, float("nan"), dtype=torch.bfloat16, device="cuda")
        residual = r
    co = torch.full((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), float("nan"), dtype=torch.bfloat16,
                    device="cuda")
    before = ctx.counters()
    y, co = c3c.conv3d_causal_cached_fused(ctx, sp, x, cache, w, wpack, b, scale, shift,
                                           residual, y, co)
    torch.cuda.synchronize()
    after = ctx.counters()
    if expect_fast is not None:
        assert after["fast"] - before["fast"] == (1 if expect_fast else 0)
    ref_y, ref_c = oracle.conv3d_fused(
        sp, host(x), host(cache) if cache is not None else None, host(w), host(b),
        host(scale) if pro else None, host(shift) if pro else None, r_host)
    m = check(as_f64(y), ref_y, "bf16", str(sp))
    frac = _check_cache(_bits(co), ref_c, sp) if L else 0.0
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f} cache steps={frac:.2e}")
    return ctx, y, co


# ---------------------------------------------------------------- fast 3x3
FAST3 = [
    dict(N=1, Ci=48, Co=80, T=3, Tc=2, H=37, W=72),      # 96-channel tile, ragged rows
    dict(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80),     # 160-channel tiles
    dict(N=2, Ci=40, Co=192, T=2, Tc=1, H=16, W=64),     # 192-channel tile, chunk tail
    dict(N=1, Ci=32, Co=3, T=2, Tc=2, H=20, W=40),       # 16-channel head tile
    dict(N=1, Ci=24, Co=40, T=2, Tc=2, H=11, W=37),      # W not a multiple of 8
    dict(N=1, Ci=24, Co=40, T=2, Tc=3, H=11, W=64),      # p_l < 0
    dict(N=1, Ci=32, Co=64, T=3, Tc=0, H=16, W=48),      # first chunk, no cache
    dict(N=1, Ci=16, Co=32, T=3, Tc=4, H=12, W=40, d_t=2),
]


@pytest.mark.parametrize("over", FAST3)
def test_fused_fast_3x3(over):
    _run(spec(**over), expect_fast=True)


# The 160- and 192-channel cases above run unsplit on 64-channel 4x64 tiles
# (they fill few compute units); C3C_MODE_CHANNEL_TILES keeps their own tiles.
@pytest.mark.parametrize("over,tile", [(FAST3[1], (160, 4, 80)), (FAST3[2], (192, 4, 64))])
def test_fused_fast_3x3_on_the_channel_tiles(over, tile):
    sp = spec(**over)
    plans = [c3c.plan_query(c3c.Context(m), sp, "bf16") for m in (0, c3c.MODE_CHANNEL_TILES)]
    assert [(p["tile_co"], p["tile_h"], p["tile_w"]) for p in plans] == [(64, 4, 64), tile], plans
    _run(sp, mode=c3c.MODE_CHANNEL_TILES, expect_fast=True)


@pytest.mark.parametrize("mode", [0, c3c.MODE_CHANNEL_TILES])
@pytest.mark.parametrize("pro,res,inplace", [(True, False, False), (False, True, False),
                                             (True, True, True), (False, False, False)])
def test_fused_parts_and_in_place(pro, res, inplace, mode):
    _run(spec(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80), mode=mode, pro=pro, res=res,
         inplace=inplace, expect_fast=True)
    _run(spec(N=1, Ci=24, Co=40, T=2, Tc=2, H=11, W=37), mode=mode, pro=pro, res=res,
         inplace=inplace, expect_fast=True)


@pytest.mark.parametrize("over", [dict(N=1, Ci=128, Co=128, T=1, Tc=2, H=16, W=32),
                                  dict(N=1, Ci=128, Co=96, T=1, Tc=2, H=30, W=40)])
@pytest.mark.parametrize("inplace", [False, True])
def test_fused_split_k(over, inplace):
    _run(spec(**over), ws=True, inplace=inplace, expect_fast=True)


# ---------------------------------------------------------------- fast 1x1
FAST1 = [
    dict(N=1, Ci=64, Co=96, T=3, Tc=2, H=16, W=40),
    dict(N=1, Ci=40, Co=56, T=2, Tc=2, H=5, W=7),               # H*W not a multiple of 8
    dict(N=1, Ci=64, Co=384, T=8, Tc=1, H=16, W=40, s_t=2, p_base=1),
    dict(N=2, Ci=48, Co=200, T=2, Tc=2, H=64, W=80),             # wide pointwise tiles
]


@pytest.mark.parametrize("over", FAST1)
def test_fused_fast_1x1(over):
    _run(spec(Kh=1, Kw=1, **over), expect_fast=True)
    _run(spec(Kh=1, Kw=1, **over), inplace=True, expect_fast=True)


# ---------------------------------------------------------------- fallback
FALLBACK = [
    (dict(N=1, Ci=24, Co=40, T=2, Tc=2, H=11, W=37), c3c.MODE_FORCE_FALLBACK),
    (dict(N=1, Ci=64, Co=48, T=2, Tc=0, H=8, W=16, Kt=1, Kh=1, Kw=1), 0),  # 1x1x1: pointwise
    # 1x1x1 on the resident-weight kernel: a cached frame (no prologue), a
    # right-padded frame (bias and residual alone), a channel tail, N = 2;
    # then 320 tiles, some workgroups taking two of different batch elements
    (dict(N=2, Ci=40, Co=72, T=3, Tc=1, H=16, W=24, Kt=1, Kh=1, Kw=1, p_base=1, p_r=1), 0),
    (dict(N=2, Ci=64, Co=160, T=5, Tc=0, H=64, W=128, Kt=1, Kh=1, Kw=1), 0),
    (dict(N=1, Ci=12, Co=20, T=3, Tc=2, H=10, W=13, Kh=5, Kw=3), 0),       # 5x3: generic
    (dict(N=1, Ci=16, Co=24, T=4, Tc=2, H=12, W=16, s_t=2), 0),            # 3x3 at stride 2
]


@pytest.mark.parametrize("over,mode", FALLBACK)
def test_fused_fallback(over, mode):
    _run(spec(**over), mode=mode, expect_fast=False)
    _run(spec(**over), mode=mode, inplace=True, expect_fast=False)


@pytest.mark.parametrize("pro,res", [(True, False), (False, True)])
def test_fused_parts_on_the_resident_1x1x1_kernel(pro, res):
    """The prologue alone and the residual alone (the kernel's two fused
    instances) on a 1x1x1 call whose weights fit in LDS."""
    sp = spec(N=2, Ci=40, Co=72, T=3, Tc=1, H=16, W=24, Kt=1, Kh=1, Kw=1, p_base=1, p_r=1)
    _run(sp, pro=pro, res=res, expect_fast=False)


# ---------------------------------------------------------------- streaming
@pytest.mark.parametrize("kh", [3, 1])
def test_fused_stream_matches_oracle_stream(kh):
    """Chunks through the fused form, the cache carried: every chunk's output
    and the final cache against the oracle's own stream of fused calls."""
    base = spec(N=1, Ci=32, Co=64, T=2, Tc=0, H=16, W=40, Kh=kh, Kw=kh)
    ctx = c3c.Context()
    w, b = layer(base, "bf16", WID, 7)
    wpack = c3c.weight_repack(ctx, base, w)
    cache_d, cache_h = None, None
    for i, T in enumerate((2, 3, 1, 2)):
        sp = dict(base, T=T, Tc=0 if cache_d is None else cache_d.shape[2])
        say(f"stream chunk {i} {sp}")
        x = chunk(sp, "bf16", WID, 7, 10 + i)
        scale, shift = inputs.affine_inputs(sp, WID, 7, 0, "cuda")
        To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
        r = inputs.residual_input((1, 64, To, Ho, Wo), "bf16", WID, 7, 10 + i, "cuda")
        y, co = c3c.conv3d_causal_cached_fused(ctx, sp, x, cache_d, w, wpack, b, scale, shift, r)
        torch.cuda.synchronize()
        ref_y, ref_c = oracle.conv3d_fused(sp, host(x), cache_h, host(w), host(b), host(scale),
                                           host(shift), host(r))
        check(as_f64(y), ref_y, "bf16", f"chunk {i}")
        _check_cache(_bits(co), ref_c, sp)
        # carry the library's own cache forward; the oracle takes the same bits
        cache_d, cache_h = co, _bits(co)
    assert ctx.counters()["fast"] == 4


# ---------------------------------------------------------------- memory
def test_calls_allocate_no_device_memory():
    """The library allocates nothing in a compute call (plain, fused, split-K
    with the caller's workspace, fallback): after one warm-up call of each
    kind (which loads its kernels' code), repeated calls leave the device's
    free memory unchanged."""
    ctx = c3c.Context()
    cases = []
    for over, mode, ws in [(dict(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80), 0, False),
                           (dict(N=1, Ci=128, Co=128, T=1, Tc=2, H=16, W=32), 0, True),
                           (dict(N=1, Ci=12, Co=20, T=3, Tc=2, H=10, W=13, Kh=5, Kw=3), 0, False)]:
        sp = spec(**over)
        w, b = layer(sp, "bf16", WID, 3)
        x = chunk(sp, "bf16", WID, 3, 0)
        cache = chunk(dict(sp, T=sp["Tc"]), "bf16", WID, 3, 1)
        wpack = c3c.weight_repack(ctx, sp, w) if c3c.route_query(None, sp, "bf16")[0] == "fast" else None
        To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
        y = torch.empty((sp["N"], sp["Co"], To, Ho, Wo), dtype=torch.bfloat16, device="cuda")
        co = torch.empty((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), dtype=torch.bfloat16, device="cuda")
        scale, shift = inputs.affine_inputs(sp, WID, 3, 0, "cuda")
        r = inputs.residual_input(tuple(y.shape), "bf16", WID, 3, 0, "cuda")
        wsb = torch.empty(max(c3c.workspace_bytes(sp, "bf16"), 4) // 4, dtype=torch.float32,
                          device="cuda") if ws else None
        cases.append((sp, x, cache, w, wpack, b, y, co, scale, shift, r, wsb))

    def all_calls():
        for sp, x, cache, w, wpack, b, y, co, scale, shift, r, wsb in cases:
            ctx.set_workspace(wsb)
            c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b, y, co)
            c3c.conv3d_causal_cached_fused(ctx, sp, x, cache, w, wpack, b, scale, shift, r, y, co)
            c3c.conv3d_causal_cached_fused(ctx, sp, x, cache, w, wpack, b, None, None, r, y, co)
        ctx.set_workspace(None)

    all_calls()
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(5):
        all_calls()
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    say(f"free before {free0} after {free1}")
    assert free1 == free0


# ---------------------------------------------------------------- prologue pass
@pytest.mark.parametrize("over,split", [(dict(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80), False),
                                        (dict(N=2, Ci=40, Co=96, T=3, Tc=1, H=13, W=37), False),
                                        (dict(N=1, Ci=128, Co=128, T=1, Tc=2, H=16, W=32), True),
                                        (dict(N=1, Ci=32, Co=3, T=2, Tc=2, H=20, W=40), False)])
def test_prologue_pass_equals_in_kernel_prologue(over, split):
    """With a workspace of c3c_fused_workspace_bytes, the prologue runs as a
    pass of its own into the workspace: y and the new cache are bit-identical
    to the in-kernel prologue's (the same SiLU code on the same values), and
    match the oracle.  With split, the workspace's remainder also splits K."""
    sp = spec(**over)
    need = c3c.fused_workspace_bytes(sp, "bf16")
    assert need > 0
    assert (c3c.workspace_bytes(sp, "bf16") > 0) == split
    _, y0, c0 = _run(sp, expect_fast=True)
    ctx = c3c.Context()
    ctx.set_workspace(torch.empty(need // 4, dtype=torch.float32, device="cuda"))
    _, y1, c1 = _run(sp, ctx=ctx, expect_fast=True)
    if not split:  # split-K sums in another order: equal to the oracle, not bitwise
        assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    assert torch.equal(c0.view(torch.int16), c1.view(torch.int16))
