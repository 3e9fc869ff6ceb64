"""GPU parity of the normalised block form (c3c_conv3d_causal_cached_block)
against the oracle's composition (oracle.conv3d_block) on the same seeded
inputs: the new chunk normalised per pixel over its channels (RMS, eps inside
the root), gain and bias per channel, SiLU, one bf16 rounding; the cached
causal convolution on [cache; u]; the residual after the bias.

Bar: the activated chunk (read back from the workspace) and the new cache's
activated frames against the oracle's, element by element, at most 1e-3 of
them differing at all, and each difference within what the kernel's fp32
evaluation allows: one bf16 step of the oracle's value (a pre-activation
within a few fp32 ulp of a bf16 rounding midpoint may round the other way),
plus 1.1 x 2^-20 x (|x r gamma| + |beta|) -- the pre-activation
v = x r gamma + beta is formed in fp32 from a reciprocal square root and a
product that each carry a few ulp of relative error, so where gamma and beta
nearly cancel, v (and SiLU(v), whose slope is at most 1.1) carries an
absolute error of a few fp32 ulp of |x r gamma| + |beta| that can be many
bf16 steps of a near-zero result.  Old-cache frames bit-exact; y within
max|err| / max|ref| <= 2e-2.  Outputs start NaN-filled (every element
written); the counters are those of the plain call.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs
from paper_2609_31938_amd.inputs import spec

from gpu_util import as_f64, check, chunk, host, layer, say
from test_gpu_fused import _bits

pytestmark = pytest.mark.gpu

WID = 911
EPS = 1e-6


def _widen(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def _check_activated(got, ref, mag, what):
    """got / ref: bf16 bits of activated values; mag: |x r gamma| + |beta| of
    each element (fp64).  Returns the number of differing elements."""
    diff = got != ref
    n = int(np.count_nonzero(diff))
    assert n <= max(1, got.size // 1000), (what, n, got.size)
    if n:
        g, r, m = _widen(got[diff]), _widen(ref[diff]), mag[diff]
        # one bf16 step at the oracle's value (the spacing just above |r|)
        step = np.abs(_widen(ref[diff] + np.uint16(1)) - r)
        bound = step + 1.1 * 2.0 ** -20 * m
        assert np.all(np.abs(g - r) <= bound), (what, float(np.max(np.abs(g - r) / bound)))
    return n


def _magnitude(sp, hx, gamma, beta):
    """|x r gamma| + |beta| per element of the new chunk, from the oracle's rms."""
    _, rms = oracle.rms_prologue_bf16(sp, hx, gamma, beta, EPS, with_rms=True)
    x = _widen(hx.contiguous().view(torch.int16).numpy().view(np.uint16))
    g = gamma.numpy().astype(np.float64)[None, :, None, None, None]
    b = beta.numpy().astype(np.float64)[None, :, None, None, None]
    return np.abs(x / rms[:, None] * g) + np.abs(b)


def _run(sp, mode=0, res=True, inplace=False, seed=0, ctx=None, x=None, cache=None,
         expect_fast=None, kernel=None):
    say(f"block case {sp} mode={mode} res={res} inplace={inplace}")
    ctx = ctx or c3c.Context(mode)
    w, b = layer(sp, "bf16", WID, seed)
    x = chunk(sp, "bf16", WID, seed, 0) if x is None else x
    if cache is None and sp["Tc"]:
        cache = chunk(dict(sp, T=sp["Tc"]), "bf16", WID, seed, 1)
    route = c3c.route_query(None, sp, "bf16")[0]
    wpack = c3c.weight_repack(ctx, sp, w) if route == "fast" else None
    if kernel is not None:
        assert c3c.plan_query(ctx, sp, "bf16", c3c.block_workspace_bytes(sp))["kernel"] == kernel
    To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
    yshape = (sp["N"], sp["Co"], To, Ho, Wo)
    gamma, beta = inputs.norm_inputs(sp, WID, seed, "cuda")
    r = inputs.residual_input(yshape, "bf16", WID, seed, 0, "cuda") if res else None
    r_host = host(r) if r is not None else None
    need = c3c.block_workspace_bytes(sp)
    ws = torch.full(((need + 3) // 4,), float("nan"), dtype=torch.float32, device="cuda")
    ctx.set_workspace(ws)
    if inplace:
        y = r.clone()
        residual = y
    else:
        y = torch.full(yshape, float("nan"), dtype=torch.bfloat16, device="cuda")
        residual = r
    co = torch.full((sp["N"], sp["Ci"], L, sp["H"], sp["W"]), float("nan"), dtype=torch.bfloat16,
                    device="cuda")
    before = ctx.counters()
    y, co = c3c.conv3d_causal_cached_block(ctx, sp, x, cache, w, wpack, b, gamma, beta, EPS,
                                           residual, y, co)
    torch.cuda.synchronize()
    after = ctx.counters()
    assert after["calls"] - before["calls"] == 1 and after["failed"] == before["failed"]
    if expect_fast is not None:
        assert after["fast"] - before["fast"] == (1 if expect_fast else 0)
    hx, hc = host(x), host(cache) if cache is not None else None
    # the activated chunk, read back from the workspace
    nx = x.numel()
    u_got = ws.view(torch.int16)[:nx].cpu().numpy().view(np.uint16).reshape(tuple(x.shape))
    hg, hb = host(gamma), host(beta)
    u_ref = oracle.rms_prologue_bf16(sp, hx, hg, hb, EPS)
    mag = _magnitude(sp, hx, hg, hb)
    nu = _check_activated(u_got, u_ref, mag, "u")
    ref_y, ref_c = oracle.conv3d_block(sp, hx, hc, host(w), host(b), hg, hb, EPS, r_host)
    m = check(as_f64(y), ref_y, "bf16", str(sp))
    nc = 0
    if L:
        got_c = _bits(co)
        Z = sp["Tc"] + sp["T"]
        for j in range(L):
            f = Z - L + j
            if f < sp["Tc"]:   # a frame of the old cache: bit-exact
                assert np.array_equal(got_c[:, :, j], ref_c[:, :, j]), f"cache frame {j}"
            else:              # an activated frame of the new chunk
                nc += _check_activated(got_c[:, :, j], ref_c[:, :, j], mag[:, :, f - sp["Tc"]],
                                       f"cache frame {j}")
    say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f} u differing={nu} cache differing={nc}")
    ctx.set_workspace(None)
    return ctx, y, co


CASES = [
    (dict(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80), "conv3d_bf16"),     # 160 channels
    (dict(N=1, Ci=48, Co=80, T=3, Tc=2, H=37, W=72), "conv3d_bf16"),      # 96-channel tile
    (dict(N=2, Ci=40, Co=192, T=2, Tc=1, H=16, W=64), "conv3d_bf16"),     # 192 channels, N = 2
    (dict(N=1, Ci=32, Co=3, T=2, Tc=2, H=20, W=40), "head"),              # head kernel (no residual)
    (dict(N=1, Ci=24, Co=40, T=2, Tc=2, H=11, W=37), "conv3d_bf16"),      # H*W not a multiple of 8
    (dict(N=1, Ci=320, Co=96, T=2, Tc=3, H=9, W=16), "conv3d_bf16"),      # many channels, p_l < 0
    (dict(N=1, Ci=32, Co=64, T=3, Tc=0, H=16, W=48), "conv3d_bf16"),      # no cache
    (dict(N=1, Ci=64, Co=200, T=2, Tc=2, H=12, W=16, Kh=1, Kw=1), None),  # 1x1 temporal
    (dict(N=1, Ci=48, Co=40, T=3, Tc=0, H=10, W=24, Kt=1, Kh=1, Kw=1, p_base=0), "pointwise"),
    (dict(N=1, Ci=384, Co=384, T=1, Tc=2, H=12, W=26), "conv3d_bf16"),    # split-K in the workspace
    (dict(N=1, Ci=160, Co=160, T=2, Tc=2, H=8, W=80), "conv3d_bf16"),     # pass: 12 rows per lane
    (dict(N=1, Ci=400, Co=32, T=1, Tc=2, H=6, W=16), "conv3d_bf16"),      # pass: > 384 channels, loop
]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_block_matches_oracle(i):
    over, kernel = CASES[i]
    sp = spec(**over)
    fast = c3c.route_query(None, sp, "bf16")[0] == "fast"
    # the head kernel serves calls without a residual
    _run(sp, expect_fast=fast, kernel=kernel, res=kernel != "head")


@pytest.mark.parametrize("i,tile", [(0, (160, 4, 80)), (2, (192, 4, 64))])
def test_block_on_the_channel_tiles(i, tile):
    """The 160- and 192-channel cases above fill few compute units and run on
    64-channel 4x64 tiles; C3C_MODE_CHANNEL_TILES keeps their own tiles."""
    over, kernel = CASES[i]
    sp = spec(**over)
    need = c3c.block_workspace_bytes(sp)
    for mode, want in ((0, (64, 4, 64)), (c3c.MODE_CHANNEL_TILES, tile)):
        pl = c3c.plan_query(c3c.Context(mode), sp, "bf16", need)
        assert (pl["tile_co"], pl["tile_h"], pl["tile_w"]) == want, pl
    _run(sp, mode=c3c.MODE_CHANNEL_TILES, expect_fast=True, kernel=kernel)


def test_block_split_k_uses_the_rest_of_the_workspace():
    sp = spec(N=1, Ci=384, Co=384, T=1, Tc=2, H=12, W=26)
    assert c3c.workspace_bytes(sp, "bf16") > 0
    assert c3c.plan_query(None, sp, "bf16", c3c.workspace_bytes(sp, "bf16"))["splits"] > 1


@pytest.mark.parametrize("res,inplace", [(False, False), (True, True)])
def test_block_residual_parts(res, inplace):
    _run(spec(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80), res=res, inplace=inplace,
         expect_fast=True)


def test_block_forced_fallback():
    ctx, _, _ = _run(spec(N=1, Ci=24, Co=40, T=2, Tc=2, H=11, W=37), mode=c3c.MODE_FORCE_FALLBACK,
                     expect_fast=False)
    assert ctx.counters()["forced"] == 1


def test_block_stream_carries_activated_cache():
    """Three chunks with the cache carried: each call's outputs and new cache
    against the oracle fed the previous oracle cache (whose activated frames
    may differ by a bf16 step from the kernel's, so the kernel's own cache is
    carried and compared within that bar)."""
    base = spec(N=1, Ci=48, Co=96, T=2, Tc=0, H=18, W=40)
    ctx = c3c.Context()
    cache = None
    for c in range(3):
        sp = dict(base, Tc=0 if cache is None else cache.shape[2])
        x = chunk(sp, "bf16", WID, 5, 10 + c)
        _, _, cache = _run(sp, seed=5, ctx=ctx, x=x, cache=cache, expect_fast=True)
    assert ctx.counters()["fast"] == 3
