"""The allocation-free entry point (c3c_conv3d_causal_cached_noalloc),
called through the C ABI: its split-K partial sums live in the library's
device scratch, not in a caller workspace.

Two calls in a row that both split (the second smaller, so it reuses the
scratch the first left behind) must give exactly what the existing entry
point gives with a caller workspace of the same size (the same split, the
same summation order: bit-identical), and so match the oracle within the
bf16 bar, with the new cache bit-exact and guard bands around the outputs
untouched.  Device free memory must not change across the calls, and a call
whose split would need more than the scratch holds is refused (EINVAL, not
counted)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c
from paper_2609_31938_amd.inputs import spec

from gpu_util import as_f64, check, chunk, guarded, guards_intact, host, layer, say

pytestmark = pytest.mark.gpu

# both split their stages (4 ways at 60x104: 38 MB of partial sums; the
# second is smaller)
CALLS = [spec(N=1, Ci=384, Co=384, T=1, Tc=2, H=60, W=104),
         spec(N=1, Ci=256, Co=160, T=1, Tc=2, H=24, W=72)]


def _inputs(sp, seed):
    w, b = layer(sp, "bf16", 950, seed)
    x = chunk(sp, "bf16", 950, seed, 0)
    cache = chunk(dict(sp, T=sp["Tc"]), "bf16", 950, seed, 1)
    return w, b, x, cache


def test_noalloc_equals_the_workspace_call_twice():
    prepared = []
    for i, sp in enumerate(CALLS):
        need = c3c.workspace_bytes(sp, "bf16")
        assert 0 < need <= c3c.NOALLOC_SCRATCH_BYTES, (sp, need)
        w, b, x, cache = _inputs(sp, i)
        ctx_ws = c3c.Context()
        wpack = c3c.weight_repack(ctx_ws, sp, w)
        ws = torch.empty(need // 4, dtype=torch.float32, device="cuda")
        ctx_ws.set_workspace(ws)
        assert c3c.plan_query(ctx_ws, sp, "bf16", need)["splits"] > 1
        y_ref, c_ref = c3c.conv3d_causal_cached(ctx_ws, sp, x, cache, w, wpack, b)
        To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
        y, ybuf = guarded((1, sp["Co"], To, Ho, Wo), "bf16")
        co, cbuf = guarded((1, sp["Ci"], L, sp["H"], sp["W"]), "bf16")
        prepared.append((sp, w, b, x, cache, wpack, y_ref, c_ref, y, ybuf, co, cbuf))
    torch.cuda.synchronize()
    ctx = c3c.Context()
    # The scratch array's memory is committed when the library first looks it
    # up on this device (one time, at most the array plus its code object);
    # after that no call changes the device's free memory.
    sp, w, b, x, cache, wpack, y_ref, c_ref, _, _, _, _ = prepared[0]
    free_a, _ = torch.cuda.mem_get_info()
    c3c.conv3d_causal_cached_noalloc(c3c.Context(), sp, x, cache, w, wpack, b,
                                     torch.empty_like(y_ref), torch.empty_like(c_ref))
    torch.cuda.synchronize()
    free_b, _ = torch.cuda.mem_get_info()
    say(f"first use on the device: {free_a - free_b} bytes")
    assert free_a - free_b <= c3c.NOALLOC_SCRATCH_BYTES + (16 << 20) + 2 * y_ref.numel() * 2 * 2
    free0, _ = torch.cuda.mem_get_info()
    for sp, w, b, x, cache, wpack, y_ref, c_ref, y, ybuf, co, cbuf in prepared:
        say(f"noalloc call {sp['Ci']}->{sp['Co']} {sp['H']}x{sp['W']}")
        c3c.conv3d_causal_cached_noalloc(ctx, sp, x, cache, w, wpack, b, y, co)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    say(f"free before {free0} after {free1}")
    assert free1 == free0
    c = ctx.counters()
    assert (c["calls"], c["fast"], c["fallback"], c["failed"]) == (2, 2, 0, 0)
    for sp, w, b, x, cache, wpack, y_ref, c_ref, y, ybuf, co, cbuf in prepared:
        assert guards_intact(ybuf) and guards_intact(cbuf)
        assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
        assert torch.equal(co.view(torch.int16), c_ref.view(torch.int16))
        hx, hc = host(x), host(cache)
        ref = oracle.conv3d(sp, "bf16", hx, hc, host(w), host(b))
        m = check(as_f64(y), ref, "bf16", str(sp))
        ref_c = oracle.cache_update(sp, "bf16", hx, hc)
        assert np.array_equal(host(co).view(torch.int16).numpy().view(np.uint16), ref_c)
        say(f"  rel={m['rel']:.3e} cos={m['cos']:.8f}")


def test_noalloc_call_that_does_not_split():
    """A call that runs unsplit uses no scratch; it equals the plain call."""
    sp = spec(N=1, Ci=64, Co=160, T=3, Tc=2, H=40, W=160)
    assert c3c.workspace_bytes(sp, "bf16") == 0
    w, b, x, cache = _inputs(sp, 7)
    ctx = c3c.Context()
    wpack = c3c.weight_repack(ctx, sp, w)
    y_ref, c_ref = c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b)
    y, co = torch.empty_like(y_ref), torch.empty_like(c_ref)
    c3c.conv3d_causal_cached_noalloc(ctx, sp, x, cache, w, wpack, b, y, co)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
    assert torch.equal(co.view(torch.int16), c_ref.view(torch.int16))


def test_noalloc_refuses_a_split_larger_than_the_scratch():
    sp = spec(N=1, Ci=384, Co=192, T=1, Tc=2, H=184, W=160)
    assert c3c.workspace_bytes(sp, "bf16") > c3c.NOALLOC_SCRATCH_BYTES
    w, b, x, cache = _inputs(sp, 8)
    ctx = c3c.Context()
    wpack = c3c.weight_repack(ctx, sp, w)
    To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
    y = torch.empty((1, 192, To, Ho, Wo), dtype=torch.bfloat16, device="cuda")
    co = torch.empty((1, 384, L, 184, 160), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(c3c.C3CError) as e:
        c3c.conv3d_causal_cached_noalloc(ctx, sp, x, cache, w, wpack, b, y, co)
    assert e.value.status == c3c.E_INVAL and "scratch" in str(e.value)
    assert ctx.counters()["calls"] == 0
