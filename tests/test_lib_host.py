"""Host-side checks of libc3c that need no GPU: the library loads and exports
every symbol its header declares; its host maths (Eq. 3 output sizes, Eq. 4
intervals, the FLOP count) and its route rule agree with the oracle's
independent implementation; argument errors, strict-mode rejections and the
counters behave as documented.

The calls below that pass fake device addresses are all rejected before any
device access (argument validation or strict mode); they are skipped where a
GPU is present so that a validation bug could never turn into a launch on a
bogus pointer.
"""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from paper_2609_31938_amd import c3c
from paper_2609_31938_amd.inputs import spec

from test_oracle_pins import ROUTE_TABLE, _random_spec

no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                            reason="fake-pointer argument tests run on CPU-only hosts")


def test_every_declared_symbol_is_exported():
    names = c3c.declared_symbols()
    assert names == sorted([
        "c3c_ctx_create", "c3c_ctx_destroy", "c3c_set_mode", "c3c_get_mode",
        "c3c_output_dims", "c3c_tap_interval", "c3c_flops", "c3c_route_query",
        "c3c_weight_pack_bytes", "c3c_weight_repack", "c3c_weight_unpack",
        "c3c_conv3d_causal_cached", "c3c_counters_get", "c3c_counters_reset",
        "c3c_fallback_shapes", "c3c_strerror", "c3c_last_error",
        "c3c_workspace_bytes", "c3c_ctx_set_workspace", "c3c_conv3d_causal_cached_fused",
        "c3c_mfma_probe", "c3c_fused_workspace_bytes", "c3c_plan_query",
        "c3c_conv3d_causal_cached_noalloc", "c3c_block_workspace_bytes",
        "c3c_conv3d_causal_cached_block"])
    for n in names:
        assert hasattr(c3c.lib, n), n


def test_descriptor_layout_matches_header():
    # 21 int64 fields + 2 int32 = 176 bytes, no padding surprises
    assert C.sizeof(c3c.Desc) == 21 * 8 + 2 * 4
    assert C.sizeof(c3c.Counters) == 9 * 8
    assert C.sizeof(c3c.Plan) == 4 * 4 + 4 * 8 + 2 * 4


@pytest.mark.parametrize("case", range(300))
def test_host_maths_match_oracle(case):
    rng = np.random.default_rng(90000 + case)
    sp = _random_spec(rng)
    assert c3c.output_dims(sp) == oracle.output_dims(sp)
    assert c3c.flops(sp) == oracle.flops(sp)
    for dt in ("bf16", "f32", "f16"):
        assert c3c.route_query(None, sp, dt) == oracle.route(sp, dt)
    if sp["s_t"] == 1:
        for k in range(sp["Kt"]):
            assert c3c.tap_interval(sp, k) == oracle.tap_interval(sp, k)


@pytest.mark.parametrize("over,dtype,forced,reason", ROUTE_TABLE)
def test_route_table(over, dtype, forced, reason):
    sp = spec(N=1, Ci=2, Co=2, T=2, Tc=2, H=4, W=4)
    sp.update(over)
    ctx = c3c.Context(c3c.MODE_FORCE_FALLBACK if forced else 0)
    r, why = c3c.route_query(ctx, sp, dtype)
    assert why == reason
    assert r == ("fast" if reason == "none" else "fallback")
    assert ctx.counters()["calls"] == 0  # a query counts nothing


def test_workload_routes():
    from paper_2609_31938_amd.inputs import WORKLOADS
    for name, wl in WORKLOADS.items():
        for lname, sp in wl["layers"]:
            r, why = c3c.route_query(None, sp, wl["dtype"])
            if sp["Kt"] == 1:
                assert (r, why) == ("fallback", "kt1")
            else:
                assert (r, why) == ("fast", "none"), (name, lname)


def test_pack_bytes_closed_form():
    for Ci, Co in [(384, 384), (192, 192), (96, 96), (320, 160), (640, 640), (48, 80), (3, 5)]:
        sp = spec(Ci=Ci, Co=Co, T=4, Tc=2, H=8, W=8)
        # bf16: 16-row x 32-channel fragments; fp32: 32-row x 2-channel fragments
        chunks, frags = -(-Ci // 32), -(-Co // 16)
        assert c3c.weight_pack_bytes(sp, "bf16") == 27 * chunks * frags * 64 * 8 * 2
        chunks2, frags2 = -(-Ci // 2), -(-Co // 32)
        assert c3c.weight_pack_bytes(sp, "f32") == 27 * chunks2 * frags2 * 64 * 4
    # no fast layout for a call that does not route fast
    assert c3c.weight_pack_bytes(spec(Ci=4, Co=4, Kt=1, Kh=1, Kw=1, T=2), "bf16") == 0


def test_invalid_descriptors_are_rejected():
    bad = [dict(N=0), dict(Ci=0), dict(H=0), dict(T=-1), dict(Tc=-1), dict(Kt=0),
           dict(s_h=0), dict(d_t=0), dict(p_base=-1), dict(p_h=-1), dict(groups=3),
           dict(H=1, p_h=0)]  # Ho < 1
    for over in bad:
        sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=4, W=4)
        sp.update(over)
        with pytest.raises(c3c.C3CError) as e:
            c3c.output_dims(sp)
        assert e.value.status == c3c.E_INVAL
    d = c3c.make_desc(spec(Ci=4, Co=4, T=2, H=4, W=4), "bf16")
    d.dtype = 9
    assert c3c.lib.c3c_output_dims(C.byref(d), None, None, None, None) == c3c.E_INVAL
    d.dtype = 1
    d.has_bias = 2
    assert c3c.lib.c3c_output_dims(C.byref(d), None, None, None, None) == c3c.E_INVAL


def test_context_modes():
    ctx = c3c.Context()
    assert ctx.mode == 0
    ctx.mode = c3c.MODE_STRICT | c3c.MODE_FORCE_FALLBACK
    assert ctx.mode == 3
    ctx.mode = c3c.MODE_CHANNEL_TILES | c3c.MODE_STRICT
    assert ctx.mode == 9
    with pytest.raises(c3c.C3CError):
        ctx.mode = 16
    assert ctx.mode == 9
    h = C.c_void_p()
    assert c3c.lib.c3c_ctx_create(16, C.byref(h)) == c3c.E_INVAL
    assert c3c.lib.c3c_ctx_create(0, None) == c3c.E_INVAL
    assert c3c.lib.c3c_ctx_destroy(None) == c3c.OK
    assert c3c.lib.c3c_strerror(2).decode().startswith("unsupported")


# ---------------------------------------------------------------------------
# calls rejected before any device access (fake, never-dereferenced addresses)
# ---------------------------------------------------------------------------

FAKE = {"x": 0x10000000, "cache": 0x20000000, "w": 0x30000000, "wpack": 0x40000000,
        "b": 0x50000000, "y": 0x60000000, "co": 0x70000000}


def _call(ctx, sp, dtype="bf16", **over):
    p = dict(FAKE)
    p.update(over)
    return c3c.lib.c3c_conv3d_causal_cached(ctx._h if ctx else None,
                                            C.byref(c3c.make_desc(sp, dtype)), p["x"],
                                            p["cache"], p["w"], p["wpack"], p["b"], p["y"],
                                            p["co"], None)


@no_gpu
def test_argument_errors_are_not_counted():
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    ctx = c3c.Context()
    assert _call(None, sp) == c3c.E_INVAL
    assert _call(ctx, sp, x=None) == c3c.E_INVAL
    assert _call(ctx, sp, cache=None) == c3c.E_INVAL
    assert _call(ctx, sp, w=None) == c3c.E_INVAL
    assert _call(ctx, sp, b=None) == c3c.E_INVAL
    assert _call(ctx, sp, y=None) == c3c.E_INVAL
    assert _call(ctx, sp, co=None) == c3c.E_INVAL
    assert _call(ctx, sp, wpack=None) == c3c.E_INVAL        # routes fast without wpack
    assert "wpack" in ctx.last_error
    # cache_out aliasing the cache (in-place cache update is refused)
    assert _call(ctx, sp, co=FAKE["cache"]) == c3c.E_INVAL
    assert _call(ctx, sp, co=FAKE["x"] + 64) == c3c.E_INVAL
    assert _call(ctx, sp, y=FAKE["x"]) == c3c.E_INVAL
    assert _call(ctx, sp, y=FAKE["wpack"] + 2) == c3c.E_INVAL
    bad = dict(sp, Ci=0)
    assert _call(ctx, bad) == c3c.E_INVAL
    assert ctx.counters() == dict(calls=0, fast=0, fallback=0, unsupported=0, forced=0,
                                  fast_error=0, strict_rejects=0, repacks=0, failed=0)


@no_gpu
def test_strict_mode_rejects_without_device_work():
    ctx = c3c.Context(c3c.MODE_STRICT)
    shortcut = spec(N=1, Ci=4, Co=4, T=2, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1)
    assert _call(ctx, shortcut, cache=None, co=None, wpack=None) == c3c.E_UNSUPPORTED
    ctx.mode = c3c.MODE_STRICT | c3c.MODE_FORCE_FALLBACK
    assert _call(ctx, spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)) == c3c.E_UNSUPPORTED
    ctx.mode = c3c.MODE_STRICT | c3c.MODE_INJECT_FAST_FAILURE
    assert _call(ctx, spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)) == c3c.E_INJECTED
    assert "injected" in ctx.last_error
    c = ctx.counters()
    assert c["calls"] == 3 and c["strict_rejects"] == 3
    assert c["fast"] == c["fallback"] == 0
    assert ctx.fallback_shapes() == []
    ctx.reset()
    assert ctx.counters()["calls"] == 0


# ---------------------------------------------------------------------------
# split-K workspace (host side)
# ---------------------------------------------------------------------------

@no_gpu
def test_workspace_bytes_of_the_workloads():
    """With 256 compute units (what the library assumes without a device),
    only the 60x104 single-frame layer splits (60 workgroups of 36 stages,
    into 4 splits of fp32 partial sums the size of the output).  The 44x80
    640-channel layer (176 workgroups) would spend more on moving its large
    partial sums than it gains, and stays unsplit."""
    from paper_2609_31938_amd.inputs import WORKLOADS
    got = {}
    for name, wl in WORKLOADS.items():
        for lname, sp in wl["layers"]:
            got[lname] = c3c.workspace_bytes(sp, wl["dtype"])
    assert got["c384_60x104"] == 4 * 384 * 1 * 60 * 104 * 4
    for lname, v in got.items():
        if lname != "c384_60x104":
            assert v == 0, lname


def test_workspace_bytes_only_for_fast_bf16():
    sp = spec(N=1, Ci=384, Co=384, T=1, Tc=2, H=60, W=104)
    assert c3c.workspace_bytes(sp, "f32") == 0
    assert c3c.workspace_bytes(sp, "f16") == 0
    assert c3c.workspace_bytes(dict(sp, groups=2), "bf16") == 0
    n = C.c_size_t()
    assert c3c.lib.c3c_workspace_bytes(None, C.byref(n)) == c3c.E_INVAL
    assert c3c.lib.c3c_workspace_bytes(C.byref(c3c.make_desc(sp, "bf16")), None) == c3c.E_INVAL


def test_set_workspace_arguments():
    ctx = c3c.Context()
    f = c3c.lib.c3c_ctx_set_workspace
    assert f(None, 0x10000000, 1024) == c3c.E_INVAL
    assert f(ctx._h, None, 1024) == c3c.E_INVAL
    assert f(ctx._h, 0x10000000, 0) == c3c.E_INVAL
    assert f(ctx._h, 0x10000008, 1024) == c3c.E_INVAL      # not 16-byte aligned
    assert f(ctx._h, 0x10000000, 1024) == c3c.OK
    assert f(ctx._h, None, 0) == c3c.OK                     # detach


@no_gpu
def test_workspace_overlapping_a_tensor_is_rejected():
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    ctx = c3c.Context()
    for name in ("x", "cache", "w", "wpack", "b", "y", "co"):
        assert c3c.lib.c3c_ctx_set_workspace(ctx._h, FAKE[name] - 16, 4096) == c3c.OK
        assert _call(ctx, sp) == c3c.E_INVAL, name
        assert "workspace" in ctx.last_error
    assert ctx.counters()["calls"] == 0


# ---------------------------------------------------------------------------
# the fused entry point: argument checks (fake addresses, no device work)
# ---------------------------------------------------------------------------

FAKE_FUSE = {"scale": 0x80000000, "shift": 0x90000000, "res": 0xa0000000}


def _fcall(ctx, sp, dtype="bf16", **over):
    p = dict(FAKE, **FAKE_FUSE)
    p.update(over)
    return c3c.lib.c3c_conv3d_causal_cached_fused(
        ctx._h if ctx else None, C.byref(c3c.make_desc(sp, dtype)), p["x"], p["cache"], p["w"],
        p["wpack"], p["b"], p["scale"], p["shift"], p["res"], p["y"], p["co"], None)


@no_gpu
def test_fused_call_argument_checks():
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    # strict + forced fallback: every valid call is rejected before device work
    ctx = c3c.Context(c3c.MODE_STRICT | c3c.MODE_FORCE_FALLBACK)
    assert _fcall(None, sp) == c3c.E_INVAL
    assert _fcall(ctx, sp, shift=None) == c3c.E_INVAL
    assert "together" in ctx.last_error
    assert _fcall(ctx, sp, scale=None) == c3c.E_INVAL
    assert _fcall(ctx, sp, dtype="f32") == c3c.E_INVAL
    assert "bf16" in ctx.last_error
    assert _fcall(ctx, sp, dtype="f32", scale=None, shift=None) == c3c.E_INVAL  # residual alone
    assert _fcall(ctx, sp, scale=FAKE["y"]) == c3c.E_INVAL
    assert _fcall(ctx, sp, shift=FAKE["co"] + 4) == c3c.E_INVAL
    assert _fcall(ctx, sp, res=FAKE["y"] + 2) == c3c.E_INVAL   # partial overlap with y
    assert _fcall(ctx, sp, res=FAKE["co"]) == c3c.E_INVAL
    assert _fcall(ctx, sp, y=FAKE["x"]) == c3c.E_INVAL          # the plain call's checks hold
    assert ctx.counters()["calls"] == 0
    # valid: full form, in place (residual == y), prologue only, residual only, plain
    assert _fcall(ctx, sp) == c3c.E_UNSUPPORTED
    assert _fcall(ctx, sp, res=FAKE["y"]) == c3c.E_UNSUPPORTED
    assert _fcall(ctx, sp, res=None) == c3c.E_UNSUPPORTED
    assert _fcall(ctx, sp, scale=None, shift=None) == c3c.E_UNSUPPORTED
    assert _fcall(ctx, sp, scale=None, shift=None, res=None) == c3c.E_UNSUPPORTED
    c = ctx.counters()
    assert c["calls"] == 5 and c["strict_rejects"] == 5


def test_mfma_probe_argument_checks():
    fl = C.c_double()
    f = c3c.lib.c3c_mfma_probe
    assert f(0, 10, 0x10000000, C.byref(fl), None) == c3c.E_INVAL
    assert f(4, 0, 0x10000000, C.byref(fl), None) == c3c.E_INVAL
    assert f(4, 10, None, C.byref(fl), None) == c3c.E_INVAL
    assert f(4, 10, 0x10000000, None, None) == c3c.E_INVAL
    assert f(1 << 31, 10, 0x10000000, C.byref(fl), None) == c3c.E_INVAL


def test_fused_workspace_bytes():
    sp = spec(N=1, Ci=64, Co=160, T=2, Tc=2, H=24, W=80)
    xb = 64 * 2 * 24 * 80 * 2
    assert c3c.fused_workspace_bytes(sp, "bf16") == (xb + 255) // 256 * 256 + c3c.workspace_bytes(sp, "bf16")
    small = spec(N=1, Ci=128, Co=128, T=1, Tc=2, H=16, W=32)  # a call that splits
    assert c3c.workspace_bytes(small, "bf16") > 0
    assert c3c.fused_workspace_bytes(small, "bf16") == \
        (128 * 16 * 32 * 2 + 255) // 256 * 256 + c3c.workspace_bytes(small, "bf16")
    assert c3c.fused_workspace_bytes(sp, "f32") == 0
    assert c3c.fused_workspace_bytes(spec(N=1, Ci=8, Co=8, T=2, Tc=2, H=8, W=8, Kh=1, Kw=1), "bf16") == 0
    assert c3c.fused_workspace_bytes(spec(N=1, Ci=8, Co=8, T=2, Tc=2, H=8, W=8, s_t=2), "bf16") == 0
    n = C.c_size_t()
    assert c3c.lib.c3c_fused_workspace_bytes(C.byref(c3c.make_desc(sp, "bf16")), None) == c3c.E_INVAL


# ---------------------------------------------------------------------------
# a call whose kernels cannot be launched (no device here): counted as
# failed, never as a completed fallback
# ---------------------------------------------------------------------------

@no_gpu
def test_failed_launch_is_not_counted_as_a_fallback():
    ctx = c3c.Context()
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    # a fallback call (f16 has no fast kernel), then a fast call whose fast
    # launch and then fallback launch both fail
    assert _call(ctx, sp, dtype="f16") == c3c.E_DEVICE
    assert _call(ctx, sp) == c3c.E_DEVICE
    ctx.mode = c3c.MODE_FORCE_FALLBACK
    assert _call(ctx, sp) == c3c.E_DEVICE
    c = ctx.counters()
    assert (c["calls"], c["failed"]) == (3, 3)
    assert c["fast"] == c["fallback"] == c["unsupported"] == c["forced"] == c["fast_error"] == 0
    assert c["calls"] == c["fast"] + c["fallback"] + c["strict_rejects"] + c["failed"]
    assert ctx.fallback_shapes() == []
    # strict mode: the failed fast launch is a strict reject, not a failure
    ctx.mode = c3c.MODE_STRICT
    assert _call(ctx, sp) == c3c.E_DEVICE
    c = ctx.counters()
    assert (c["calls"], c["strict_rejects"], c["failed"]) == (4, 1, 3)


# ---------------------------------------------------------------------------
# the launch plan (c3c_plan_query)
# ---------------------------------------------------------------------------

@no_gpu
def test_plan_of_the_workloads():
    """The kernel and tile each benchmarked layer takes (256 compute units,
    what the library assumes without a device)."""
    from paper_2609_31938_amd.inputs import WORKLOADS
    want = {
        "c32_32x32": ("fast_f32", 32, 4, 32, 1),
        # one output frame, 60 tiles of 192 x 4 x 64: unsplit (no workspace),
        # the 64 x 4 x 64 tiling (180 workgroups, less modelled time)
        "c384_60x104": ("conv3d_bf16", 64, 4, 64, 1),
        "c192_240x416": ("conv3d_bf16", 192, 4, 64, 1),
        "c384to192_240x416": ("conv3d_bf16", 192, 4, 64, 1),
        "c96_480x832": ("conv3d_bf16", 96, 6, 64, 1),
        "c640_44x80": ("conv3d_bf16", 128, 4, 80, 1),
        "c320_176x320": ("conv3d_bf16", 160, 4, 80, 1),
        "c320to160_352x640": ("conv3d_bf16", 160, 4, 80, 1),
        "c160_704x1280": ("conv3d_bf16", 160, 4, 80, 1),
        "shortcut_1x1x1_320to160_352x640": ("pointwise", 160, 0, 256, 1),
        "head_96to3_480x832": ("head", 3, 6, 48, 1),
        "tconv_up_384to768_60x104": ("tap1x1", 192, 0, 128, 1),
        "tconv_up_384to768_120x208": ("tap1x1", 192, 0, 128, 1),
        "tconv_down_s2_384_120x208": ("tap1x1", 192, 0, 128, 1),
    }
    for name, wl in WORKLOADS.items():
        for lname, sp in wl["layers"]:
            pl = c3c.plan_query(None, sp, wl["dtype"])
            got = (pl["kernel"], pl["tile_co"], pl["tile_h"], pl["tile_w"], pl["splits"])
            assert got == want[lname], (lname, pl)
            assert pl["route"] == ("fallback" if sp["Kt"] == 1 else "fast")
            if pl["kernel"] == "conv3d_bf16":
                assert pl["cache_in_kernel"]
                tiles = (-(-sp["Co"] // pl["tile_co"]) * -(-sp["H"] // pl["tile_h"]) *
                         -(-sp["W"] // pl["tile_w"]))
                To, _, _, _ = c3c.output_dims(sp, wl["dtype"])
                assert pl["workgroups"] == tiles * To * sp["N"]


@no_gpu
def test_plan_splits_with_a_workspace():
    sp = spec(N=1, Ci=384, Co=384, T=1, Tc=2, H=60, W=104)
    need = c3c.workspace_bytes(sp, "bf16")
    assert c3c.plan_query(None, sp, "bf16")["splits"] == 1
    assert c3c.plan_query(None, sp, "bf16", need - 16)["splits"] == 1
    pl = c3c.plan_query(None, sp, "bf16", need)
    assert pl["splits"] == 4 and pl["workgroups"] == 4 * 2 * 15 * 2
    forced = c3c.plan_query(c3c.Context(c3c.MODE_FORCE_FALLBACK), sp, "bf16")
    assert (forced["route"], forced["reason"], forced["kernel"]) == \
        ("fallback", "forced", "fallback_direct")
    empty = c3c.plan_query(None, dict(sp, T=0), "bf16")
    assert (empty["kernel"], empty["workgroups"]) == ("none", 0)


# ---------------------------------------------------------------------------
# the binding's size checks (host tensors of the wrong size are refused
# before their device placement is even looked at)
# ---------------------------------------------------------------------------

def test_binding_refuses_wrongly_sized_tensors():
    sp = spec(N=1, Ci=4, Co=8, T=2, Tc=2, H=8, W=8)
    To, Ho, Wo, L = c3c.output_dims(sp, "bf16")
    bf = torch.bfloat16
    ok = dict(x=torch.zeros(1, 4, 2, 8, 8, dtype=bf), cache=torch.zeros(1, 4, 2, 8, 8, dtype=bf),
              w=torch.zeros(8, 4, 3, 3, 3, dtype=bf),
              wpack=torch.zeros(c3c.weight_pack_bytes(sp, "bf16") // 2, dtype=bf),
              bias=torch.zeros(8, dtype=bf), y=torch.zeros(1, 8, To, Ho, Wo, dtype=bf),
              cache_out=torch.zeros(1, 4, L, 8, 8, dtype=bf))
    ctx = c3c.Context()
    for name in ok:
        args = dict(ok)
        args[name] = torch.zeros(ok[name].numel() - 1, dtype=bf)
        with pytest.raises(ValueError, match=f"{name} has"):
            c3c.conv3d_causal_cached(ctx, sp, args["x"], args["cache"], args["w"], args["wpack"],
                                     args["bias"], args["y"], args["cache_out"])
        with pytest.raises(ValueError, match=f"{name} has"):
            c3c.conv3d_causal_cached_fused(ctx, sp, args["x"], args["cache"], args["w"],
                                           args["wpack"], args["bias"], y=args["y"],
                                           cache_out=args["cache_out"])
    # right sizes: refused only for living in host memory
    with pytest.raises(ValueError, match="device tensor"):
        c3c.conv3d_causal_cached(ctx, sp, *ok.values())
    # a pack for a call with no fast layout
    sc = spec(N=1, Ci=4, Co=8, T=2, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1)
    with pytest.raises(ValueError, match="no fast-route weight layout"):
        c3c.conv3d_causal_cached(ctx, sc, torch.zeros(1, 4, 2, 8, 8, dtype=bf), None,
                                 torch.zeros(8, 4, 1, 1, 1, dtype=bf), ok["wpack"], ok["bias"])
    with pytest.raises(ValueError, match="residual has"):
        c3c.conv3d_causal_cached_fused(ctx, sp, ok["x"], ok["cache"], ok["w"], ok["wpack"],
                                       ok["bias"], residual=torch.zeros(5, dtype=bf), y=ok["y"],
                                       cache_out=ok["cache_out"])
    assert ctx.counters()["calls"] == 0


@no_gpu
def test_plan_of_the_160_channel_parity_cases():
    """The GPU parity cases drawn for the 160-channel tiles land on them:
    4x80 (ragged rows, columns and channel tiles) and, where it takes fewer
    rounds of workgroups, 10x32; and on the 128-channel 4x80 tile where that
    pads no more channels and takes less time in whole rounds (181 channels:
    two ragged tiles of 128 against two of 160)."""
    want = [(dict(N=1, Ci=64, Co=160, T=3, Tc=2, H=22, W=170), (160, 4, 80)),
            (dict(N=1, Ci=72, Co=130, T=2, Tc=2, H=13, W=96), (160, 4, 80)),
            (dict(N=2, Ci=40, Co=181, T=2, Tc=1, H=9, W=83), (128, 4, 80)),
            (dict(N=1, Ci=40, Co=256, T=2, Tc=2, H=9, W=90), (128, 4, 80)),
            (dict(N=1, Ci=48, Co=320, T=2, Tc=2, H=10, W=88), (160, 4, 80)),
            (dict(N=1, Ci=40, Co=150, T=4, Tc=2, H=333, W=30), (160, 10, 32))]
    ctx = c3c.Context(c3c.MODE_CHANNEL_TILES)
    for over, tile in want:
        pl = c3c.plan_query(ctx, spec(**over), "bf16")
        assert pl["kernel"] == "conv3d_bf16"
        assert (pl["tile_co"], pl["tile_h"], pl["tile_w"]) == tile, (over, pl)


@no_gpu
def test_unsplit_calls_that_fill_few_compute_units_take_smaller_tiles():
    """An unsplit bf16 3x3 call whose tiles fill less than one round of the
    compute units takes, of its own tiling, the 128 x 4x80 tiling (from the
    192-channel one) and the 64 x 4x64 tiling, the one of least rounds x tile
    work x c (c = 1.7 for the 64-channel tile, 1 for the others).  A call
    that splits, and C3C_MODE_CHANNEL_TILES, keep the output-channel tiling;
    a call that fills the device is never re-tiled."""
    def tile(sp, ctx=None, ws=0):
        pl = c3c.plan_query(ctx, sp, "bf16", ws)
        return pl["tile_co"], pl["tile_h"], pl["tile_w"], pl["workgroups"], pl["splits"]
    c2 = spec(N=1, Ci=384, Co=384, T=1, Tc=2, H=60, W=104)
    assert tile(c2) == (64, 4, 64, 6 * 2 * 15, 1)
    assert tile(c2, c3c.Context(c3c.MODE_CHANNEL_TILES)) == (192, 4, 64, 60, 1)
    assert tile(c2, ws=c3c.workspace_bytes(c2, "bf16")) == (192, 4, 64, 4 * 60, 4)
    # two output frames: 180 workgroups of 128 x 4x80 (cost 1 x 40960) against
    # two rounds of 360 of 64 x 4x64 (2 x 16384 x 1.7 = 55706)
    assert tile(dict(c2, T=2)) == (128, 4, 80, 3 * 2 * 15 * 2, 1)
    # 192 -> 192: 30 workgroups of 192 x 4x64 (128 x 4x80 pads to 256 channels)
    assert tile(spec(N=1, Ci=192, Co=192, T=1, Tc=2, H=60, W=104)) == (64, 4, 64, 90, 1)
    # a full round of 192-channel tiles stays
    big = spec(N=1, Ci=192, Co=192, T=4, Tc=2, H=240, W=416)
    assert tile(big)[:3] == (192, 4, 64)
    # 96 channels or fewer keep their own tiles
    assert tile(spec(N=1, Ci=96, Co=96, T=1, Tc=2, H=20, W=64))[:3] == (96, 6, 64)


@no_gpu
def test_head_kernel_takes_calls_whose_weight_table_fits():
    """The head kernel gathers its B operands into an LDS table of
    Kt x chunks x column-fragment entries (1 KiB each) beside its stage
    buffers: up to 26 entries beside four, 59 beside three.  A call whose
    table fits neither goes to the 3x3 kernel's 16-channel tile."""
    def kern(**over):
        return c3c.plan_query(None, spec(**over), "bf16")["kernel"]
    assert kern(N=1, Ci=96, Co=3, T=4, Tc=2, H=24, W=64) == "head"     # 3 x 3 x 2 = 18
    assert kern(N=1, Ci=96, Co=5, T=3, Tc=2, H=24, W=64) == "head"     # 3 x 3 x 3 = 27
    assert kern(N=1, Ci=192, Co=5, T=3, Tc=2, H=24, W=64) == "head"    # 3 x 6 x 3 = 54
    assert kern(N=1, Ci=224, Co=5, T=3, Tc=2, H=24, W=64) == "conv3d_bf16"  # 63
    assert kern(N=1, Ci=288, Co=3, T=3, Tc=2, H=24, W=64) == "head"    # 3 x 9 x 2 = 54
    assert kern(N=1, Ci=320, Co=3, T=3, Tc=2, H=24, W=64) == "conv3d_bf16"  # 60
    assert kern(N=1, Ci=608, Co=1, T=3, Tc=2, H=24, W=64) == "head"    # 3 x 19 x 1 = 57
    assert kern(N=1, Ci=640, Co=1, T=3, Tc=2, H=24, W=64) == "conv3d_bf16"  # 60


@no_gpu
def test_noalloc_refuses_an_oversized_split_before_device_work():
    ctx = c3c.Context()
    big = spec(N=1, Ci=384, Co=192, T=1, Tc=2, H=184, W=160)
    assert c3c.workspace_bytes(big, "bf16") > c3c.NOALLOC_SCRATCH_BYTES
    d = c3c.make_desc(big, "bf16")
    f = c3c.lib.c3c_conv3d_causal_cached_noalloc
    p = FAKE
    assert f(ctx._h, C.byref(d), p["x"], p["cache"], p["w"], p["wpack"], p["b"], p["y"], p["co"],
             None) == c3c.E_INVAL
    assert "scratch" in ctx.last_error and str(64 << 20) in ctx.last_error
    assert f(None, C.byref(d), p["x"], p["cache"], p["w"], p["wpack"], p["b"], p["y"], p["co"],
             None) == c3c.E_INVAL
    assert ctx.counters()["calls"] == 0
    # forced onto the fallback, the same call needs no scratch: it is counted
    # (and fails here only for want of a device)
    ctx.mode = c3c.MODE_FORCE_FALLBACK
    assert f(ctx._h, C.byref(d), p["x"], p["cache"], p["w"], p["wpack"], p["b"], p["y"], p["co"],
             None) == c3c.E_DEVICE
    assert ctx.counters()["failed"] == 1


# ---------------------------------------------------------------- normalised block form
def _block(ctx, sp, dtype="bf16", gamma=0x11000000, beta=0x12000000, eps=1e-6, res=None, **over):
    p = dict(FAKE)
    p.update(over)
    return c3c.lib.c3c_conv3d_causal_cached_block(
        ctx._h if ctx else None, C.byref(c3c.make_desc(sp, dtype)), p["x"], p["cache"], p["w"],
        p["wpack"], p["b"], gamma, beta, eps, res, p["y"], p["co"], None)


def test_block_workspace_bytes_closed_form():
    for Ci, Co, T, H, W in [(384, 192, 4, 240, 416), (3, 5, 1, 7, 9), (384, 384, 1, 60, 104)]:
        sp = spec(N=1, Ci=Ci, Co=Co, T=T, Tc=2, H=H, W=W)
        xb = Ci * T * H * W * 2
        want = -(-xb // 256) * 256 + c3c.workspace_bytes(sp, "bf16")
        assert c3c.block_workspace_bytes(sp) == want
    # the 1x1x1 shortcut (fallback route): the activated chunk only
    sc = spec(N=1, Ci=32, Co=16, T=4, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1)
    assert c3c.block_workspace_bytes(sc) == 32 * 4 * 64 * 2
    with pytest.raises(c3c.C3CError):
        c3c.block_workspace_bytes(sc, "f32")


@no_gpu
def test_block_call_argument_errors_are_not_counted():
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    ctx = c3c.Context()
    # no workspace
    assert _block(ctx, sp) == c3c.E_INVAL and "workspace" in ctx.last_error
    need = c3c.block_workspace_bytes(sp)
    assert c3c.lib.c3c_ctx_set_workspace(ctx._h, 0x80000000, need - 16) == c3c.OK
    assert _block(ctx, sp) == c3c.E_INVAL                       # one slot short
    assert c3c.lib.c3c_ctx_set_workspace(ctx._h, 0x80000000, need) == c3c.OK
    assert _block(ctx, sp, gamma=None) == c3c.E_INVAL
    assert _block(ctx, sp, beta=None) == c3c.E_INVAL
    assert _block(ctx, sp, eps=-1.0) == c3c.E_INVAL
    assert _block(ctx, sp, eps=float("nan")) == c3c.E_INVAL
    assert _block(ctx, sp, eps=float("inf")) == c3c.E_INVAL
    assert _block(ctx, sp, "f32") == c3c.E_INVAL
    assert _block(ctx, sp, x=0x80000000 + 64) == c3c.E_INVAL    # x inside the workspace
    assert _block(ctx, sp, gamma=FAKE["y"]) == c3c.E_INVAL      # gamma overlapping y
    assert _block(ctx, sp, res=0x80000000) == c3c.E_INVAL       # residual in the workspace
    assert _block(ctx, sp, y=FAKE["x"]) == c3c.E_INVAL
    assert _block(None, sp) == c3c.E_INVAL
    assert ctx.counters()["calls"] == 0


@no_gpu
def test_block_call_strict_rejection_runs_no_pass():
    """A strict call that does not route fast is rejected before the
    normalisation pass: no device work (a launch would fail on this host and
    count the call as failed instead)."""
    sc = spec(N=1, Ci=4, Co=4, T=2, Tc=0, H=8, W=8, Kt=1, Kh=1, Kw=1)
    ctx = c3c.Context(c3c.MODE_STRICT)
    assert c3c.lib.c3c_ctx_set_workspace(ctx._h, 0x80000000, c3c.block_workspace_bytes(sc)) == c3c.OK
    assert _block(ctx, sc, cache=None, co=None, wpack=None) == c3c.E_UNSUPPORTED
    ctx.mode = c3c.MODE_STRICT | c3c.MODE_INJECT_FAST_FAILURE
    sp = spec(N=1, Ci=4, Co=4, T=2, Tc=2, H=8, W=8)
    assert c3c.lib.c3c_ctx_set_workspace(ctx._h, 0x80000000, c3c.block_workspace_bytes(sp)) == c3c.OK
    assert _block(ctx, sp) == c3c.E_INJECTED
    c = ctx.counters()
    assert (c["calls"], c["strict_rejects"], c["failed"], c["fast"], c["fallback"]) == (2, 2, 0, 0, 0)
