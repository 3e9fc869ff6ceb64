"""Seeded random call shapes for the fuzz parity test, grouped by the kernel
each group is drawn to reach.  No convolution arithmetic here: a case is a
(dtype, spec overrides, kernel the plan must name, context mode, split-K workspace?)
record, and the CPU test suite checks that every case's plan names the kernel
its group targets, so the GPU fuzz run covers every kernel by construction.
"""
import numpy as np

from paper_2609_31938_amd.inputs import spec

# C3C_MODE_CHANNEL_TILES: an unsplit call that fills few compute units keeps
# its output-channel tiling instead of the 64-channel 4x64 tiles (half of the
# wider cases run with it, so both tilings are drawn)
CHANNEL_TILES = 8


def _i(rng, lo, hi):
    return int(rng.integers(lo, hi + 1))


def _temporal(rng, Kt_choices=(2, 3, 3)):
    """Kt, d_t, p_base, Tc and T: causal padding with a cache of 0 .. p_base + 1
    frames (more than p_base exercises a negative effective left pad)."""
    Kt = int(rng.choice(Kt_choices))
    d_t = int(rng.choice([1, 1, 1, 2]))
    p_base = d_t * (Kt - 1)
    return dict(Kt=Kt, d_t=d_t, p_base=p_base, Tc=_i(rng, 0, p_base + 1), T=_i(rng, 1, 4))


def _conv3x3(rng, co_lo, co_hi, hw=(1, 40, 1, 150)):
    return dict(N=_i(rng, 1, 2), Ci=_i(rng, 1, 96), Co=_i(rng, co_lo, co_hi),
                H=_i(rng, hw[0], hw[1]), W=_i(rng, hw[2], hw[3]), **_temporal(rng))


def cases():
    rng = np.random.default_rng(20261202)
    out = []
    # bf16 3x3 on the implicit-GEMM kernel: every tile width (<= 16, <= 96,
    # 160-wide for 97..400 output channels except multiples of 192, 192-wide)
    for _ in range(20):
        out.append(("bf16", _conv3x3(rng, 6, 96), "conv3d_bf16", 0, False))
    for _ in range(10):
        o = _conv3x3(rng, 6, 16)
        o["W"] = _i(rng, 1, 60) * 2 + 1  # odd widths: never the head kernel
        out.append(("bf16", o, "conv3d_bf16", 0, False))
    for k in range(30):
        o = _conv3x3(rng, 97, 400, hw=(1, 30, 1, 120))
        if o["Co"] % 192 == 0:
            o["Co"] += 1
        out.append(("bf16", o, "conv3d_bf16", CHANNEL_TILES if k % 2 else 0, False))
    for k in range(10):
        o = _conv3x3(rng, 192, 192, hw=(1, 24, 1, 100))
        o["Co"] = int(rng.choice([192, 384]))
        out.append(("bf16", o, "conv3d_bf16", CHANNEL_TILES if k % 2 else 0, False))
    # fp32 3x3 and 1x1
    for _ in range(15):
        out.append(("f32", _conv3x3(rng, 1, 80, hw=(1, 24, 1, 70)), "fast_f32", 0, False))
    for _ in range(5):
        o = _conv3x3(rng, 1, 80, hw=(1, 16, 1, 40))
        o.update(Kh=1, Kw=1, s_t=_i(rng, 1, 3))
        out.append(("f32", o, "fast_f32", 0, False))
    # the head kernel: Co <= 5, W a multiple of 8
    for _ in range(20):
        o = _conv3x3(rng, 1, 5, hw=(1, 40, 1, 30))
        o["W"] *= 8
        out.append(("bf16", o, "head", 0, False))
    # 1x1 temporal convolutions on the pointwise kernel (small or unaligned),
    # temporal stride 1 .. 3
    for _ in range(20):
        o = _conv3x3(rng, 1, 300, hw=(1, 20, 1, 40))
        o.update(Kh=1, Kw=1, s_t=_i(rng, 1, 3), Ci=_i(rng, 1, 200))
        out.append(("bf16", o, "pointwise", 0, False))
    # ... and on the 192 x 128 kernel (aligned, enough workgroups, Co whose
    # 192-wide padding is close to the 160-wide one)
    n = 0
    while n < 20:
        o = dict(N=_i(rng, 1, 2), Ci=_i(rng, 8, 160), Co=int(rng.choice([180, 192, 350, 384, 576, 768])),
                 H=_i(rng, 8, 48), W=8 * _i(rng, 8, 20), Kh=1, Kw=1, **_temporal(rng))
        o["s_t"] = _i(rng, 1, 3)
        o["T"] = _i(rng, 4, 12)
        # the kernel needs half a workgroup per compute unit (256 of them)
        Z, p_l = o["Tc"] + o["T"], o["p_base"] - o["Tc"]
        To = (Z + p_l - o["d_t"] * (o["Kt"] - 1) - 1) // o["s_t"] + 1
        if -(-o["H"] * o["W"] // 128) * -(-o["Co"] // 192) * To * o["N"] * 2 < 256:
            continue
        out.append(("bf16", o, "tap1x1", 0, False))
        n += 1
    # split-K with a workspace: few output tiles, many channels
    for _ in range(20):
        o = dict(N=1, Ci=_i(rng, 128, 512), Co=int(rng.choice([96, 160, 192, 256, 384])),
                 H=_i(rng, 4, 24), W=_i(rng, 8, 64), Kt=3, d_t=1, p_base=2, Tc=2, T=_i(rng, 1, 2))
        out.append(("bf16", o, "conv3d_bf16", 0, True))
    # a single temporal tap (1,3,3): a per-frame spatial convolution
    for _ in range(10):
        o = _conv3x3(rng, 1, 200, hw=(1, 20, 1, 90))
        o.update(Kt=1, p_base=0, Tc=0, d_t=1)
        out.append(("bf16" if _ % 3 else "f32", o, None, 0, False))
    # the fallback: calls forced off the fast route, and unsupported shapes
    # (strides, dilations, groups, other kernel sizes, f16)
    for _ in range(15):
        o = _conv3x3(rng, 1, 120, hw=(1, 16, 1, 60))
        out.append((str(rng.choice(["bf16", "f32"])), o, "fallback_direct", 2, False))
    for _ in range(15):
        Kh, Kw = _i(rng, 1, 5), _i(rng, 1, 5)
        # spatial stride 2 keeps every case off both fast forms
        o = dict(N=_i(rng, 1, 2), Ci=4 * _i(rng, 1, 8), Co=4 * _i(rng, 1, 10),
                 H=_i(rng, 9, 20), W=_i(rng, 5, 40), Kh=Kh, Kw=Kw,
                 s_h=2, s_w=_i(rng, 1, 2), d_h=_i(rng, 1, 2), d_w=1,
                 p_h=_i(rng, 0, 2), p_w=_i(rng, 0, 2), groups=int(rng.choice([1, 2, 4])),
                 **_temporal(rng, (1, 2, 3)))
        o["s_t"] = _i(rng, 1, 2)
        out.append((str(rng.choice(["bf16", "f32", "f16"])), o, "fallback_direct", 0, False))
    res = []
    for dtype, over, kernel, mode, ws in out:
        sp = spec(**over)
        res.append((dtype, sp, kernel, mode, ws))
    return res
