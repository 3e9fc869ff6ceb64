"""Pins for the oracle's fused residual-block form (CPU only).

The fused call is a composition: u = RNE_bf16(SiLU(x * s[n, c] + t[n, c])) on
the new chunk, the cached causal convolution on [C; u], plus a residual after
the bias.  Each part is pinned to something other than itself:

* the bf16 rounding: every finite bf16 value rounds to itself (exhaustive),
  exact midpoints go to the even neighbour, the overflow and subnormal edges
  sit where the format puts them, and it agrees with the integer form of
  round-to-nearest-even on fp32 inputs;
* SiLU: closed forms at +-ln 3 and +-ln 7 (sigmoid = 3/4, 7/8), its odd
  identity SiLU(v) - SiLU(-v) = v, and its limits;
* the prologue's per-(n, c) indexing, with distinct scale / shift per pair;
* the whole fused call: a brute-force seven-loop evaluation on a tiny case,
  chunked streaming equal to one whole-sequence call (the cache carries
  activated frames), residual linearity, and the plain convolution when there
  is neither prologue nor residual.
"""
import math

import numpy as np
import pytest

import oracle as O


def bf16_to_f64(bits):
    with np.errstate(invalid="ignore"):  # NaN patterns widen to NaN
        return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- rounding
def test_round_bf16_is_identity_on_every_finite_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    v = bf16_to_f64(bits)
    finite = np.isfinite(v)
    back = O.round_bf16(v[finite])
    assert np.array_equal(back, bits[finite])


def test_round_bf16_midpoints_go_to_even():
    rng = np.random.default_rng(5)
    # positive finite patterns below the largest finite value, both signs
    b = rng.integers(0x0000, 0x7f7f, size=2000).astype(np.uint16)
    for sign in (0, 0x8000):
        lo = (b | sign).astype(np.uint16)
        hi = ((b + 1) | sign).astype(np.uint16)
        mid = (bf16_to_f64(lo) + bf16_to_f64(hi)) / 2  # exact in fp64
        got = O.round_bf16(mid)
        want = np.where((lo & 1) == 0, lo, hi)
        assert np.array_equal(got, want)
        # just off the midpoint: the nearer neighbour
        eps = np.abs(bf16_to_f64(hi) - bf16_to_f64(lo)) * 2.0**-20
        toward_lo = O.round_bf16(mid - np.sign(mid) * eps)
        toward_hi = O.round_bf16(mid + np.sign(mid) * eps)
        assert np.array_equal(toward_lo, lo)
        assert np.array_equal(toward_hi, hi)


def test_round_bf16_edges():
    max_bf16 = float(bf16_to_f64(np.array([0x7f7f]))[0])
    assert max_bf16 == (2 - 2.0**-7) * 2.0**127
    half_q = 2.0**(127 - 8)
    assert O.round_bf16([max_bf16 + half_q * 0.99])[0] == 0x7f7f
    assert O.round_bf16([max_bf16 + half_q])[0] == 0x7f80  # tie, odd -> up -> inf
    assert O.round_bf16([-max_bf16 - half_q])[0] == 0xff80
    assert O.round_bf16([2.0**-133])[0] == 0x0001          # smallest subnormal
    assert O.round_bf16([2.0**-134])[0] == 0x0000          # tie with 0 -> even
    assert O.round_bf16([3 * 2.0**-134])[0] == 0x0002      # tie between 1 and 2
    assert O.round_bf16([-0.0])[0] == 0x8000
    assert O.round_bf16([math.inf])[0] == 0x7f80
    assert O.round_bf16([math.nan])[0] & 0x7fff > 0x7f80


def test_round_bf16_matches_integer_rne_on_fp32_values():
    rng = np.random.default_rng(6)
    f = (rng.standard_normal(20000) * np.exp(rng.uniform(-60, 60, 20000))).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    want = ((u + 0x7fff + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    assert np.array_equal(O.round_bf16(f.astype(np.float64)), want)


# ---------------------------------------------------------------- SiLU
def test_silu_closed_forms_and_identities():
    l3, l7 = math.log(3), math.log(7)
    got = O.silu([0.0, l3, -l3, l7, -l7])
    want = [0.0, 0.75 * l3, -0.25 * l3, 0.875 * l7, -0.125 * l7]
    assert np.allclose(got, want, rtol=1e-15, atol=0)
    rng = np.random.default_rng(7)
    v = rng.uniform(-12, 12, 500)
    assert np.allclose(O.silu(v) - O.silu(-v), v, rtol=1e-13, atol=1e-13)
    assert O.silu([50.0])[0] == pytest.approx(50.0, rel=1e-15)
    assert O.silu([-50.0])[0] == pytest.approx(-50.0 * math.exp(-50.0), rel=1e-12)


# ---------------------------------------------------------------- prologue
def _spec(**kw):
    s = dict(N=1, Ci=3, Co=2, T=2, Tc=2, H=4, W=5, Kt=3, Kh=3, Kw=3,
             s_t=1, s_h=1, s_w=1, d_t=1, d_h=1, d_w=1, p_base=2, p_r=0, p_h=1, p_w=1,
             groups=1, has_bias=1)
    s.update(kw)
    return s


def _bf16(rng, shape, scale=1.0):
    return O.round_bf16(rng.standard_normal(shape) * scale)


def test_prologue_uses_scale_and_shift_of_its_own_batch_and_channel():
    rng = np.random.default_rng(8)
    sp = _spec(N=2, Ci=3, T=2, H=2, W=3)
    x = _bf16(rng, (2, 3, 2, 2, 3))
    sc = (1.0 + np.arange(6, dtype=np.float32).reshape(2, 3) / 4).astype(np.float32)
    sh = (np.arange(6, dtype=np.float32).reshape(2, 3) / 8 - 0.3).astype(np.float32)
    u = O.prologue_bf16(sp, x, sc, sh)
    xv = bf16_to_f64(x)
    want = np.empty_like(u)
    for n in range(2):
        for c in range(3):
            v = xv[n, c] * float(sc[n, c]) + float(sh[n, c])
            want[n, c] = O.round_bf16(O.silu(v.ravel())).reshape(v.shape)
    assert np.array_equal(u, want)
    zero = O.prologue_bf16(sp, np.zeros_like(x), np.ones((2, 3), np.float32),
                           np.zeros((2, 3), np.float32))
    assert not zero.any()


# ---------------------------------------------------------------- fused call
def _operands(rng, sp):
    N, Ci, Co = sp["N"], sp["Ci"], sp["Co"]
    x = _bf16(rng, (N, Ci, sp["T"], sp["H"], sp["W"]))
    cache = _bf16(rng, (N, Ci, sp["Tc"], sp["H"], sp["W"])) if sp["Tc"] else None
    w = _bf16(rng, (Co, Ci, sp["Kt"], sp["Kh"], sp["Kw"]), 0.3)
    b = _bf16(rng, (Co,), 0.5)
    sc = rng.uniform(0.5, 1.5, (N, Ci)).astype(np.float32)
    sh = rng.uniform(-0.5, 0.5, (N, Ci)).astype(np.float32)
    return x, cache, w, b, sc, sh


def test_fused_matches_brute_force():
    rng = np.random.default_rng(9)
    sp = _spec(N=2, Ci=3, Co=2, T=3, Tc=2, H=4, W=5)
    x, cache, w, b, sc, sh = _operands(rng, sp)
    To, Ho, Wo, L = O.output_dims(sp)
    r = _bf16(rng, (2, 2, To, Ho, Wo))
    y, c_new = O.conv3d_fused(sp, x, cache, w, b, sc, sh, r)
    # seven loops over the definition: z = [cache; SiLU(x s + t) rounded]
    xv, cv, wv, bv, rv = (bf16_to_f64(a) for a in (x, cache, w, b, r))
    Z = sp["Tc"] + sp["T"]
    z = np.zeros((2, 3, Z, 4, 5))
    z[:, :, :sp["Tc"]] = cv
    for n in range(2):
        for c in range(3):
            for f in range(sp["T"]):
                for h in range(4):
                    for q in range(5):
                        v = xv[n, c, f, h, q] * float(sc[n, c]) + float(sh[n, c])
                        z[n, c, sp["Tc"] + f, h, q] = bf16_to_f64(
                            [O.round_bf16([v / (1 + math.exp(-v))])[0]])[0]
    p_l = sp["p_base"] - sp["Tc"]
    want = np.zeros((2, 2, To, Ho, Wo))
    for n in range(2):
        for co in range(2):
            for t in range(To):
                for h in range(Ho):
                    for q in range(Wo):
                        acc = 0.0
                        for c in range(3):
                            for k in range(3):
                                f = t + k - p_l
                                if not 0 <= f < Z:
                                    continue
                                for i in range(3):
                                    for j in range(3):
                                        hh, qq = h + i - 1, q + j - 1
                                        if 0 <= hh < 4 and 0 <= qq < 5:
                                            acc += wv[co, c, k, i, j] * z[n, c, f, hh, qq]
                        want[n, co, t, h, q] = acc + bv[co] + rv[n, co, t, h, q]
    assert np.allclose(y, want, rtol=1e-12, atol=1e-12)
    assert np.array_equal(bf16_to_f64(c_new), z[:, :, Z - L:])


def test_fused_streaming_equals_whole_sequence():
    rng = np.random.default_rng(10)
    whole = _spec(N=1, Ci=4, Co=3, T=7, Tc=0, H=3, W=6, p_base=2)
    x, _, w, b, sc, sh = _operands(rng, whole)
    y_all, c_all = O.conv3d_fused(whole, x, None, w, b, sc, sh)
    ys, cache, t0 = [], None, 0
    for T in (1, 3, 2, 1):
        sp = dict(whole, T=T, Tc=0 if cache is None else cache.shape[2])
        y, cache = O.conv3d_fused(sp, x[:, :, t0:t0 + T], cache, w, b, sc, sh)
        ys.append(y)
        t0 += T
    assert np.array_equal(np.concatenate(ys, axis=2), y_all)
    assert np.array_equal(cache, c_all)


def test_fused_residual_is_added_once_and_plain_call_is_the_conv():
    rng = np.random.default_rng(11)
    sp = _spec(N=1, Ci=5, Co=4, T=2, Tc=2, H=5, W=4)
    x, cache, w, b, sc, sh = _operands(rng, sp)
    To, Ho, Wo, _ = O.output_dims(sp)
    r = _bf16(rng, (1, 4, To, Ho, Wo))
    y0, c0 = O.conv3d_fused(sp, x, cache, w, b, sc, sh)
    y1, c1 = O.conv3d_fused(sp, x, cache, w, b, sc, sh, r)
    assert np.allclose(y1 - y0, bf16_to_f64(r), rtol=0, atol=1e-12)
    assert np.array_equal(c0, c1)
    yp, cp = O.conv3d_fused(sp, x, cache, w, b)
    assert np.array_equal(yp, O.conv3d(sp, "bf16", x, cache, w, b))
    assert np.array_equal(cp, O.cache_update(sp, "bf16", x, cache))
    with pytest.raises(ValueError):
        O.conv3d_fused(sp, x, cache, w, b, sc, None)
