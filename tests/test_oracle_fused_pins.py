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


# ---------------------------------------------------------------- normalised prologue
# u = RNE_bf16(SiLU(x / rms * gamma[c] + beta[c])), rms = sqrt(mean_c x^2 + eps)
# per pixel (n, t, p).  Pinned by reduction to the affine prologue (pinned
# above), exact invariances, locality, and closed forms built from the
# rounding and SiLU pinned above.

def _bf16_bits(v):
    return O.round_bf16(np.asarray(v, np.float64))


def _unit_rms_chunk(rng, N, Ci, T, H, W):
    """bf16 chunks whose every pixel has mean square exactly 1 over the
    channels: signed, permuted copies of a fixed vector."""
    base = {1: [1.0], 2: [1.0, 1.0], 3: [1.0, 1.0, 1.0], 5: [2.0, 1.0, 0.0, 0.0, 0.0],
            8: [2.0, 1.0, 1.0, 1.0, 1.0, 0.0, 0.0, 0.0]}[Ci]
    x = np.empty((N, Ci, T, H, W))
    for n in range(N):
        for t in range(T):
            for h in range(H):
                for w in range(W):
                    v = rng.permutation(base) * rng.choice([-1.0, 1.0], Ci)
                    x[n, :, t, h, w] = v
    assert np.allclose((x ** 2).mean(axis=1), 1.0)
    return _bf16_bits(x)


@pytest.mark.parametrize("Ci", [1, 2, 3, 5, 8])
def test_rms_prologue_reduces_to_the_affine_prologue_at_unit_rms(Ci):
    rng = np.random.default_rng(700 + Ci)
    sp = dict(N=2, Ci=Ci, T=2, H=3, W=4)
    x = _unit_rms_chunk(rng, 2, Ci, 2, 3, 4)
    g = rng.normal(1.0, 0.5, Ci).astype(np.float32)
    b = rng.normal(0.0, 0.5, Ci).astype(np.float32)
    u, rms = O.rms_prologue_bf16(sp, x, g, b, 0.0, with_rms=True)
    assert np.array_equal(rms, np.ones_like(rms))
    # the same per-channel gain and bias for every batch element
    want = O.prologue_bf16(sp, x, np.tile(g, (2, 1)), np.tile(b, (2, 1)))
    assert np.array_equal(u, want)


def test_rms_prologue_is_invariant_to_a_power_of_two_scale_of_each_pixel():
    rng = np.random.default_rng(711)
    sp = dict(N=2, Ci=7, T=3, H=4, W=5)
    x = _bf16_bits(rng.normal(0, 1, (2, 7, 3, 4, 5)))
    k = rng.integers(-3, 4, (2, 1, 3, 4, 5)).astype(np.float64)
    xs = _bf16_bits(bf16_to_f64(x) * 2.0 ** k)  # exact: a power of two per pixel
    g = rng.normal(1.0, 0.3, 7).astype(np.float32)
    b = rng.normal(0.0, 0.3, 7).astype(np.float32)
    u0, r0 = O.rms_prologue_bf16(sp, x, g, b, 0.0, with_rms=True)
    u1, r1 = O.rms_prologue_bf16(sp, xs, g, b, 0.0, with_rms=True)
    assert np.array_equal(u0, u1)
    assert np.allclose(r1, r0 * 2.0 ** k[:, 0], rtol=1e-15)


def test_rms_prologue_is_local_to_each_pixel():
    rng = np.random.default_rng(712)
    sp = dict(N=2, Ci=6, T=3, H=4, W=5)
    x = _bf16_bits(rng.normal(0, 1, (2, 6, 3, 4, 5)))
    g = rng.normal(1.0, 0.3, 6).astype(np.float32)
    b = rng.normal(0.0, 0.3, 6).astype(np.float32)
    u0 = O.rms_prologue_bf16(sp, x, g, b, 1e-6)
    x2 = x.copy()
    x2[1, :, 2, 3, 1] = _bf16_bits(rng.normal(0, 3, 6))
    u1 = O.rms_prologue_bf16(sp, x2, g, b, 1e-6)
    diff = np.any(u0 != u1, axis=1)  # (N, T, H, W): pixels whose u changed
    assert diff[1, 2, 3, 1] and diff.sum() == 1


def test_rms_prologue_closed_forms():
    sp = dict(N=1, Ci=2, T=1, H=1, W=1)
    g = np.array([1.0, 1.0], np.float32)
    b = np.zeros(2, np.float32)
    # (3, 4): rms = sqrt(12.5)
    x = _bf16_bits(np.array([3.0, 4.0]).reshape(1, 2, 1, 1, 1))
    u, rms = O.rms_prologue_bf16(sp, x, g, b, 0.0, with_rms=True)
    assert rms.item() == math.sqrt(12.5)
    assert np.array_equal(u.ravel(), _bf16_bits([O.silu(np.array([3.0 / math.sqrt(12.5)]))[0],
                                                 O.silu(np.array([4.0 / math.sqrt(12.5)]))[0]]))
    # eps inside the root: x = (1, 1), eps = 3 -> rms = 2, x / rms = 1/2
    x = _bf16_bits(np.ones((1, 2, 1, 1, 1)))
    g2 = np.array([2.0, -6.0], np.float32)
    b2 = np.array([0.25, 0.5], np.float32)
    u, rms = O.rms_prologue_bf16(sp, x, g2, b2, 3.0, with_rms=True)
    assert rms.item() == 2.0
    assert np.array_equal(u.ravel(), _bf16_bits(O.silu(np.array([0.5 * 2.0 + 0.25,
                                                                 0.5 * -6.0 + 0.5]))))
    # a zero pixel: u = SiLU(beta) for any eps > 0
    x = np.zeros((1, 2, 1, 1, 1), np.uint16)
    u = O.rms_prologue_bf16(sp, x, g2, b2, 1e-5)
    assert np.array_equal(u.ravel(), _bf16_bits(O.silu(b2.astype(np.float64))))


def test_block_call_equals_the_affine_fused_call_at_unit_rms():
    """With every pixel at unit RMS and eps = 0 the normalised block call is
    the affine fused call with scale = gamma, shift = beta (output, cache')."""
    rng = np.random.default_rng(720)
    sp = dict(N=1, Ci=5, Co=6, T=3, Tc=2, H=5, W=6, Kt=3, Kh=3, Kw=3, s_t=1, s_h=1, s_w=1,
              d_t=1, d_h=1, d_w=1, p_base=2, p_r=0, p_h=1, p_w=1, groups=1, has_bias=1)
    x = _unit_rms_chunk(rng, 1, 5, 3, 5, 6)
    cache = _bf16_bits(rng.normal(0, 1, (1, 5, 2, 5, 6)))
    w = _bf16_bits(rng.normal(0, 0.2, (6, 5, 3, 3, 3)))
    bias = _bf16_bits(rng.normal(0, 0.3, 6))
    res = _bf16_bits(rng.normal(0, 1, (1, 6, 3, 5, 6)))
    g = rng.normal(1.0, 0.3, 5).astype(np.float32)
    b = rng.normal(0.0, 0.3, 5).astype(np.float32)
    y1, c1 = O.conv3d_block(sp, x, cache, w, bias, g, b, 0.0, res)
    y2, c2 = O.conv3d_fused(sp, x, cache, w, bias, g[None, :], b[None, :], res)
    assert np.array_equal(y1, y2) and np.array_equal(c1, c2)


def test_block_call_streams_like_one_whole_sequence():
    """The normalisation is local to each frame, so chunked streaming with
    the carried (activated) cache equals one call over the whole sequence."""
    rng = np.random.default_rng(721)
    base = dict(N=1, Ci=4, Co=3, Tc=0, H=4, W=5, Kt=3, Kh=3, Kw=3, s_t=1, s_h=1, s_w=1,
                d_t=1, d_h=1, d_w=1, p_base=2, p_r=0, p_h=1, p_w=1, groups=1, has_bias=1)
    xs = _bf16_bits(rng.normal(0, 1, (1, 4, 6, 4, 5)))
    w = _bf16_bits(rng.normal(0, 0.2, (3, 4, 3, 3, 3)))
    bias = _bf16_bits(rng.normal(0, 0.3, 3))
    g = rng.normal(1.0, 0.3, 4).astype(np.float32)
    b = rng.normal(0.0, 0.3, 4).astype(np.float32)
    whole, _ = O.conv3d_block(dict(base, T=6), xs, None, w, bias, g, b, 1e-6)
    cache, outs = None, []
    for t0, t1 in ((0, 2), (2, 3), (3, 6)):
        sp = dict(base, T=t1 - t0, Tc=0 if cache is None else cache.shape[2])
        y, cache = O.conv3d_block(sp, np.ascontiguousarray(xs[:, :, t0:t1]), cache, w, bias,
                                  g, b, 1e-6)
        outs.append(y)
    assert np.array_equal(np.concatenate(outs, axis=2), whole)
