"""The pins must be strong enough to catch a plausible slip in the oracle.

Each mutant below is a copy of the oracle's C source with one deliberate
mistake (a dropped tap, a flipped sign in the source-frame index of Eq. 1,
cache and chunk frames swapped, the bias added per tap, a transposed weight
index, the wrong effective left pad of Eq. 3, the wrong cache rule, a wrong
spatial pad sign, an off-by-one in Eq. 4, a missing route clause; in the
fused form's parts, bf16 ties rounded away from zero, one significand bit
short, the sign of SiLU's exponent, the shift of the wrong channel; in the
normalised prologue, the sum of squares instead of their mean, eps outside
the root, no root, one channel left out, the gain of the wrong channel).  The copy
is compiled to a temporary library and the pin suite is run against it in a
child process; every mutant must make the suite fail.  Nothing here touches
the HIP library or the GPU.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "conv3d_oracle.c")

MUTANTS = {
    "drop_last_tap": [("for (int64_t k = 0; k < d->Kt; ++k) {\n      int64_t tz = t * d->s_t + k * d->d_t - p_l; /* Eq. 1 */",
                       "for (int64_t k = 0; k < d->Kt - 1; ++k) {\n      int64_t tz = t * d->s_t + k * d->d_t - p_l; /* Eq. 1 */")],
    "eq1_sign": [("int64_t tz = t * d->s_t + k * d->d_t - p_l; /* Eq. 1 */",
                  "int64_t tz = t * d->s_t + k * d->d_t + p_l; /* Eq. 1 */")],
    "chunk_before_cache": [("  if (f < d->Tc) {\n    *off = ((n * d->Ci + c) * d->Tc + f) * hw;\n    return cache;\n  }\n  *off = ((n * d->Ci + c) * d->T + (f - d->Tc)) * hw;\n  return x;",
                            "  if (f < d->T) {\n    *off = ((n * d->Ci + c) * d->T + f) * hw;\n    return x;\n  }\n  *off = ((n * d->Ci + c) * d->Tc + (f - d->T)) * hw;\n  return cache;")],
    "bias_per_tap": [("      if (tz < 0 || tz >= Z) continue;\n      for (int64_t i = 0; i < d->Kh; ++i) {\n        int64_t hz = h * d->s_h + i * d->d_h - d->p_h;\n        if (hz < 0 || hz >= d->H) continue;\n        int64_t off;",
                      "      if (tz < 0 || tz >= Z) continue;\n      if (d->has_bias && c == 0) for (int64_t q = 0; q < Wo; ++q) acc[q] += bd[co];\n      for (int64_t i = 0; i < d->Kh; ++i) {\n        int64_t hz = h * d->s_h + i * d->d_h - d->p_h;\n        if (hz < 0 || hz >= d->H) continue;\n        int64_t off;"),
                     ("  if (d->has_bias)\n    for (int64_t w = 0; w < Wo; ++w) acc[w] += bd[co];\n}", "}")],
    "weight_ij_transposed": [("double wv = wd[(((co * cig + c) * d->Kt + k) * d->Kh + i) * d->Kw + j];",
                              "double wv = wd[(((co * cig + c) * d->Kt + k) * d->Kh + j % d->Kh) * d->Kw + i % d->Kw];")],
    "left_pad_sign": [("int64_t p_l = d->p_base - d->Tc;", "int64_t p_l = d->p_base + d->Tc;")],
    "cache_keeps_first_frames": [("z_frame(d, x, cache, n, c, Z - L + j, &off);",
                                  "z_frame(d, x, cache, n, c, j, &off);")],
    "spatial_pad_sign": [("        int64_t hz = h * d->s_h + i * d->d_h - d->p_h;\n        if (hz < 0 || hz >= d->H) continue;\n        int64_t off;",
                          "        int64_t hz = h * d->s_h + i * d->d_h + d->p_h;\n        if (hz < 0 || hz >= d->H) continue;\n        int64_t off;")],
    "eq4_off_by_one": [("int64_t hi = Z - delta < To ? Z - delta : To;",
                        "int64_t hi = Z - delta - 1 < To ? Z - delta - 1 : To;")],
    "route_kt_clause_missing": [("else if (d->Kt < 2 && !k3x3)", "else if (d->Kt < 1 && !k3x3)")],
    # the fused form's parts
    "bf16_ties_away_from_zero": [("double r = nearbyint(a / q) * q;", "double r = round(a / q) * q;")],
    "bf16_one_bit_short": [("q = ldexp(1.0, ex - 1 - 7);", "q = ldexp(1.0, ex - 1 - 6);")],
    "silu_sign": [("return v / (1.0 + exp(-v));", "return v / (1.0 + exp(v));")],
    "prologue_shift_of_next_channel": [("double sc = (double)s[nc], sh = (double)t[nc];",
                                        "double sc = (double)s[nc], sh = (double)t[(nc + 1) % (N * Ci)];")],
    # the normalised prologue
    "rms_sum_not_mean": [("double r = sqrt(ss / (double)Ci + eps);", "double r = sqrt(ss + eps);")],
    "rms_eps_outside_root": [("double r = sqrt(ss / (double)Ci + eps);",
                              "double r = sqrt(ss / (double)Ci) + eps;")],
    "rms_without_root": [("double r = sqrt(ss / (double)Ci + eps);", "double r = ss / (double)Ci + eps;")],
    "rms_over_one_channel_short": [("    for (int64_t c = 0; c < Ci; ++c) {\n      double v = widen(x, ORA_BF16, (n * Ci + c) * T * hw + tp);",
                                    "    for (int64_t c = 0; c + 1 < Ci; ++c) {\n      double v = widen(x, ORA_BF16, (n * Ci + c) * T * hw + tp);")],
    "rms_gain_of_next_channel": [("/ r * (double)g[c] + (double)b[c]", "/ r * (double)g[(c + 1) % Ci] + (double)b[c]")],
}
PIN_FILES = ["test_oracle_pins.py", "test_oracle_fused_pins.py"]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    src = open(SRC).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) >= 1, f"mutation site for {name} not found"
        src = src.replace(old, new)
    csrc = tmp_path / "mutant.c"
    csrc.write_text(src)
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-std=c11", "-O1", "-fPIC", "-shared", "-fopenmp",
                           "-ffp-contract=off", str(csrc), "-o", str(lib), "-lm"])
    env = dict(os.environ, C3C_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *[os.path.join(ROOT, "tests", f) for f in PIN_FILES]],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
