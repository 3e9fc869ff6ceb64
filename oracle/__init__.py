"""CPU oracle for the cached causal Conv3D -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports it and shares no code with it.

The arithmetic lives in ``conv3d_oracle.c`` (plain C, fp64, OpenMP); this
module only marshals numpy arrays into it.  The definition it follows is the
plain zero-padded causal Conv3D over the cache-augmented input Z = [C; X]_T of
the paper's Sec. 4 (Eq. 1-4), with the bias added exactly once and the cache
replaced by the last min(p_base, |Z|) frames of Z.

The fused residual-block form is the composition of plain parts: the new
chunk goes through ``u = RNE_bf16(SiLU(x * scale[n, c] + shift[n, c]))`` (fp64,
one rounding), the convolution runs on ``[C; u]`` (so the new cache holds
activated frames), and a residual of the output's shape is added in fp64 after
the bias (``conv3d_fused``).

A call is described by a plain ``spec`` dict with the keys
``N Ci Co T Tc H W Kt Kh Kw s_t s_h s_w d_t d_h d_w p_base p_r p_h p_w groups
has_bias``.  Element types are named ``"f64" "f32" "bf16" "f16"``; bf16 data is
carried in ``numpy.uint16`` arrays holding the raw bits.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# C3C_ORACLE_LIB loads another build of the oracle: the mutation test's
# deliberately broken copies (in child processes) and the sanitizer build of
# the host-side test run; nothing else sets it.
_LIB_PATH = os.environ.get("C3C_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

_FIELDS = ["N", "Ci", "Co", "T", "Tc", "H", "W", "Kt", "Kh", "Kw",
           "s_t", "s_h", "s_w", "d_t", "d_h", "d_w",
           "p_base", "p_r", "p_h", "p_w", "groups", "has_bias"]

_DTYPES = {"f64": 0, "f32": 1, "bf16": 2, "f16": 3}
_NP = {"f64": np.float64, "f32": np.float32, "bf16": np.uint16, "f16": np.float16}
_FAST_DTYPES = ("bf16", "f32")

REASONS = ["none", "forced", "dtype", "groups", "stride_t", "pad_right",
           "no_output", "no_tap", "kt1", "spatial"]


class _Desc(C.Structure):
    _fields_ = [(f, C.c_int64) for f in _FIELDS]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        lib = C.CDLL(_LIB_PATH)
        P = C.POINTER
        vp, i64, dp = C.c_void_p, C.c_int64, P(C.c_double)
        lib.ora_output_dims.argtypes = [P(_Desc), P(i64), P(i64), P(i64), P(i64)]
        lib.ora_tap_interval.argtypes = [P(_Desc), i64, P(i64), P(i64)]
        lib.ora_route.argtypes = [P(_Desc), C.c_int, C.c_int, P(C.c_int), P(C.c_int)]
        lib.ora_conv3d_rows.argtypes = [P(_Desc), C.c_int, vp, vp, vp, vp, i64, i64, dp]
        lib.ora_conv3d.argtypes = [P(_Desc), C.c_int, vp, vp, vp, vp, dp]
        lib.ora_conv3d_points.argtypes = [P(_Desc), C.c_int, vp, vp, vp, vp, i64,
                                          P(i64), dp]
        lib.ora_cache_update.argtypes = [P(_Desc), C.c_int, vp, vp, vp]
        lib.ora_flops.argtypes = [P(_Desc)]
        lib.ora_flops.restype = C.c_double
        lib.ora_num_threads.restype = C.c_int
        lib.ora_round_bf16.argtypes = [C.c_double]
        lib.ora_round_bf16.restype = C.c_uint16
        lib.ora_silu.argtypes = [C.c_double]
        lib.ora_silu.restype = C.c_double
        lib.ora_prologue_bf16.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp]
        lib.ora_rms_prologue_bf16.argtypes = [i64, i64, i64, i64, vp, vp, vp, C.c_double, vp,
                                              vp]
        _lib = lib
    return _lib


def _desc(spec: dict) -> _Desc:
    d = _Desc()
    for f in _FIELDS:
        setattr(d, f, int(spec[f]))
    return d


def _host(a, dtype: str):
    """A C-contiguous numpy view of ``a`` in the element type ``dtype``.

    Accepts numpy arrays and CPU torch tensors (bf16 tensors are viewed as
    their raw 16-bit patterns)."""
    if a is None:
        return None
    if hasattr(a, "detach"):  # torch tensor, CPU only
        t = a.detach()
        if t.device.type != "cpu":
            raise ValueError("oracle takes host memory only")
        if dtype == "bf16":
            import torch
            t = t.contiguous().view(torch.int16)
        a = t.contiguous().numpy()
        if dtype == "bf16":
            a = a.view(np.uint16)
    a = np.ascontiguousarray(a)
    want = _NP[dtype]
    if dtype == "f16" and a.dtype == np.uint16:
        a = a.view(np.float16)
    if a.dtype != want:
        raise TypeError(f"expected {np.dtype(want)} data for {dtype}, got {a.dtype}")
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def num_threads() -> int:
    return _load().ora_num_threads()


def output_dims(spec: dict):
    """(T_o, H_o, W_o, L): Eq. 3 and its spatial analogue, and the cache length."""
    lib = _load()
    v = [C.c_int64() for _ in range(4)]
    _check(lib.ora_output_dims(C.byref(_desc(spec)), *[C.byref(x) for x in v]),
           "output_dims")
    return tuple(int(x.value) for x in v)


def tap_interval(spec: dict, k: int):
    """Eq. 4: the output-frame interval [o_l, o_h) that tap k contributes to."""
    lib = _load()
    lo, hi = C.c_int64(), C.c_int64()
    _check(lib.ora_tap_interval(C.byref(_desc(spec)), k, C.byref(lo), C.byref(hi)),
           "tap_interval")
    return int(lo.value), int(hi.value)


def route(spec: dict, dtype: str, force_fallback: bool = False):
    """("fast"|"fallback", reason name) for one call under the written rule."""
    lib = _load()
    r, why = C.c_int(), C.c_int()
    _check(lib.ora_route(C.byref(_desc(spec)), int(dtype in _FAST_DTYPES),
                         int(bool(force_fallback)), C.byref(r), C.byref(why)), "route")
    return ("fast" if r.value == 0 else "fallback"), REASONS[why.value]


def flops(spec: dict) -> float:
    return float(_load().ora_flops(C.byref(_desc(spec))))


def _inputs(spec, dtype, x, cache, w, b):
    x = _host(x, dtype)
    cache = _host(cache, dtype) if spec["Tc"] > 0 else None
    w = _host(w, dtype)
    b = _host(b, dtype) if spec["has_bias"] else None
    N, Ci, Co = spec["N"], spec["Ci"], spec["Co"]
    hw = spec["H"] * spec["W"]
    if x is not None and x.size != N * Ci * spec["T"] * hw:
        raise ValueError("x has the wrong number of elements")
    if cache is not None and cache.size != N * Ci * spec["Tc"] * hw:
        raise ValueError("cache has the wrong number of elements")
    nw = Co * (Ci // spec["groups"]) * spec["Kt"] * spec["Kh"] * spec["Kw"]
    if w.size != nw:
        raise ValueError("w has the wrong number of elements")
    if b is not None and b.size != Co:
        raise ValueError("bias has the wrong number of elements")
    return x, cache, w, b


def conv3d(spec: dict, dtype: str, x, cache, w, b) -> np.ndarray:
    """The whole output, fp64, shaped (N, Co, T_o, H_o, W_o)."""
    lib = _load()
    To, Ho, Wo, _ = output_dims(spec)
    x, cache, w, b = _inputs(spec, dtype, x, cache, w, b)
    y = np.empty((spec["N"], spec["Co"], To, Ho, Wo), np.float64)
    _check(lib.ora_conv3d(C.byref(_desc(spec)), _DTYPES[dtype], _ptr(x), _ptr(cache),
                          _ptr(w), _ptr(b),
                          y.ctypes.data_as(C.POINTER(C.c_double))), "conv3d")
    return y


def conv3d_rows(spec: dict, dtype: str, x, cache, w, b, row0: int, row1: int):
    """Output rows [row0, row1) of the flattened (n, co, t, h) space, fp64."""
    lib = _load()
    _, _, Wo, _ = output_dims(spec)
    x, cache, w, b = _inputs(spec, dtype, x, cache, w, b)
    y = np.empty((row1 - row0, Wo), np.float64)
    _check(lib.ora_conv3d_rows(C.byref(_desc(spec)), _DTYPES[dtype], _ptr(x),
                               _ptr(cache), _ptr(w), _ptr(b), row0, row1,
                               y.ctypes.data_as(C.POINTER(C.c_double))), "conv3d_rows")
    return y


def conv3d_points(spec: dict, dtype: str, x, cache, w, b, idx) -> np.ndarray:
    """Selected outputs by flat NCTHW index, fp64."""
    lib = _load()
    x, cache, w, b = _inputs(spec, dtype, x, cache, w, b)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, np.float64)
    _check(lib.ora_conv3d_points(C.byref(_desc(spec)), _DTYPES[dtype], _ptr(x),
                                 _ptr(cache), _ptr(w), _ptr(b), idx.size,
                                 idx.ctypes.data_as(C.POINTER(C.c_int64)),
                                 out.ctypes.data_as(C.POINTER(C.c_double))),
           "conv3d_points")
    return out


def cache_update(spec: dict, dtype: str, x, cache) -> np.ndarray:
    """cache' = last L frames of [C; X], bytes copied, shaped (N, Ci, L, H, W)."""
    lib = _load()
    _, _, _, L = output_dims(spec)
    x = _host(x, dtype)
    cache = _host(cache, dtype) if spec["Tc"] > 0 else None
    out = np.empty((spec["N"], spec["Ci"], L, spec["H"], spec["W"]), _NP[dtype])
    _check(lib.ora_cache_update(C.byref(_desc(spec)), _DTYPES[dtype], _ptr(x),
                                _ptr(cache), _ptr(out)), "cache_update")
    return out


# ---------------------------------------------------------------- fused form
def round_bf16(v) -> np.ndarray:
    """Nearest bf16 (ties to even) of each fp64 value, as uint16 bits."""
    lib = _load()
    v = np.ascontiguousarray(v, dtype=np.float64)
    return np.array([lib.ora_round_bf16(float(e)) for e in v.ravel()], np.uint16).reshape(v.shape)


def silu(v) -> np.ndarray:
    """SiLU(v) = v / (1 + e^-v) in fp64, elementwise."""
    lib = _load()
    v = np.ascontiguousarray(v, dtype=np.float64)
    return np.array([lib.ora_silu(float(e)) for e in v.ravel()], np.float64).reshape(v.shape)


def prologue_bf16(spec: dict, x, scale, shift) -> np.ndarray:
    """u = RNE_bf16(SiLU(x * scale[n, c] + shift[n, c])) over the new chunk x
    (N, Ci, T, H, W) bf16 bits; scale / shift are fp32 (N, Ci)."""
    lib = _load()
    N, Ci, T, hw = spec["N"], spec["Ci"], spec["T"], spec["H"] * spec["W"]
    x = _host(x, "bf16")
    sc = np.ascontiguousarray(_host(scale, "f32")).reshape(-1)
    sh = np.ascontiguousarray(_host(shift, "f32")).reshape(-1)
    if x.size != N * Ci * T * hw or sc.size != N * Ci or sh.size != N * Ci:
        raise ValueError("prologue arguments have the wrong number of elements")
    u = np.empty((N, Ci, T, spec["H"], spec["W"]), np.uint16)
    _check(lib.ora_prologue_bf16(N, Ci, T, hw, _ptr(x), _ptr(sc), _ptr(sh), _ptr(u)),
           "prologue_bf16")
    return u


def rms_prologue_bf16(spec: dict, x, gamma, beta, eps: float, with_rms: bool = False):
    """u = RNE_bf16(SiLU(x / rms[n, t, p] * gamma[c] + beta[c])) over the new
    chunk x (N, Ci, T, H, W) bf16 bits, rms = sqrt(mean over the Ci channels of
    x^2 + eps) per pixel; gamma / beta fp32 (Ci,).  With ``with_rms`` also the
    fp64 rms (N, T, H, W)."""
    lib = _load()
    N, Ci, T, hw = spec["N"], spec["Ci"], spec["T"], spec["H"] * spec["W"]
    x = _host(x, "bf16")
    g = np.ascontiguousarray(_host(gamma, "f32")).reshape(-1)
    b = np.ascontiguousarray(_host(beta, "f32")).reshape(-1)
    if x.size != N * Ci * T * hw or g.size != Ci or b.size != Ci:
        raise ValueError("normalised prologue arguments have the wrong number of elements")
    u = np.empty((N, Ci, T, spec["H"], spec["W"]), np.uint16)
    rms = np.empty((N, T, spec["H"], spec["W"]), np.float64)
    _check(lib.ora_rms_prologue_bf16(N, Ci, T, hw, _ptr(x), _ptr(g), _ptr(b), float(eps),
                                     _ptr(u), _ptr(rms)), "rms_prologue_bf16")
    return (u, rms) if with_rms else u


def _widen_bf16(a) -> np.ndarray:
    a = _host(a, "bf16")
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def conv3d_block(spec: dict, x, cache, w, b, gamma, beta, eps: float, residual=None):
    """The normalised residual-block call, bf16: the new chunk through
    rms_prologue_bf16, the convolution on [C; u], the residual (bf16, y's
    shape, or None) added after the bias.  Returns (y fp64, cache' bf16 bits)."""
    u = rms_prologue_bf16(spec, x, gamma, beta, eps)
    y = conv3d(spec, "bf16", u, cache, w, b)
    if residual is not None:
        r = _widen_bf16(residual)
        if r.size != y.size:
            raise ValueError("residual has the wrong number of elements")
        y = y + r.reshape(y.shape)
    return y, cache_update(spec, "bf16", u, cache)


def conv3d_fused(spec: dict, x, cache, w, b, scale=None, shift=None, residual=None):
    """The fused residual-block call, bf16: (y fp64 (N, Co, T_o, H_o, W_o),
    cache' bf16 bits (N, Ci, L, H, W)).  scale and shift are given together or
    not at all (then u = x); residual (bf16, y's shape) may be None."""
    if (scale is None) != (shift is None):
        raise ValueError("scale and shift go together")
    u = prologue_bf16(spec, x, scale, shift) if scale is not None else _host(x, "bf16")
    y = conv3d(spec, "bf16", u, cache, w, b)
    if residual is not None:
        r = _widen_bf16(residual)
        if r.size != y.size:
            raise ValueError("residual has the wrong number of elements")
        y = y + r.reshape(y.shape)
    return y, cache_update(spec, "bf16", u, cache)
