"""Python binding of libc3c (ctypes): argument marshalling only.

Every step of the cached causal Conv3D runs in the HIP library; this module
turns torch device tensors into pointers, passes torch's current HIP stream,
and maps status codes to exceptions.  It imports nothing else from this
repository.  Importing it raises if ``libc3c.so`` has not been built (run
``python -m paper_2609_31938_amd.build``): there is no CPU fallback.

Call shapes are described by the same plain ``spec`` dict the input module
builds (keys ``N Ci Co T Tc H W Kt Kh Kw s_t s_h s_w d_t d_h d_w p_base p_r
p_h p_w groups has_bias``); element types are ``"bf16" "f32" "f16"``.
"""
from __future__ import annotations

import ctypes as C
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
# C3C_LIB selects another build of the same library (the sanitizer build of
# the host-side test run); by default the in-tree build next to this file
LIB_PATH = os.environ.get("C3C_LIB") or os.path.join(_HERE, "libc3c.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "c3c.h")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with "
                      "`python -m paper_2609_31938_amd.build` (no CPU fallback exists)")

# torch first: the library must bind to the HIP runtime torch loads, so that
# both use one runtime (and see the same devices, streams and memory).  Loaded
# the other way round, the library would load the system runtime next to
# torch's bundled one, and its calls would find no device.
import torch  # noqa: E402,F401

OK, E_INVAL, E_UNSUPPORTED, E_DEVICE, E_INJECTED = 0, 1, 2, 3, 4
DTYPES = {"bf16": 1, "f32": 2, "f16": 3}
MODE_STRICT, MODE_FORCE_FALLBACK, MODE_INJECT_FAST_FAILURE, MODE_CHANNEL_TILES = 1, 2, 4, 8
ROUTES = ["fast", "fallback"]
REASONS = ["none", "forced", "dtype", "groups", "stride_t", "pad_right", "no_output",
           "no_tap", "kt1", "spatial", "fast_error"]
NOALLOC_SCRATCH_BYTES = 64 << 20  # C3C_NOALLOC_SCRATCH_BYTES
KERNELS = ["none", "conv3d_bf16", "head", "tap1x1", "pointwise", "fast_f32", "fallback_direct"]


class C3CError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"c3c status {status}: {msg}")
        self.status = status


class Desc(C.Structure):
    _fields_ = [(n, C.c_int64) for n in
                ("N", "Ci", "Co", "T", "Tc", "H", "W", "Kt", "Kh", "Kw",
                 "stride_t", "stride_h", "stride_w", "dil_t", "dil_h", "dil_w",
                 "pad_t_base", "pad_t_right", "pad_h", "pad_w", "groups")] + \
               [("dtype", C.c_int32), ("has_bias", C.c_int32)]


class Counters(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in ("calls", "fast", "fallback", "unsupported", "forced",
                                          "fast_error", "strict_rejects", "repacks", "failed")]


class Plan(C.Structure):
    _fields_ = [("route", C.c_int32), ("reason", C.c_int32), ("kernel", C.c_int32),
                ("splits", C.c_int32), ("tile_co", C.c_int64), ("tile_h", C.c_int64),
                ("tile_w", C.c_int64), ("workgroups", C.c_int64), ("cache_in_kernel", C.c_int32),
                ("reserved", C.c_int32)]


class SigCount(C.Structure):
    _fields_ = [("reason", C.c_int32), ("reserved", C.c_int32), ("desc", Desc),
                ("count", C.c_uint64)]


lib = C.CDLL(LIB_PATH)
_P, _vp, _i64 = C.POINTER, C.c_void_p, C.c_int64
lib.c3c_ctx_create.argtypes = [C.c_uint32, _P(_vp)]
lib.c3c_ctx_destroy.argtypes = [_vp]
lib.c3c_set_mode.argtypes = [_vp, C.c_uint32]
lib.c3c_get_mode.argtypes = [_vp, _P(C.c_uint32)]
lib.c3c_output_dims.argtypes = [_P(Desc), _P(_i64), _P(_i64), _P(_i64), _P(_i64)]
lib.c3c_tap_interval.argtypes = [_P(Desc), _i64, _P(_i64), _P(_i64)]
lib.c3c_flops.argtypes = [_P(Desc), _P(C.c_double)]
lib.c3c_route_query.argtypes = [_vp, _P(Desc), _P(C.c_int), _P(C.c_int)]
lib.c3c_plan_query.argtypes = [_vp, _P(Desc), C.c_size_t, _P(Plan)]
lib.c3c_weight_pack_bytes.argtypes = [_P(Desc), _P(C.c_size_t)]
lib.c3c_workspace_bytes.argtypes = [_P(Desc), _P(C.c_size_t)]
lib.c3c_fused_workspace_bytes.argtypes = [_P(Desc), _P(C.c_size_t)]
lib.c3c_ctx_set_workspace.argtypes = [_vp, _vp, C.c_size_t]
lib.c3c_weight_repack.argtypes = [_vp, _P(Desc), _vp, _vp, _vp]
lib.c3c_weight_unpack.argtypes = [_P(Desc), _vp, _vp, _vp]
lib.c3c_conv3d_causal_cached.argtypes = [_vp, _P(Desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
lib.c3c_conv3d_causal_cached_fused.argtypes = [_vp, _P(Desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                               _vp, _vp, _vp, _vp]
lib.c3c_conv3d_causal_cached_noalloc.argtypes = [_vp, _P(Desc), _vp, _vp, _vp, _vp, _vp, _vp,
                                                 _vp, _vp]
lib.c3c_block_workspace_bytes.argtypes = [_P(Desc), _P(C.c_size_t)]
lib.c3c_conv3d_causal_cached_block.argtypes = [_vp, _P(Desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                               C.c_float, _vp, _vp, _vp, _vp]
lib.c3c_counters_get.argtypes = [_vp, _P(Counters)]
lib.c3c_mfma_probe.argtypes = [C.c_int64, C.c_int64, _vp, _P(C.c_double), _vp]
lib.c3c_counters_reset.argtypes = [_vp]
lib.c3c_fallback_shapes.argtypes = [_vp, _P(SigCount), C.c_int, _P(C.c_int)]
lib.c3c_strerror.argtypes = [C.c_int]
lib.c3c_strerror.restype = C.c_char_p
lib.c3c_last_error.argtypes = [_vp]
lib.c3c_last_error.restype = C.c_char_p


def declared_symbols():
    """Function names declared in include/c3c.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(c3c_\w+)\s*\(", text, re.M)))


def make_desc(spec: dict, dtype: str) -> Desc:
    d = Desc()
    d.N, d.Ci, d.Co, d.T, d.Tc = spec["N"], spec["Ci"], spec["Co"], spec["T"], spec["Tc"]
    d.H, d.W, d.Kt, d.Kh, d.Kw = spec["H"], spec["W"], spec["Kt"], spec["Kh"], spec["Kw"]
    d.stride_t, d.stride_h, d.stride_w = spec["s_t"], spec["s_h"], spec["s_w"]
    d.dil_t, d.dil_h, d.dil_w = spec["d_t"], spec["d_h"], spec["d_w"]
    d.pad_t_base, d.pad_t_right = spec["p_base"], spec["p_r"]
    d.pad_h, d.pad_w, d.groups = spec["p_h"], spec["p_w"], spec["groups"]
    d.dtype = DTYPES[dtype]
    d.has_bias = int(spec["has_bias"])
    return d


def _raise(status, ctx=None, what=""):
    if status != OK:
        msg = lib.c3c_strerror(status).decode()
        if ctx is not None:
            extra = lib.c3c_last_error(ctx._h).decode()
            if extra:
                msg += f" ({extra})"
        raise C3CError(status, f"{what}: {msg}")


class Context:
    """A c3c_ctx: mode bits, route counters and the fallback-shape histogram."""

    def __init__(self, mode: int = 0):
        h = _vp()
        _raise(lib.c3c_ctx_create(mode, C.byref(h)), what="c3c_ctx_create")
        self._h = h

    def close(self):
        if self._h:
            lib.c3c_ctx_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def mode(self) -> int:
        m = C.c_uint32()
        _raise(lib.c3c_get_mode(self._h, C.byref(m)), self, "c3c_get_mode")
        return m.value

    @mode.setter
    def mode(self, m: int):
        _raise(lib.c3c_set_mode(self._h, m), self, "c3c_set_mode")

    def counters(self) -> dict:
        c = Counters()
        _raise(lib.c3c_counters_get(self._h, C.byref(c)), self, "c3c_counters_get")
        return {n: int(getattr(c, n)) for n, _ in Counters._fields_}

    def reset(self):
        _raise(lib.c3c_counters_reset(self._h), self, "c3c_counters_reset")

    def fallback_shapes(self):
        """[(reason, desc fields dict, count)] in first-seen order."""
        n = C.c_int()
        _raise(lib.c3c_fallback_shapes(self._h, None, 0, C.byref(n)), self, "c3c_fallback_shapes")
        arr = (SigCount * max(n.value, 1))()
        _raise(lib.c3c_fallback_shapes(self._h, arr, n.value, C.byref(n)), self,
               "c3c_fallback_shapes")
        out = []
        for i in range(n.value):
            e = arr[i]
            out.append((REASONS[e.reason], {f: getattr(e.desc, f) for f, _ in Desc._fields_},
                        int(e.count)))
        return out

    @property
    def last_error(self) -> str:
        return lib.c3c_last_error(self._h).decode()

    def set_workspace(self, ws=None):
        """Attach a device tensor as the split-K workspace (None detaches).
        The context keeps a reference so the memory outlives its use."""
        if ws is None:
            _raise(lib.c3c_ctx_set_workspace(self._h, None, 0), self, "c3c_ctx_set_workspace")
            self._ws = None
            return
        if not ws.is_cuda or not ws.is_contiguous():
            raise ValueError("workspace must be a contiguous device tensor")
        nbytes = ws.numel() * ws.element_size()
        _raise(lib.c3c_ctx_set_workspace(self._h, ws.data_ptr() or None, nbytes), self,
               "c3c_ctx_set_workspace")
        self._ws = ws


# ---------------------------------------------------------------- host maths

def output_dims(spec: dict, dtype: str = "bf16"):
    v = [_i64() for _ in range(4)]
    _raise(lib.c3c_output_dims(C.byref(make_desc(spec, dtype)), *[C.byref(x) for x in v]),
           what="c3c_output_dims")
    return tuple(int(x.value) for x in v)


def tap_interval(spec: dict, k: int, dtype: str = "bf16"):
    lo, hi = _i64(), _i64()
    _raise(lib.c3c_tap_interval(C.byref(make_desc(spec, dtype)), k, C.byref(lo), C.byref(hi)),
           what="c3c_tap_interval")
    return int(lo.value), int(hi.value)


def flops(spec: dict, dtype: str = "bf16") -> float:
    f = C.c_double()
    _raise(lib.c3c_flops(C.byref(make_desc(spec, dtype)), C.byref(f)), what="c3c_flops")
    return f.value


def route_query(ctx, spec: dict, dtype: str):
    r, why = C.c_int(), C.c_int()
    _raise(lib.c3c_route_query(ctx._h if ctx is not None else None,
                               C.byref(make_desc(spec, dtype)), C.byref(r), C.byref(why)),
           ctx, "c3c_route_query")
    return ROUTES[r.value], REASONS[why.value]


def plan_query(ctx, spec: dict, dtype: str, ws_bytes: int = 0) -> dict:
    """What a plain call would launch (c3c_plan_query): route, reason, kernel
    name, workgroup tile (tile_h == 0: tile_w pixels of the flattened plane),
    workgroups, split-K factor, and whether the kernel writes the cache."""
    p = Plan()
    _raise(lib.c3c_plan_query(ctx._h if ctx is not None else None,
                              C.byref(make_desc(spec, dtype)), ws_bytes, C.byref(p)),
           ctx, "c3c_plan_query")
    return dict(route=ROUTES[p.route], reason=REASONS[p.reason], kernel=KERNELS[p.kernel],
                splits=p.splits, tile_co=p.tile_co, tile_h=p.tile_h, tile_w=p.tile_w,
                workgroups=p.workgroups, cache_in_kernel=bool(p.cache_in_kernel))


def weight_pack_bytes(spec: dict, dtype: str) -> int:
    n = C.c_size_t()
    _raise(lib.c3c_weight_pack_bytes(C.byref(make_desc(spec, dtype)), C.byref(n)),
           what="c3c_weight_pack_bytes")
    return int(n.value)


def workspace_bytes(spec: dict, dtype: str) -> int:
    """Split-K workspace bytes this call would use (0: it runs unsplit)."""
    n = C.c_size_t()
    _raise(lib.c3c_workspace_bytes(C.byref(make_desc(spec, dtype)), C.byref(n)),
           what="c3c_workspace_bytes")
    return int(n.value)


def fused_workspace_bytes(spec: dict, dtype: str) -> int:
    """Workspace bytes with which a fused call runs its prologue as a pass of
    its own (plus split-K); 0 when it would not use one."""
    n = C.c_size_t()
    _raise(lib.c3c_fused_workspace_bytes(C.byref(make_desc(spec, dtype)), C.byref(n)),
           what="c3c_fused_workspace_bytes")
    return int(n.value)


def block_workspace_bytes(spec: dict, dtype: str = "bf16") -> int:
    """Context workspace bytes the normalised block form needs: the activated
    chunk (rounded up to 256 bytes), then the split-K bytes."""
    n = C.c_size_t()
    _raise(lib.c3c_block_workspace_bytes(C.byref(make_desc(spec, dtype)), C.byref(n)),
           what="c3c_block_workspace_bytes")
    return int(n.value)


# ---------------------------------------------------------------- device calls

_TORCH = {}


def _torch_dtype(dtype):
    import torch
    return {"bf16": torch.bfloat16, "f32": torch.float32, "f16": torch.float16}[dtype]


def dtype_of(t) -> str:
    import torch
    return {torch.bfloat16: "bf16", torch.float32: "f32", torch.float16: "f16"}[t.dtype]


def _check(t, name, dtype, numel=None):
    """A tensor's dtype, layout and element count (every extent the kernels
    use comes from the descriptor, so a short buffer would be read or written
    out of bounds)."""
    if t is None:
        return
    if t.dtype != _torch_dtype(dtype):
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")


def _ptr(t, name, dtype, numel=None):
    """The device address of a checked tensor."""
    if t is None:
        return None
    _check(t, name, dtype, numel)
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    return t.data_ptr() or None


def _sizes(spec: dict, dtype: str):
    """Element counts of every tensor of a call: x, cache, w, wpack (0 when
    the call has no fast layout), bias, y, cache_out."""
    To, Ho, Wo, L = output_dims(spec, dtype)
    hw = spec["H"] * spec["W"]
    nci = spec["N"] * spec["Ci"]
    es = 4 if dtype == "f32" else 2
    return dict(x=nci * spec["T"] * hw, cache=nci * spec["Tc"] * hw,
                w=spec["Co"] * (spec["Ci"] // spec["groups"]) * spec["Kt"] * spec["Kh"] * spec["Kw"],
                wpack=weight_pack_bytes(spec, dtype) // es, bias=spec["Co"],
                y=spec["N"] * spec["Co"] * To * Ho * Wo, cache_out=nci * L * hw)


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def weight_repack(ctx, spec: dict, w, wpack=None, stream=None):
    """Pack w into the fast route's matrix-core layout (a new device buffer
    unless ``wpack`` is given).  Returns the packed buffer."""
    import torch
    dtype = dtype_of(w)
    nbytes = weight_pack_bytes(spec, dtype)
    if wpack is None:
        wpack = torch.empty(nbytes // w.element_size(), dtype=w.dtype, device=w.device)
    _raise(lib.c3c_weight_repack(ctx._h if ctx is not None else None,
                                 C.byref(make_desc(spec, dtype)), _ptr(w, "w", dtype),
                                 _ptr(wpack, "wpack", dtype, nbytes // w.element_size()),
                                 _stream(stream)), ctx, "c3c_weight_repack")
    return wpack


def weight_unpack(spec: dict, wpack, out=None, stream=None):
    import torch
    dtype = dtype_of(wpack)
    if out is None:
        out = torch.empty((spec["Co"], spec["Ci"] // spec["groups"], spec["Kt"], spec["Kh"],
                           spec["Kw"]), dtype=wpack.dtype, device=wpack.device)
    _raise(lib.c3c_weight_unpack(C.byref(make_desc(spec, dtype)), _ptr(wpack, "wpack", dtype),
                                 _ptr(out, "w_out", dtype), _stream(stream)),
           what="c3c_weight_unpack")
    return out


def conv3d_causal_cached(ctx, spec: dict, x, cache, w, wpack, bias, y=None, cache_out=None,
                         stream=None):
    """One cached causal Conv3D call.  Returns (y, cache_out); allocates the
    outputs with torch when they are not given."""
    import torch
    dtype = dtype_of(w)
    To, Ho, Wo, L = output_dims(spec, dtype)
    dev = w.device
    if y is None:
        y = torch.empty((spec["N"], spec["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
    if cache_out is None:
        cache_out = torch.empty((spec["N"], spec["Ci"], L, spec["H"], spec["W"]),
                                dtype=w.dtype, device=dev)
    n = _sizes(spec, dtype)
    st = lib.c3c_conv3d_causal_cached(
        ctx._h, C.byref(make_desc(spec, dtype)), *_call_ptrs(spec, dtype, n, x, cache, w, wpack,
                                                            bias, y, cache_out),
        _stream(stream))
    _raise(st, ctx, "c3c_conv3d_causal_cached")
    return y, cache_out


def conv3d_causal_cached_noalloc(ctx, spec: dict, x, cache, w, wpack, bias, y, cache_out,
                                 stream=None):
    """The allocation-free call (c3c_conv3d_causal_cached_noalloc): the
    plain call with any split-K partial sums in the library's own device
    scratch.  The caller passes every output; nothing is allocated here or in
    the library.  Returns (y, cache_out)."""
    dtype = dtype_of(w)
    n = _sizes(spec, dtype)
    if y is None or (cache_out is None and n["cache_out"] > 0):
        raise ValueError("the allocation-free call takes caller-allocated y and cache_out")
    st = lib.c3c_conv3d_causal_cached_noalloc(
        ctx._h, C.byref(make_desc(spec, dtype)), *_call_ptrs(spec, dtype, n, x, cache, w, wpack,
                                                            bias, y, cache_out),
        _stream(stream))
    _raise(st, ctx, "c3c_conv3d_causal_cached_noalloc")
    return y, cache_out


def _call_ptrs(spec, dtype, n, x, cache, w, wpack, bias, y, cache_out):
    """Checked addresses of (x, cache, w, wpack, bias, y, cache_out).  wpack
    must hold exactly the packed layout when the call has one (a pack made
    for another layer would be read out of bounds); it may be None only
    where the call does not route fast (the library then rejects it)."""
    if wpack is not None and n["wpack"] == 0:
        raise ValueError("wpack given, but this call has no fast-route weight layout")
    for t, name in ((x, "x"), (cache if spec["Tc"] else None, "cache"), (w, "w"),
                    (wpack, "wpack"), (bias if spec["has_bias"] else None, "bias"), (y, "y"),
                    (cache_out, "cache_out")):
        _check(t, name, dtype, n[name])
    return (_ptr(x, "x", dtype, n["x"]),
            _ptr(cache, "cache", dtype, n["cache"]) if spec["Tc"] else None,
            _ptr(w, "w", dtype, n["w"]),
            _ptr(wpack, "wpack", dtype, n["wpack"]),
            _ptr(bias, "bias", dtype, n["bias"]) if spec["has_bias"] else None,
            _ptr(y, "y", dtype, n["y"]),
            _ptr(cache_out, "cache_out", dtype, n["cache_out"]))


def conv3d_causal_cached_fused(ctx, spec: dict, x, cache, w, wpack, bias, scale=None, shift=None,
                               residual=None, y=None, cache_out=None, stream=None):
    """The fused residual-block form (bf16): the new chunk read as
    RNE_bf16(SiLU(x * scale[n, ci] + shift[n, ci])) when scale / shift (fp32,
    (N, Ci)) are given, residual (y's shape) added before the rounding.
    ``residual`` may be ``y`` itself.  Returns (y, cache_out)."""
    import torch
    dtype = dtype_of(w)
    To, Ho, Wo, L = output_dims(spec, dtype)
    dev = w.device
    if y is None:
        y = torch.empty((spec["N"], spec["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
    if cache_out is None:
        cache_out = torch.empty((spec["N"], spec["Ci"], L, spec["H"], spec["W"]),
                                dtype=w.dtype, device=dev)
    nc = spec["N"] * spec["Ci"]
    n = _sizes(spec, dtype)
    _check(scale, "scale", "f32", nc)
    _check(shift, "shift", "f32", nc)
    _check(residual, "residual", dtype, n["y"])
    px, pc, pw, pp, pb, py, po = _call_ptrs(spec, dtype, n, x, cache, w, wpack, bias, y, cache_out)
    st = lib.c3c_conv3d_causal_cached_fused(
        ctx._h, C.byref(make_desc(spec, dtype)), px, pc, pw, pp, pb,
        _ptr(scale, "scale", "f32", nc), _ptr(shift, "shift", "f32", nc),
        _ptr(residual, "residual", dtype, n["y"]), py, po, _stream(stream))
    _raise(st, ctx, "c3c_conv3d_causal_cached_fused")
    return y, cache_out


def conv3d_causal_cached_block(ctx, spec: dict, x, cache, w, wpack, bias, gamma, beta,
                               eps: float, residual=None, y=None, cache_out=None, stream=None):
    """The normalised residual-block form (bf16): the new chunk normalised per
    pixel over its channels (RMS with eps), scaled by gamma and shifted by
    beta (fp32, (Ci,)), through SiLU into the context's workspace (which must
    hold block_workspace_bytes), then the convolution on [cache; u] with
    residual (y's shape, may be ``y``) added before the rounding.  Returns
    (y, cache_out)."""
    import torch
    dtype = dtype_of(w)
    To, Ho, Wo, L = output_dims(spec, dtype)
    dev = w.device
    if y is None:
        y = torch.empty((spec["N"], spec["Co"], To, Ho, Wo), dtype=w.dtype, device=dev)
    if cache_out is None:
        cache_out = torch.empty((spec["N"], spec["Ci"], L, spec["H"], spec["W"]),
                                dtype=w.dtype, device=dev)
    n = _sizes(spec, dtype)
    _check(gamma, "gamma", "f32", spec["Ci"])
    _check(beta, "beta", "f32", spec["Ci"])
    _check(residual, "residual", dtype, n["y"])
    px, pc, pw, pp, pb, py, po = _call_ptrs(spec, dtype, n, x, cache, w, wpack, bias, y, cache_out)
    st = lib.c3c_conv3d_causal_cached_block(
        ctx._h, C.byref(make_desc(spec, dtype)), px, pc, pw, pp, pb,
        _ptr(gamma, "gamma", "f32", spec["Ci"]), _ptr(beta, "beta", "f32", spec["Ci"]),
        float(eps), _ptr(residual, "residual", dtype, n["y"]), py, po, _stream(stream))
    _raise(st, ctx, "c3c_conv3d_causal_cached_block")
    return y, cache_out


def mfma_probe(blocks: int, iters: int, stream=None):
    """One launch of the matrix-core rate probe (c3c_mfma_probe), enqueued on
    the stream; returns (out tensor, FLOP count).  The caller times it."""
    import torch
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    fl = C.c_double()
    st = lib.c3c_mfma_probe(blocks, iters, out.data_ptr(), C.byref(fl), _stream(stream))
    _raise(st, None, "c3c_mfma_probe")
    return out, fl.value
