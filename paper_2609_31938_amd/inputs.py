"""Seeded synthetic inputs and the layer shapes they are drawn for.

This module is plumbing shared by the tests, the benchmark and the smoke
check: it draws random tensors and describes call shapes.  It holds none of
the convolution's arithmetic.

Distributions (the decoder-layer stand-ins; no model weights are used):
  x ~ N(0, 1),  w ~ N(0, 1 / (Ci * Kt * Kh * Kw)),  b ~ N(0, 0.1)  (variance),
drawn in fp32 and rounded to nearest-even into the call's dtype.  The fused
form's extra operands: scale ~ 1 + N(0, 0.2^2) and shift ~ N(0, 0.5^2) per
(batch element, input channel), fp32 (a folded normalisation's scale and
shift), and a residual ~ N(0, 1) shaped like the output; the normalised block
form's gain ~ 1 + N(0, 0.2^2) and bias ~ N(0, 0.5^2) per input channel.  Each tensor
has its own seed, derived from (workload, layer, tensor, chunk); weights and
bias use chunk 0 so that a layer keeps its weights over a stream.
"""
from __future__ import annotations

import hashlib
import math

import numpy as np

TENSOR_X, TENSOR_W, TENSOR_B = 0, 1, 2
TENSOR_SCALE, TENSOR_SHIFT, TENSOR_RES = 3, 4, 5
TENSOR_GAMMA, TENSOR_BETA = 6, 7


def spec(N=1, Ci=1, Co=1, T=1, Tc=0, H=1, W=1, Kt=3, Kh=3, Kw=3,
         s_t=1, s_h=1, s_w=1, d_t=1, d_h=1, d_w=1, p_base=None, p_r=0,
         p_h=None, p_w=None, groups=1, has_bias=1) -> dict:
    """A call description.  By default the temporal pad sits wholly on the
    left (p_base = d_t (Kt - 1), p_r = 0) and the spatial pad is 'same' for
    odd kernels."""
    if p_base is None:
        p_base = d_t * (Kt - 1)
    if p_h is None:
        p_h = d_h * (Kh - 1) // 2
    if p_w is None:
        p_w = d_w * (Kw - 1) // 2
    return dict(N=N, Ci=Ci, Co=Co, T=T, Tc=Tc, H=H, W=W, Kt=Kt, Kh=Kh, Kw=Kw,
                s_t=s_t, s_h=s_h, s_w=s_w, d_t=d_t, d_h=d_h, d_w=d_w,
                p_base=p_base, p_r=p_r, p_h=p_h, p_w=p_w, groups=groups,
                has_bias=int(has_bias))


def seed_of(workload: int, layer: int, tensor: int, chunk: int) -> int:
    ss = np.random.SeedSequence([workload, layer, tensor, chunk])
    return int(ss.generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def _torch_dtype(dtype: str):
    import torch
    return {"bf16": torch.bfloat16, "f32": torch.float32, "f16": torch.float16,
            "f64": torch.float64}[dtype]


def randn(shape, seed: int, std: float, dtype: str, device="cpu"):
    """N(0, std^2) drawn in fp32 with a seeded torch generator on ``device``,
    then rounded to ``dtype``.  The same (seed, shape, device kind) always
    gives the same bytes."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        t.mul_(std)
    return t.to(_torch_dtype(dtype))


def layer_tensors(sp: dict, dtype: str, workload: int, layer: int, device="cpu"):
    """(w, b) for one layer: w ~ N(0, 1/(Ci Kt Kh Kw)), b ~ N(0, 0.1)."""
    cig = sp["Ci"] // sp["groups"]
    fan_in = cig * sp["Kt"] * sp["Kh"] * sp["Kw"]
    w = randn((sp["Co"], cig, sp["Kt"], sp["Kh"], sp["Kw"]),
              seed_of(workload, layer, TENSOR_W, 0), 1.0 / math.sqrt(fan_in),
              dtype, device)
    b = randn((sp["Co"],), seed_of(workload, layer, TENSOR_B, 0), math.sqrt(0.1),
              dtype, device)
    return w, b


def chunk_input(sp: dict, dtype: str, workload: int, layer: int, chunk: int,
                device="cpu"):
    """x ~ N(0, 1) for one chunk, shaped (N, Ci, T, H, W)."""
    return randn((sp["N"], sp["Ci"], sp["T"], sp["H"], sp["W"]),
                 seed_of(workload, layer, TENSOR_X, chunk), 1.0, dtype, device)


def affine_inputs(sp: dict, workload: int, layer: int, chunk: int, device="cpu"):
    """(scale, shift), fp32 (N, Ci): 1 + N(0, 0.04) and N(0, 0.25)."""
    shape = (sp["N"], sp["Ci"])
    scale = randn(shape, seed_of(workload, layer, TENSOR_SCALE, chunk), 0.2, "f32", device)
    scale.add_(1.0)
    shift = randn(shape, seed_of(workload, layer, TENSOR_SHIFT, chunk), 0.5, "f32", device)
    return scale, shift


def norm_inputs(sp: dict, workload: int, layer: int, device="cpu"):
    """(gamma, beta), fp32 (Ci,): 1 + N(0, 0.04) and N(0, 0.25), the
    normalised block form's per-channel gain and bias (a layer's own, chunk 0)."""
    gamma = randn((sp["Ci"],), seed_of(workload, layer, TENSOR_GAMMA, 0), 0.2, "f32", device)
    gamma.add_(1.0)
    beta = randn((sp["Ci"],), seed_of(workload, layer, TENSOR_BETA, 0), 0.5, "f32", device)
    return gamma, beta


def residual_input(shape, dtype: str, workload: int, layer: int, chunk: int, device="cpu"):
    """A residual ~ N(0, 1) of the given (output) shape."""
    return randn(shape, seed_of(workload, layer, TENSOR_RES, chunk), 1.0, dtype, device)


def zero_cache(sp: dict, dtype: str, device="cpu"):
    import torch
    return torch.zeros((sp["N"], sp["Ci"], sp["Tc"], sp["H"], sp["W"]),
                       dtype=_torch_dtype(dtype), device=device)


def sha256(t) -> str:
    """SHA-256 of a tensor's bytes (host copy), for provenance records."""
    import torch
    a = t.detach().contiguous().cpu()
    if a.dtype in (torch.bfloat16, torch.float16):
        a = a.view(torch.int16)
    return hashlib.sha256(a.numpy().tobytes()).hexdigest()


# ---------------------------------------------------------------------------
# Workloads: Wan-VAE-decoder-shaped causal Conv3D layers (N = 1, 3x3x3,
# stride 1, spatial pad 1, a 2-frame temporal cache that starts at zeros).
# Each entry: name -> dict(dtype, chunks, layers=[(layer_name, spec), ...]).
# ---------------------------------------------------------------------------

def _c(Ci, Co, T, H, W, Tc=2):
    return spec(N=1, Ci=Ci, Co=Co, T=T, Tc=Tc, H=H, W=W)


WORKLOADS = {
    # 1: tiny fp32 case that the oracle finishes at once
    "tiny_f32": dict(id=1, dtype="f32", chunks=4,
                     layers=[("c32_32x32", _c(32, 32, 2, 32, 32))]),
    # 2: lowest-resolution decoder layer, one new frame per chunk
    "low_res": dict(id=2, dtype="bf16", chunks=21,
                    layers=[("c384_60x104", _c(384, 384, 1, 60, 104))]),
    # 3: mid-resolution decoder layers
    "mid_res": dict(id=3, dtype="bf16", chunks=5,
                    layers=[("c192_240x416", _c(192, 192, 4, 240, 416)),
                            ("c384to192_240x416", _c(384, 192, 4, 240, 416))]),
    # 4: full-resolution short-temporal layer
    "full_res": dict(id=4, dtype="bf16", chunks=5,
                     layers=[("c96_480x832", _c(96, 96, 4, 480, 832))]),
    # 5: 720p wide-channel decode stack plus a 1x1x1 shortcut conv
    "stack_720p": dict(id=5, dtype="bf16", chunks=5,
                       layers=[("c640_44x80", _c(640, 640, 4, 44, 80)),
                               ("c320_176x320", _c(320, 320, 4, 176, 320)),
                               ("c320to160_352x640", _c(320, 160, 4, 352, 640)),
                               ("c160_704x1280", _c(160, 160, 4, 704, 1280)),
                               ("shortcut_1x1x1_320to160_352x640",
                                spec(N=1, Ci=320, Co=160, T=4, Tc=0, H=352, W=640,
                                     Kt=1, Kh=1, Kw=1))]),
    # 7: the decoder's output head (to 3 channels, RGB) at full resolution
    "head": dict(id=7, dtype="bf16", chunks=5,
                 layers=[("head_96to3_480x832", _c(96, 3, 4, 480, 832))]),
    # 6: temporal convolutions (kernel 3x1x1) of the decoder's temporal
    # upsampling (channels doubled, then split into two frames by the
    # decoder) and of an encoder's stride-2 temporal downsampling
    "temporal": dict(id=6, dtype="bf16", chunks=5,
                     layers=[("tconv_up_384to768_60x104",
                              spec(N=1, Ci=384, Co=768, T=1, Tc=2, H=60, W=104, Kh=1, Kw=1)),
                             ("tconv_up_384to768_120x208",
                              spec(N=1, Ci=384, Co=768, T=2, Tc=2, H=120, W=208, Kh=1, Kw=1)),
                             ("tconv_down_s2_384_120x208",
                              spec(N=1, Ci=384, Co=384, T=8, Tc=1, H=120, W=208, Kh=1, Kw=1,
                                   s_t=2, p_base=1))]),
}
