"""Helpers shared by the GPU tests: seeded inputs, host copies for the oracle,
error metrics, sampled output indices.  No convolution arithmetic here."""
import sys

import numpy as np
import torch

import oracle
from paper_2609_31938_amd import c3c, inputs

TOL = {"bf16": 2e-2, "f32": 1e-5, "f16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host(t):
    return t.detach().cpu()


def as_f64(t):
    """Exact widening of a host tensor's values (bf16/f16/f32) to fp64."""
    return t.detach().cpu().to(torch.float64).numpy()


def metrics(got, ref):
    """max|err|/max|ref|, max|err|, RMSE, cosine (fp64), NaN/Inf count."""
    g = np.asarray(got, dtype=np.float64).ravel()
    r = np.asarray(ref, dtype=np.float64).ravel()
    if r.size == 0:
        return dict(rel=0.0, max_abs=0.0, rmse=0.0, cos=1.0, nonfinite=0)
    err = np.abs(g - r)
    m = np.max(np.abs(r))
    nf = int(np.count_nonzero(~np.isfinite(g)))
    denom = np.linalg.norm(g) * np.linalg.norm(r)
    return dict(rel=float(np.max(err) / m) if m > 0 else float(np.max(err)),
                max_abs=float(np.max(err)), rmse=float(np.sqrt(np.mean(err ** 2))),
                cos=float(g @ r / denom) if denom > 0 else 1.0, nonfinite=nf)


def check(got, ref, dtype, what=""):
    m = metrics(got, ref)
    assert m["nonfinite"] == 0, (what, m)
    assert m["rel"] <= TOL[dtype], (what, m)
    return m


def layer(sp, dtype, wid=900, lid=0, device="cuda"):
    w, b = inputs.layer_tensors(sp, dtype, wid, lid, device)
    return w, b


def chunk(sp, dtype, wid=900, lid=0, ci=0, device="cuda"):
    return inputs.chunk_input(sp, dtype, wid, lid, ci, device)


def sample_indices(shape, n_random=2048, seed=0):
    """Flat NCTHW indices: random ones plus every tile-border row/column of a
    few (n, co, t) planes (first/last rows and columns, multiples of 32
    around them)."""
    N, Co, To, Ho, Wo = shape
    rng = np.random.default_rng(seed)
    total = N * Co * To * Ho * Wo
    idx = [rng.integers(0, total, n_random)]
    hs = sorted({0, 1, Ho - 2, Ho - 1} & set(range(Ho)))
    ws = sorted(({0, 1, 31, 32, 33, 63, 64, 65, Wo - 33, Wo - 32, Wo - 2, Wo - 1}) & set(range(Wo)))
    for n in {0, N - 1}:
        for co in {0, Co - 1, Co // 2, min(31, Co - 1), min(32, Co - 1)}:
            for t in {0, To - 1}:
                base = ((n * Co + co) * To + t) * Ho * Wo
                for h in hs:
                    for w_ in ws:
                        idx.append(np.array([base + h * Wo + w_]))
    out = np.unique(np.concatenate(idx))
    return out[(out >= 0) & (out < total)]


def run(ctx, sp, x, cache, w, wpack, b):
    y, co = c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b)
    torch.cuda.synchronize()
    return y, co


def oracle_args(sp, x, cache, w, b):
    """Host copies in the form the oracle takes."""
    return (host(x), host(cache) if sp["Tc"] else None, host(w),
            host(b) if sp["has_bias"] else None)
