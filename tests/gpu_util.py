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


def tile_borders(extent, tile):
    """Indices on both sides of every tile boundary along one axis, plus the
    first and last index."""
    out = {0, extent - 1}
    if tile > 0:
        for b in range(tile, extent, tile):
            out.update((b - 1, b))
    return sorted(i for i in out if 0 <= i < extent)


def sample_indices(shape, plan=None, n_random=2048, seed=0, n_planes=6, per_border=3):
    """Flat NCTHW indices: random ones, plus points on the tile borders of the
    workgroup grid the call actually used (``plan`` from c3c.plan_query) in
    several (n, co, t) planes -- every border row with a few random columns,
    every border column with a few random rows (for a kernel that tiles the
    flattened plane, every tile boundary of that plane) -- and the first and
    last channel of every output-channel tile."""
    N, Co, To, Ho, Wo = shape
    rng = np.random.default_rng(seed)
    total = N * Co * To * Ho * Wo
    if total == 0:
        return np.zeros(0, np.int64)
    idx = [rng.integers(0, total, n_random)]
    th = plan["tile_h"] if plan else 0
    tw = plan["tile_w"] if plan else 32
    tco = plan["tile_co"] if plan else 32
    cos = set(tile_borders(Co, tco))
    planes = {(0, 0, 0), (N - 1, Co - 1, To - 1)}
    for _ in range(n_planes):
        planes.add((int(rng.integers(N)), int(rng.choice(sorted(cos))), int(rng.integers(To))))
    for n, co, t in planes:
        base = ((n * Co + co) * To + t) * Ho * Wo
        if th > 0:
            for h in tile_borders(Ho, th):
                idx.append(base + h * Wo + rng.integers(0, Wo, per_border))
                idx.append(base + h * Wo + np.array([0, Wo - 1]))
            for w_ in tile_borders(Wo, tw):
                idx.append(base + rng.integers(0, Ho, per_border) * Wo + w_)
                idx.append(base + np.array([0, Ho - 1]) * Wo + w_)
        else:
            idx.append(base + np.array(tile_borders(Ho * Wo, tw)))
    # every output-channel tile's edge channels, at random positions
    for co in cos:
        n, t = int(rng.integers(N)), int(rng.integers(To))
        base = ((n * Co + co) * To + t) * Ho * Wo
        idx.append(base + rng.integers(0, Ho * Wo, per_border))
    out = np.unique(np.concatenate([np.asarray(i, np.int64).ravel() for i in idx]))
    return out[(out >= 0) & (out < total)]


def check_planes(y, sp, dtype, planes, oracle_in, what=""):
    """Whole output planes (n, co, t) compared with the oracle, fp64."""
    N, Co, To, Ho, Wo = y.shape
    hx, hc, hw_, hb = oracle_in
    worst = 0.0
    for n, co, t in planes:
        r0 = ((n * Co + co) * To + t) * Ho
        ref = oracle.conv3d_rows(sp, dtype, hx, hc, hw_, hb, r0, r0 + Ho)
        m = check(as_f64(y[n, co, t]), ref, dtype, f"{what} plane n={n} co={co} t={t}")
        worst = max(worst, m["rel"])
    return worst


GUARD = 4096  # elements of poison on each side of an output


def guarded(shape, dtype, device="cuda"):
    """(tensor, backing buffer): a NaN-filled output inside a larger NaN-filled
    buffer, GUARD elements of poison on each side (16-byte aligned)."""
    td = {"bf16": torch.bfloat16, "f32": torch.float32, "f16": torch.float16}[dtype]
    n = int(np.prod(shape))
    buf = torch.full((n + 2 * GUARD,), float("nan"), dtype=td, device=device)
    return buf[GUARD:GUARD + n].view(shape), buf


def guards_intact(buf):
    """True when the poison on both sides of a guarded output is untouched."""
    return bool(torch.isnan(buf[:GUARD]).all().item()) and bool(torch.isnan(buf[-GUARD:]).all().item())


def run(ctx, sp, x, cache, w, wpack, b):
    y, co = c3c.conv3d_causal_cached(ctx, sp, x, cache, w, wpack, b)
    torch.cuda.synchronize()
    return y, co


def oracle_args(sp, x, cache, w, b):
    """Host copies in the form the oracle takes."""
    return (host(x), host(cache) if sp["Tc"] else None, host(w),
            host(b) if sp["has_bias"] else None)
