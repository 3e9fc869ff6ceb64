"""The fuzz cases reach the kernels they are drawn for (host-side plan
query, no GPU needed), so that the GPU fuzz run covers every kernel."""
from collections import Counter

from paper_2609_31938_amd import c3c

from fuzz_cases import cases


def test_fuzz_cases_cover_every_kernel():
    got, tiles = Counter(), Counter()
    for dtype, sp, kernel, mode, ws in cases():
        ctx = c3c.Context(mode)
        need = c3c.workspace_bytes(sp, dtype) if ws else 0
        pl = c3c.plan_query(ctx, sp, dtype, need)
        if kernel is not None:
            assert pl["kernel"] == kernel, (dtype, sp, pl)
        if pl["kernel"] == "conv3d_bf16":
            tiles[pl["tile_co"], pl["tile_h"], pl["tile_w"]] += 1
        if mode & c3c.MODE_FORCE_FALLBACK:
            assert pl["route"] == "fallback"
        elif kernel == "fallback_direct":
            assert pl["route"] == "fallback" and pl["reason"] != "none", (sp, pl)
        else:
            assert pl["route"] == "fast", (dtype, sp, pl)
        if ws:
            assert pl["splits"] > 1, (sp, pl)
            got["split-K"] += 1
        got[pl["kernel"]] += 1
    n = sum(v for k, v in got.items() if k != "split-K")
    assert n >= 200
    for k in ("conv3d_bf16", "head", "tap1x1", "pointwise", "fast_f32", "fallback_direct",
              "split-K"):
        assert got[k] >= 10, got
    # every tile of the implicit-GEMM kernel
    for t in ((16, 8, 64), (96, 6, 64), (128, 4, 80), (160, 4, 80), (192, 4, 64), (64, 4, 64)):
        assert tiles[t] >= 3, tiles
