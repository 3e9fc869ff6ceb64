"""The test helpers' own index logic (CPU)."""
import numpy as np

from gpu_util import sample_indices, tile_borders


def test_tile_borders():
    assert tile_borders(10, 4) == [0, 3, 4, 7, 8, 9]
    assert tile_borders(5, 0) == [0, 4]
    assert tile_borders(1, 4) == [0]


def test_sample_indices_hit_every_tile_border():
    shape = (1, 20, 3, 13, 170)
    plan = dict(tile_co=16, tile_h=4, tile_w=80)
    idx = sample_indices(shape, plan, 100, seed=0)
    assert idx.min() >= 0 and idx.max() < np.prod(shape)
    w = idx % 170
    h = (idx // 170) % 13
    co = (idx // (170 * 13 * 3)) % 20
    for b in (79, 80, 159, 160):
        assert (w == b).any()
    for b in (3, 4, 7, 8, 11, 12):
        assert (h == b).any()
    for c in (0, 15, 16, 19):
        assert (co == c).any()
    flat = sample_indices(shape, dict(tile_co=160, tile_h=0, tile_w=256), 10, seed=1)
    assert ((flat % (13 * 170)) == 255).any() and ((flat % (13 * 170)) == 256).any()
