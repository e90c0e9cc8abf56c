"""Pins for the oracle's shifted block frame and pooling (Section 2.2.2;
Section 2.2.1, Eq. 1).  Each check is independent of the oracle's own code
path: a hand-worked example, a brute-force forward map of the roll, and the
library 2-D average pool."""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ssba_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _forward_map(grid_h, grid_w, tile, sy, sx):
    """Brute force: where each original token lands (roll moves y to y + s)."""
    nx = grid_w // tile
    where = {}
    for y in range(grid_h):
        for x in range(grid_w):
            y2, x2 = (y + sy) % grid_h, (x + sx) % grid_w
            t = (y2 // tile) * nx + x2 // tile
            s = (y2 % tile) * tile + x2 % tile
            where[y * grid_w + x] = (t, s)
    return where


def test_frame_hand_example():
    path = os.path.join(GOLDEN, "frame_grid64_shift44.txt")
    lines = [l.strip() for l in open(path) if l.strip() and not l.startswith("#")]
    cfg = dict(kv.split("=") for kv in lines[0].split()[1:])
    tiles = O.frame_tiles(int(cfg["grid_h"]), int(cfg["grid_w"]), int(cfg["tile"]),
                          int(cfg["shift_y"]), int(cfg["shift_x"]))
    for line in lines[1:]:
        head, ids = line.split(":")
        blk, s0, s1 = (int(v) for v in head.split())
        assert tiles[blk, s0:s1 + 1].tolist() == [int(v) for v in ids.split()]


@pytest.mark.parametrize("grid_h,grid_w,tile,sy,sx", [
    (16, 16, 4, 2, 2), (16, 16, 4, -2, -2), (16, 8, 4, 3, -1), (8, 16, 4, 0, 5),
    (32, 32, 8, 4, 4), (24, 16, 8, -13, 29), (32, 16, 16, 8, -8), (16, 16, 4, 0, 0),
])
def test_frame_bruteforce(grid_h, grid_w, tile, sy, sx):
    tiles = O.frame_tiles(grid_h, grid_w, tile, sy, sx)
    where = _forward_map(grid_h, grid_w, tile, sy, sx)
    assert tiles.shape == (grid_h * grid_w // tile ** 2, tile * tile)
    for tok, (t, s) in where.items():
        assert tiles[t, s] == tok
    inv = O.tile_of_token(tiles)
    for tok, (t, _) in where.items():
        assert inv[tok] == t


@pytest.mark.parametrize("grid,tile", [(32, 8), (64, 8), (16, 4), (128, 16)])
def test_half_block_shifts_give_the_same_partition(grid, tile):
    h = tile // 2
    a = {frozenset(r.tolist()) for r in O.frame_tiles(grid, grid, tile, h, h)}
    b = {frozenset(r.tolist()) for r in O.frame_tiles(grid, grid, tile, -h, -h)}
    c = {frozenset(r.tolist()) for r in O.frame_tiles(grid, grid, tile, 0, 0)}
    assert a == b and a != c


def test_whole_block_shift_only_renumbers():
    a = {frozenset(r.tolist()) for r in O.frame_tiles(32, 32, 8, 8, -16)}
    b = {frozenset(r.tolist()) for r in O.frame_tiles(32, 32, 8, 0, 0)}
    assert a == b


def test_frame_rejects_ragged_grid():
    with pytest.raises(ValueError):
        O.frame_tiles(20, 16, 8, 0, 0)


def test_pool_exact_rational_bf16():
    rng = np.random.default_rng(3)
    grid, tile, c = 16, 4, 8
    x = torch.tensor(rng.standard_normal((grid * grid, c)) * 0.5).to(torch.bfloat16).double().numpy()
    x[5, 2] *= 8.0
    sums = O.pool_sums(x, O.frame_tiles(grid, grid, tile, 2, -2))
    where = _forward_map(grid, grid, tile, 2, -2)
    exact = [[Fraction(0)] * c for _ in range(grid * grid // tile ** 2)]
    for tok, (t, _) in where.items():
        for ch in range(c):
            exact[t][ch] += Fraction(float(x[tok, ch]))
    for t in range(len(exact)):
        for ch in range(c):
            assert sums[t, ch] == float(exact[t][ch])        # bit-exact: no rounding


@pytest.mark.parametrize("grid_h,grid_w,tile,sy,sx", [(16, 16, 4, 2, 2), (32, 16, 8, -4, 4),
                                                      (32, 32, 16, 8, 8)])
def test_pool_is_mean_pool_of_rolled_grid(grid_h, grid_w, tile, sy, sx):
    rng = np.random.default_rng(7)
    c = 5
    x = rng.standard_normal((2, grid_h * grid_w, c))
    sums = O.pool_sums(x, O.frame_tiles(grid_h, grid_w, tile, sy, sx))
    g = torch.tensor(x).reshape(2, grid_h, grid_w, c).permute(0, 3, 1, 2)
    g = torch.roll(g, shifts=(sy, sx), dims=(2, 3))
    mean = F.avg_pool2d(g, tile)                                    # [2, C, ny, nx]
    ref = mean.permute(0, 2, 3, 1).reshape(2, -1, c).numpy() * tile * tile
    np.testing.assert_allclose(sums, ref, rtol=1e-12, atol=1e-12)
