"""Pins for the oracle's masked attention (Algorithm 1: expand the block gate
to tokens, pad text rows and columns with ones, attend).  References are the
library attention routine in fp64 with a mask enumerated by brute force,
block-diagonal and Swin-style shifted-window attention computed by reshaping,
and invariants: rows sum to one, permutation inside a block, equal outputs
for the two half-block offsets."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ssba_oracle as O


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _bruteforce_mask(idx_bh, grid_h, grid_w, tile, sy, sx, n_text):
    """Token mask from the definition, one pair at a time."""
    nx = grid_w // tile
    t = n_text + grid_h * grid_w
    kept = {i: set(idx_bh[i, 1:1 + idx_bh[i, 0]].tolist()) for i in range(idx_bh.shape[0])}

    def blk(tok):
        y, x = divmod(tok, grid_w)
        y2, x2 = (y + sy) % grid_h, (x + sx) % grid_w
        return (y2 // tile) * nx + x2 // tile

    m = np.zeros((t, t), dtype=bool)
    for a in range(t):
        for b in range(t):
            if a < n_text or b < n_text:
                m[a, b] = True
            else:
                m[a, b] = blk(b - n_text) in kept[blk(a - n_text)]
    return m


def _sdpa(q, k, v, mask=None, scale=None):
    return F.scaled_dot_product_attention(torch.tensor(q), torch.tensor(k), torch.tensor(v),
                                          attn_mask=None if mask is None else torch.tensor(mask),
                                          scale=scale).numpy()


@pytest.mark.parametrize("grid_h,grid_w,tile,shift,n_text,keep", [
    (8, 8, 4, (2, 2), 0, 1), (8, 16, 4, (-2, 2), 0, 3), (8, 8, 4, (0, 0), 5, 2),
    (16, 8, 4, (3, -1), 7, 4),
])
def test_topk_attention_matches_library_with_bruteforce_mask(grid_h, grid_w, tile, shift, n_text, keep):
    t = n_text + grid_h * grid_w
    q, k, v = (_rand((2, 2, t, 16), s) for s in (1, 2, 3))
    idx, o = O.ssba(q, k, v, grid_h=grid_h, grid_w=grid_w, tile=tile, shift=shift,
                    n_text=n_text, gate="topk", keep=keep)
    for b in range(2):
        for h in range(2):
            m = _bruteforce_mask(idx[b, h], grid_h, grid_w, tile, shift[0], shift[1], n_text)
            ref = _sdpa(q[b, h], k[b, h], v[b, h], m)
            np.testing.assert_allclose(o[b, h], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("n_text", [0, 9])
def test_dense_gate_equals_dense_attention(n_text):
    grid, tile = 16, 4
    t = n_text + grid * grid
    q, k, v = (_rand((1, 2, t, 32), s) for s in (4, 5, 6))
    _, o = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=(2, 2), n_text=n_text,
                  gate="dense")
    np.testing.assert_allclose(o, _sdpa(q, k, v), rtol=1e-12, atol=1e-12)
    # keep = T_b (rho = 0) is the same thing through the top-k gate
    _, o2 = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=(2, 2), n_text=n_text,
                   gate="topk", keep=16)
    np.testing.assert_allclose(o2, o, rtol=0, atol=0)


def _blockwise(q, k, v, grid_h, grid_w, tile):
    """Attention restricted to each tile x tile block of the grid, by reshape."""
    b, h, _, c = q.shape
    ny, nx = grid_h // tile, grid_w // tile

    def split(x):
        return (x.reshape(b, h, ny, tile, nx, tile, c).transpose(0, 1, 2, 4, 3, 5, 6)
                .reshape(b, h, ny * nx, tile * tile, c))
    o = _sdpa(split(q), split(k), split(v))
    return (o.reshape(b, h, ny, nx, tile, tile, c).transpose(0, 1, 2, 4, 3, 5, 6)
            .reshape(b, h, grid_h * grid_w, c))


def test_window_one_block_no_shift_is_block_diagonal():
    grid_h, grid_w, tile = 16, 8, 4
    q, k, v = (_rand((2, 2, grid_h * grid_w, 16), s) for s in (7, 8, 9))
    _, o = O.ssba(q, k, v, grid_h=grid_h, grid_w=grid_w, tile=tile, shift=(0, 0),
                  gate="window", window=(1, 1))
    np.testing.assert_allclose(o, _blockwise(q, k, v, grid_h, grid_w, tile), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shift", [(2, 2), (-2, -2), (1, 3)])
def test_window_one_block_shifted_is_swin_without_mask(shift):
    grid, tile, c = 16, 4, 16
    q, k, v = (_rand((1, 2, grid * grid, c), s) for s in (10, 11, 12))
    _, o = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=shift,
                  gate="window", window=(1, 1))

    def roll(x, s):
        return np.roll(x.reshape(1, 2, grid, grid, c), s, axis=(2, 3)).reshape(1, 2, grid * grid, c)
    ref = roll(_blockwise(roll(q, shift), roll(k, shift), roll(v, shift), grid, grid, tile),
               (-shift[0], -shift[1]))
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_rows_sum_to_one():
    grid, tile, n_text = 16, 4, 3
    t = n_text + grid * grid
    q, k = (_rand((1, 2, t, 8), s) for s in (13, 14))
    ones = np.ones((1, 2, t, 8))
    _, o = O.ssba(q, k, ones, grid_h=grid, grid_w=grid, tile=tile, shift=(2, 2),
                  n_text=n_text, keep=3)
    np.testing.assert_allclose(o, 1.0, rtol=0, atol=1e-14)


def test_permutation_within_a_block():
    grid, tile, sh = 16, 4, (2, 2)
    q, k, v = (_rand((1, 2, grid * grid, 16), s) for s in (15, 16, 17))
    q = torch.tensor(q).to(torch.bfloat16).double().numpy()     # exact sums -> same gate
    k = torch.tensor(k).to(torch.bfloat16).double().numpy()
    idx, o = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=sh, keep=4)
    tiles = O.frame_tiles(grid, grid, tile, *sh)
    rng = np.random.default_rng(0)
    perm = np.arange(grid * grid)
    for t in range(tiles.shape[0]):
        perm[tiles[t]] = tiles[t][rng.permutation(tile * tile)]
    idx2, o2 = O.ssba(q, k[:, :, perm], v[:, :, perm], grid_h=grid, grid_w=grid, tile=tile,
                      shift=sh, keep=4)
    assert (idx2 == idx).all()
    np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-12)
    idx3, o3 = O.ssba(q[:, :, perm], k, v, grid_h=grid, grid_w=grid, tile=tile, shift=sh, keep=4)
    assert (idx3 == idx).all()
    np.testing.assert_allclose(o3, o[:, :, perm], rtol=1e-12, atol=1e-12)


def test_half_block_offsets_give_equal_outputs():
    grid, tile = 16, 4
    q, k, v = (_rand((1, 2, grid * grid, 16), s) for s in (18, 19, 20))
    q = torch.tensor(q).to(torch.bfloat16).double().numpy()
    k = torch.tensor(k).to(torch.bfloat16).double().numpy()
    _, a = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=O.layer_shift(0, tile), keep=5)
    _, b = O.ssba(q, k, v, grid_h=grid, grid_w=grid, tile=tile, shift=O.layer_shift(1, tile), keep=5)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_explicit_scale_and_row_subset():
    grid, tile = 8, 4
    q, k, v = (_rand((1, 1, grid * grid, 8), s) for s in (21, 22, 23))
    idx = O.build_index(q, k, grid_h=grid, grid_w=grid, tile=tile, gate="dense")
    o = O.attention(q, k, v, idx, grid_h=grid, grid_w=grid, tile=tile, scale=0.37, rows=[3, 40])
    ref = _sdpa(q, k, v, scale=0.37)
    np.testing.assert_allclose(o[0, 0, [3, 40]], ref[0, 0, [3, 40]], rtol=1e-12, atol=1e-12)
    assert np.isnan(o[0, 0, 0]).all()
