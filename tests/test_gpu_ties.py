"""Ties in the top-k gate on the GPU.  Keys are made constant over each tile
of the shifted frame (so every pooled key sum of a tile is 64 times one row):
with one row for every tile all affinities of a query block are equal and
the gate must keep the lowest block ids; with tiles equal in pairs, ties
fall at the selection threshold and the lower id of a pair must win.  The
index from ssba_build_index and from the fused call must equal the
oracle's bit for bit (the order is (affinity descending, block id
ascending))."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import make_qkv, preset, workload_from

from _parity import gpu_desc, oracle_index, to64

pytestmark = pytest.mark.gpu


def _tied_keys(w, groups: int, seed: int) -> torch.Tensor:
    """K [B, H, T, D] whose image rows are equal within each tile and across
    the tiles of a group of consecutive block ids (groups = n_tiles / 2:
    tiles 2m and 2m + 1 share a row; groups = 1: one row everywhere)."""
    _, k, _ = make_qkv(w)
    tiles = O.frame_tiles(w.grid_h, w.grid_w, w.tile, *w.shift)   # [T_b, Bt^2] image token ids
    n_tiles = tiles.shape[0]
    g = torch.Generator().manual_seed(seed)
    rows = (torch.randn((w.batch, w.heads, groups, w.head_dim), generator=g) * 0.5).to(k.dtype)
    per_group = n_tiles // groups
    for t in range(n_tiles):
        k[:, :, w.n_text + torch.as_tensor(tiles[t]), :] = rows[:, :, t // per_group, None, :]
    return k


CASES = [
    (preset("grid64", heads=2), 1, 10),            # every affinity of a row equal
    (preset("grid64", heads=2), 32, 10),           # tiles equal in pairs
    (preset("grid64", heads=2), 32, 9),            # odd keep: a tied pair split at the threshold
    (preset("grid64", heads=2), 32, 11),
    (preset("grid64", heads=2), 32, 1),
    (preset("grid64", heads=2), 32, 63),
    (preset("grid64_text", batch=1, heads=2), 32, 10),
    (preset("grid64", heads=2, gate="topk_shared"), 32, 10),
    # head_dim 128 (the gate's channel loop runs 128 products), 32 blocks
    (workload_from(name="ties128", batch=1, heads=2, grid_h=32, grid_w=64, head_dim=128, tile=8,
                   gate="topk", keep=5, shift=(4, -4), seed=13), 16, 5),
    (workload_from(name="ties128", batch=1, heads=2, grid_h=32, grid_w=64, head_dim=128, tile=8,
                   gate="topk", keep=5, shift=(4, -4), seed=13), 1, 5),
]


@pytest.mark.parametrize("w,groups,keep", CASES,
                         ids=[f"{w.name}-{w.gate}-g{g}-k{kp}" for w, g, kp in CASES])
def test_ties_resolved_by_block_id(w, groups, keep):
    from paper_2605_15684_amd import ssba
    w = w.with_(keep=keep)
    q, _, v = make_qkv(w)
    k = _tied_keys(w, groups, seed=11)
    ref = oracle_index(w, q, k)
    if groups == 1:
        assert np.all(ref[..., 0] == keep)
        assert np.all(ref[..., 1:1 + keep] == np.arange(keep))
    qg, kg, vg = q.to("cuda"), k.to("cuda"), v.to("cuda")
    desc = gpu_desc(w, qg)
    index, _ = ssba.build_index(qg, kg, desc)
    torch.cuda.synchronize()
    assert np.array_equal(index.cpu().numpy(), ref)
    fused_index, _, _ = ssba.forward_topk(qg, kg, vg, desc)
    torch.cuda.synchronize()
    assert np.array_equal(fused_index.cpu().numpy(), ref)
