"""Seeded synthetic inputs for the SSBA forward pass (shared by the oracle
tests, the GPU parity tests and the benchmark).

This module only *produces* inputs: workload presets (shapes, gate settings,
dtypes, seeds) and a deterministic Gaussian Q/K/V generator.  It contains none
of the method's arithmetic (no frame map, pooling, affinity, gating or
attention), so the CPU oracle and the HIP path can both consume its tensors
without sharing any computation.

Stand-in data: the paper evaluates SSBA inside a trained DiT on prompt suites
(Section 4); neither the weights nor the suites are available, so Q/K/V are
seeded Gaussians with the token-grid shapes of 512/1024/2K-pixel generation
(Section 2.2: an f8 VAE plus 2x2 patchify gives one token per 16x16 pixels).

Layout: every tensor is [B, H, T, D] with T = n_text + grid_h * grid_w, text
tokens first, image tokens row-major (token id = y * grid_w + x), channels
contiguous.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import torch

__all__ = ["Workload", "PRESETS", "preset", "make_qkv", "workload_from", "heavy_key_rows",
           "LAYER_KEEP_SCHEDULE_24", "LAYER_SKIP_24"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One SSBA call: shapes, gate settings and the input recipe."""

    name: str
    batch: int
    heads: int
    grid_h: int
    grid_w: int
    head_dim: int
    tile: int
    n_text: int = 0
    dtype: str = "bf16"            # "bf16" or "f32": Q, K, V, O share it
    gate: str = "topk"             # "topk", "topk_shared", "window" or "dense"
    keep: int = 0                  # topk: key tiles kept per query tile
    window: Tuple[int, int] = (1, 1)   # window gate: window size in tiles
    shift: Tuple[int, int] = (0, 0)    # roll of the token grid (y, x)
    seed: int = 1
    sigma_img: float = 0.5         # image rows scaled by this (exact power of 2)
    heavy_key_rows: int = 0        # this many image key rows scaled by 8

    # -- derived sizes (integer bookkeeping only) --------------------------
    @property
    def t_img(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def seq_len(self) -> int:
        return self.n_text + self.t_img

    @property
    def n_tiles(self) -> int:
        return self.t_img // (self.tile * self.tile)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _p(**kw) -> Workload:
    return Workload(**kw)


# Presets.  Shapes follow the token grids of the paper's resolutions; the gate
# settings give the sparsity levels the paper reports (75% uniform, ~84%
# layer-aware average; Table 2) at 64 tiles per head.
PRESETS = {
    # 16x16 grid, 4x4 tiles (16 tiles), fp32, two heads: small enough for the
    # oracle to run in well under a second.
    "tiny": _p(name="tiny", batch=1, heads=2, grid_h=16, grid_w=16, head_dim=64,
               tile=4, dtype="f32", gate="topk", keep=4, shift=(2, 2), seed=0,
               sigma_img=1.0),
    # 1024 px class: 64x64 tokens, 8x8 tiles, keep 10 of 64 (84.375% masked).
    "grid64": _p(name="grid64", batch=1, heads=16, grid_h=64, grid_w=64,
                 head_dim=64, tile=8, gate="topk", keep=10, shift=(4, 4), seed=1),
    # grid64 plus 256 dense text tokens, batch 2, 24 heads.
    "grid64_text": _p(name="grid64_text", batch=2, heads=24, grid_h=64, grid_w=64,
                      head_dim=64, tile=8, n_text=256, gate="topk", keep=10,
                      shift=(4, 4), seed=1),
    # 2K class: 128x128 tokens, head_dim 128, 16x16 tiles, keep 7 of 64
    # (rho = 0.9), 1% of key rows scaled x8 to stress the softmax range.
    "grid128": _p(name="grid128", batch=1, heads=16, grid_h=128, grid_w=128,
                  head_dim=128, tile=16, gate="topk", keep=7, shift=(8, 8),
                  seed=1, heavy_key_rows=164),
    # Sparsity sweep base: batch 4 at the 64x64 grid.
    "sweep64": _p(name="sweep64", batch=4, heads=16, grid_h=64, grid_w=64,
                  head_dim=64, tile=8, gate="topk", keep=10, shift=(4, 4), seed=1),
}

# Sweep points over the 64-tile grid: masked fraction -> gate settings.
SWEEP_TOPK_KEEP = {0.0: 64, 0.5: 32, 0.75: 16, 0.84375: 10, 0.9375: 4}
SWEEP_WINDOW = {0.0: (8, 8), 0.5: (4, 8), 0.75: (4, 4), 0.9375: (2, 2)}


# Per-layer kept blocks (of 64) for a 24-layer stack at 8x8 blocks on the
# 64x64 grid.  The paper reports 84.16 % average sparsity for its
# layer-importance-aware scheme (Table 2) without publishing the schedule;
# this synthetic one keeps more blocks in the first and last layers and
# averages 243 / (24 * 64) kept = 84.18 % masked.
LAYER_KEEP_SCHEDULE_24 = (16, 13, 11, 10, 9, 9, 9, 9, 9, 9, 9, 9,
                          8, 9, 9, 9, 9, 9, 9, 9, 10, 11, 13, 16)
# Layers skipped by the depth-pruned stack used in the bench (every fourth
# layer from layer 3; the paper's skipped blocks come from an unpublished
# importance analysis).
LAYER_SKIP_24 = tuple(l % 4 == 3 for l in range(24))


def preset(name: str, **overrides) -> Workload:
    w = PRESETS[name]
    return w.with_(**overrides) if overrides else w


def workload_from(**kw) -> Workload:
    kw.setdefault("name", "custom")
    return Workload(**kw)


_TORCH_DTYPES = {"bf16": torch.bfloat16, "f32": torch.float32}


def heavy_key_rows(w: Workload) -> torch.Tensor:
    """Image token ids (0 .. T_img - 1) of the key rows that make_qkv scales
    by 8, sorted; empty when the workload has none.  Replays the same seeded
    draws as make_qkv."""
    if w.heavy_key_rows <= 0:
        return torch.empty(0, dtype=torch.int64)
    g = torch.Generator(device="cpu").manual_seed(int(w.seed))
    torch.randn((3, w.batch, w.heads, w.seq_len, w.head_dim), generator=g, dtype=torch.float32)
    return torch.sort(torch.randperm(w.t_img, generator=g)[: w.heavy_key_rows]).values


def make_qkv(w: Workload, device: Optional[str] = None):
    """Seeded Q, K, V for a workload, as tensors of dtype ``w.dtype``.

    Recipe: one float32 draw of shape (3, B, H, T, D) from N(0, 1) with
    ``torch.Generator().manual_seed(w.seed)``; image rows scaled by
    ``w.sigma_img``; if ``w.heavy_key_rows`` > 0, that many image key rows
    (chosen by a seeded permutation, the same rows in every head) are scaled
    by 8; then a round-to-nearest-even cast to the target dtype.  All scalings
    are powers of two, hence exact in fp32.
    """
    g = torch.Generator(device="cpu").manual_seed(int(w.seed))
    x = torch.randn((3, w.batch, w.heads, w.seq_len, w.head_dim), generator=g,
                    dtype=torch.float32)
    if w.sigma_img != 1.0:
        x[:, :, :, w.n_text:, :] *= w.sigma_img
    if w.heavy_key_rows > 0:
        rows = torch.randperm(w.t_img, generator=g)[: w.heavy_key_rows]
        x[1, :, :, w.n_text + rows, :] *= 8.0
    x = x.to(_TORCH_DTYPES[w.dtype])
    q, k, v = (x[i].contiguous() for i in range(3))
    if device is not None:
        q, k, v = q.to(device), k.to(device), v.to(device)
    return q, k, v
