"""CPU oracle for the SSBA forward pass -- TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 NumPy implementation of Shift Sparse Block Attention as the
paper states it (Section 2.2, "Sparse Block Attention" with Eq. 1 and
Algorithm 1; Section 2.2.2, "Window Shift Strategy").  It exists to check the
HIP path: only the tests, the package smoke check and the benchmark's CPU
baseline may import it.  It shares no code with the HIP path and imports
nothing from the package.

Steps, in the paper's order and notation:

  frame     -- the token grid is rolled by the layer offset Delta (torch.roll
               semantics) and cut into Bt x Bt blocks (Section 2.2.2).
  pool      -- q_b, k_b: per-block pooled queries and keys (Eq. 1).  Kept as
               sums (mean x Bt^2, an exact power-of-two scaling for Bt in
               {4, 8, 16}), accumulated strictly in slot order.
  affinity  -- S = q_b k_b^T, T_b x T_b, each product rounded once and summed
               sequentially over channels (Section 2.2.1, "Affinity Matrix").
  gate      -- drop the k = floor(T_b * rho) smallest entries of every row of S
               (Section 2.2.1, "Top-k Gating"); ties are broken by keeping the
               lower key-block index.  Also the window gate and the dense gate
               used as controls.
  shared    -- the head-shared gate variant: S summed over heads in head
               order, one kept list per (batch, query block) for every head.
  layers    -- a stack of calls: layer l uses the offset on even l and its
               negation on odd l (Section 2.2.2), a per-layer keep (the
               layer-importance-aware sparsity of Table 2) and may be skipped
               (Section 2.1.2, Sparse-Depth Pruning).
  mask      -- expand G to token resolution, pad text rows and columns with
               ones (Section 2.2.1; Algorithm 1, expand and pad steps).
  rope      -- the rotary position embedding of the image queries and keys
               that Algorithm 1 applies first (2-D axial reading, fp64,
               rounded to bf16).
  attention -- masked softmax attention over [text; image] in fp64
               (Algorithm 1, attention step).
  backward  -- gradients of the attention with respect to Q, K and V with the
               gate held fixed (the kept lists carry no gradient), the
               per-row log-sum-exp, and the key-block view of an index.

Readings where the paper is silent (each also listed in the design notes):
k counts dropped blocks per query row; sums rather than means are ranked; ties
keep the lower index; text queries attend densely; wrapped blocks get no extra
mask; the softmax scale is 1/sqrt(head_dim); the rotary embedding is the 2-D
axial form (row in the first half of the channels, column in the second,
frequency base 10000), computed in fp64 and rounded to bf16.

Pins: every function here is checked against independent facts in
tests/test_oracle_*.py (brute-force enumeration, library routines on special
cases, constructed inputs with known answers, the paper's printed sparsity).
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence

import numpy as np

GATES = ("topk", "window", "dense", "topk_shared")


# --------------------------------------------------------------------------
# Frame (Section 2.2.2): roll the grid by Delta, then partition into blocks.
# --------------------------------------------------------------------------
def frame_tiles(grid_h: int, grid_w: int, tile: int, shift_y: int, shift_x: int) -> np.ndarray:
    """Image token ids of each block of the shifted frame.

    Returns an int64 array ``tiles[T_b, Bt*Bt]``: block t (row-major over the
    rolled grid) and slot s (row-major inside the block) hold the id
    (y * grid_w + x) of the original image token found there after
    ``np.roll(grid, (shift_y, shift_x), axis=(0, 1))``.
    """
    if grid_h % tile or grid_w % tile:
        raise ValueError("grid must be a multiple of the block size")
    ids = np.arange(grid_h * grid_w, dtype=np.int64).reshape(grid_h, grid_w)
    rolled = np.roll(ids, (shift_y, shift_x), axis=(0, 1))
    ny, nx = grid_h // tile, grid_w // tile
    return rolled.reshape(ny, tile, nx, tile).transpose(0, 2, 1, 3).reshape(ny * nx, tile * tile)


def tile_of_token(tiles: np.ndarray) -> np.ndarray:
    """Inverse of :func:`frame_tiles`: block index of every image token id."""
    out = np.empty(tiles.size, dtype=np.int64)
    out[tiles.reshape(-1)] = np.repeat(np.arange(tiles.shape[0]), tiles.shape[1])
    return out


# --------------------------------------------------------------------------
# Block compression (Eq. 1) and affinity (S = q_b k_b^T).
# --------------------------------------------------------------------------
def pool_sums(x_img: np.ndarray, tiles: np.ndarray) -> np.ndarray:
    """Per-block channel sums of image tokens, fp64, summed in slot order.

    ``x_img[..., T_img, C]`` -> ``[..., T_b, C]``.  Equals MeanPool over the
    block times Bt^2.  ``np.add.accumulate`` adds strictly left to right.
    """
    g = np.asarray(x_img, dtype=np.float64)[..., tiles, :]        # [..., T_b, Bt^2, C]
    return np.add.accumulate(g, axis=-2)[..., -1, :]


def affinity(qb: np.ndarray, kb: np.ndarray) -> np.ndarray:
    """S[..., i, j] = sum_c qb[..., i, c] * kb[..., j, c] in fp64.

    Each product is rounded once; the sum runs sequentially over c (no fused
    multiply-add, no pairwise summation).
    """
    prod = qb[..., :, None, :] * kb[..., None, :, :]               # [..., T_b, T_b, C]
    return np.add.accumulate(prod, axis=-1)[..., -1]


def shared_affinity(s: np.ndarray) -> np.ndarray:
    """Head-shared affinity: S[b] = sum over heads h of S[b, h], added in head
    order 0, 1, ..., H-1 in fp64.  ``s[B, H, T_b, T_b]`` -> ``[B, T_b, T_b]``.

    The paper's gate is stated per attention call with C channels (Section
    2.2.1); one gate shared by all heads is the variant whose score is the sum
    of the per-head scores.
    """
    return np.add.accumulate(np.asarray(s, np.float64), axis=1)[:, -1]


# --------------------------------------------------------------------------
# Gates -> canonical index lists.
# --------------------------------------------------------------------------
def keep_from_rho(n_tiles: int, rho: float) -> int:
    """Blocks kept per query block when the floor(T_b * rho) smallest are dropped."""
    return n_tiles - int(math.floor(float(n_tiles) * float(rho)))


def gate_topk_row(s_row: np.ndarray, keep: int) -> np.ndarray:
    """Kept key blocks of one query block, ascending.

    Order of preference: larger affinity first, then lower block index; the
    first ``keep`` survive, i.e. the T_b - keep smallest entries are dropped.
    """
    j = np.arange(s_row.shape[0])
    order = np.lexsort((j, -s_row))          # primary key -S (ascending), then j
    return np.sort(order[:keep])


def gate_window(ny: int, nx: int, win_h: int, win_w: int) -> list:
    """Window gate: block i sees block j iff both fall in one win_h x win_w
    window of blocks (in the shifted frame).  Returns kept lists per block."""
    out = []
    for i in range(ny * nx):
        iy, ix = divmod(i, nx)
        kept = [j for j in range(ny * nx)
                if (j // nx) // win_h == iy // win_h and (j % nx) // win_w == ix // win_w]
        out.append(np.array(kept, dtype=np.int64))
    return out


def pack_index(lists_per_bh: Sequence[Sequence[np.ndarray]], n_tiles: int) -> np.ndarray:
    """Canonical index layout: int32 [B][H][T_b][1 + T_b] = count, ascending
    kept block ids, then -1 padding."""
    b_n = len(lists_per_bh)
    h_n = len(lists_per_bh[0])
    out = np.full((b_n, h_n, n_tiles, 1 + n_tiles), -1, dtype=np.int32)
    for b in range(b_n):
        for h in range(h_n):
            for i, kept in enumerate(lists_per_bh[b][h]):
                out[b, h, i, 0] = len(kept)
                out[b, h, i, 1:1 + len(kept)] = kept
    return out


def build_index(q: np.ndarray, k: np.ndarray, *, grid_h: int, grid_w: int, tile: int,
                shift=(0, 0), n_text: int = 0, gate: str = "topk", keep: int = 0,
                window=(1, 1), return_parts: bool = False):
    """Gate of one SSBA call for every (batch, head) -> canonical index.

    q, k: [B, H, T, C] with text first.  Only image rows enter the gate.
    """
    if gate not in GATES:
        raise ValueError(gate)
    b_n, h_n = q.shape[0], q.shape[1]
    tiles = frame_tiles(grid_h, grid_w, tile, shift[0], shift[1])
    n_tiles = tiles.shape[0]
    ny, nx = grid_h // tile, grid_w // tile
    parts = {}
    if gate == "topk":
        if not 1 <= keep <= n_tiles:
            raise ValueError("keep must be in [1, T_b]")
        qb = pool_sums(q[:, :, n_text:, :], tiles)
        kb = pool_sums(k[:, :, n_text:, :], tiles)
        s = affinity(qb, kb)
        lists = [[[gate_topk_row(s[b, h, i], keep) for i in range(n_tiles)]
                  for h in range(h_n)] for b in range(b_n)]
        parts = {"qb": qb, "kb": kb, "S": s, "tiles": tiles}
    elif gate == "topk_shared":
        if not 1 <= keep <= n_tiles:
            raise ValueError("keep must be in [1, T_b]")
        qb = pool_sums(q[:, :, n_text:, :], tiles)
        kb = pool_sums(k[:, :, n_text:, :], tiles)
        s = affinity(qb, kb)
        s_shared = shared_affinity(s)
        rows = [[gate_topk_row(s_shared[b, i], keep) for i in range(n_tiles)] for b in range(b_n)]
        lists = [[rows[b] for _ in range(h_n)] for b in range(b_n)]
        parts = {"qb": qb, "kb": kb, "S": s, "S_shared": s_shared, "tiles": tiles}
    elif gate == "window":
        wl = gate_window(ny, nx, window[0], window[1])
        lists = [[wl for _ in range(h_n)] for _ in range(b_n)]
    else:
        full = np.arange(n_tiles, dtype=np.int64)
        lists = [[[full] * n_tiles for _ in range(h_n)] for _ in range(b_n)]
    idx = pack_index(lists, n_tiles)
    return (idx, parts) if return_parts else idx


# --------------------------------------------------------------------------
# Token mask and masked softmax attention (Algorithm 1, expand/pad/attend).
# --------------------------------------------------------------------------
def token_mask_rows(index_bh: np.ndarray, rows: np.ndarray, *, grid_h: int, grid_w: int,
                    tile: int, shift=(0, 0), n_text: int = 0) -> np.ndarray:
    """Boolean mask M[rows, 0:T] for one (batch, head).

    A text query or a text key is always visible; an image query in block i
    sees an image key in block j iff j is in the kept list of i.
    """
    tiles = frame_tiles(grid_h, grid_w, tile, shift[0], shift[1])
    n_tiles = tiles.shape[0]
    t_img = grid_h * grid_w
    tile_of = tile_of_token(tiles)
    g = np.zeros((n_tiles, n_tiles), dtype=bool)
    for i in range(n_tiles):
        cnt = int(index_bh[i, 0])
        g[i, index_bh[i, 1:1 + cnt]] = True
    rows = np.asarray(rows, dtype=np.int64)
    m = np.ones((rows.size, n_text + t_img), dtype=bool)
    img = rows >= n_text
    if np.any(img):
        qt = tile_of[rows[img] - n_text]
        m[np.nonzero(img)[0][:, None], n_text + np.arange(t_img)[None, :]] = g[qt][:, tile_of]
    return m


def masked_attention_rows(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray,
                          mask_rows: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * q k^T with masked logits at -inf) v, fp64, by rows."""
    logits = scale * (np.asarray(q_rows, np.float64) @ np.asarray(k, np.float64).T)
    logits = np.where(mask_rows, logits, -np.inf)
    m = logits.max(axis=-1, keepdims=True)
    p = np.exp(logits - m)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ np.asarray(v, np.float64)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, index: np.ndarray, *,
              grid_h: int, grid_w: int, tile: int, shift=(0, 0), n_text: int = 0,
              scale: Optional[float] = None, rows: Optional[Iterable[int]] = None,
              heads: Optional[Iterable] = None, chunk: Optional[int] = None) -> np.ndarray:
    """SSBA output for every (batch, head), fp64.

    q, k, v: [B, H, T, C]; index: canonical int32 [B, H, T_b, 1 + T_b].
    ``rows`` restricts the query rows computed (others are left NaN);
    ``heads`` restricts (b, h) pairs likewise.  Returns [B, H, T, C].
    """
    b_n, h_n, t, c = q.shape
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(c)
    out = np.full((b_n, h_n, t, c), np.nan, dtype=np.float64)
    all_rows = np.arange(t) if rows is None else np.asarray(list(rows), dtype=np.int64)
    pairs = [(b, h) for b in range(b_n) for h in range(h_n)] if heads is None else list(heads)
    step = chunk or max(1, tile * tile)
    for b, h in pairs:
        kk = np.asarray(k[b, h], np.float64)
        vv = np.asarray(v[b, h], np.float64)
        for s0 in range(0, all_rows.size, step):
            r = all_rows[s0:s0 + step]
            mrows = token_mask_rows(index[b, h], r, grid_h=grid_h, grid_w=grid_w,
                                    tile=tile, shift=shift, n_text=n_text)
            out[b, h, r] = masked_attention_rows(np.asarray(q[b, h, r], np.float64), kk, vv,
                                                 mrows, scale)
    return out


def ssba(q, k, v, *, grid_h, grid_w, tile, shift=(0, 0), n_text=0, gate="topk", keep=0,
         window=(1, 1), scale=None):
    """Index and output of one SSBA call (all rows, all heads)."""
    q64, k64, v64 = (np.asarray(a, np.float64) for a in (q, k, v))
    idx = build_index(q64, k64, grid_h=grid_h, grid_w=grid_w, tile=tile, shift=shift,
                      n_text=n_text, gate=gate, keep=keep, window=window)
    o = attention(q64, k64, v64, idx, grid_h=grid_h, grid_w=grid_w, tile=tile, shift=shift,
                  n_text=n_text, scale=scale)
    return idx, o


# --------------------------------------------------------------------------
# Rotary position embedding of the image queries and keys (Algorithm 1,
# first step), applied before pooling.  The paper names the step but not the
# variant; the reading (listed in the design notes) is the 2-D axial form:
# channels [0, D/2) rotate with the token's row y, channels [D/2, D) with its
# column x (positions in the unshifted image grid); inside a half, pair i is
# channels (2i, 2i + 1) of that half, turned by the angle
# pos * theta**(-i / (D/4)).  Text tokens are not rotated.  The rotation runs
# in fp64 with every product rounded once (no fused multiply-add) and the
# results are rounded to bf16 (round to nearest even), the precision the
# attention then reads.
# --------------------------------------------------------------------------
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value (8 significant bits,
    ties to even), directly from fp64 (no intermediate fp32 rounding)."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)                        # x = m * 2**e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)   # np.rint rounds half to even


def rope_angles(pos: np.ndarray, n_pairs: int, theta: float) -> np.ndarray:
    """Angles [len(pos), n_pairs]: pos * theta**(-i / n_pairs), fp64."""
    inv = np.array([theta ** (-i / n_pairs) for i in range(n_pairs)], np.float64)
    return np.asarray(pos, np.float64)[:, None] * inv[None, :]


def rope_2d(x: np.ndarray, *, grid_h: int, grid_w: int, n_text: int = 0,
            theta: float = 10000.0) -> np.ndarray:
    """The rotated copy of x [..., T, D] (fp64, not rounded; text rows and
    every channel of them unchanged)."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    if d % 4:
        raise ValueError("head_dim must be a multiple of 4")
    half, n_pairs = d // 2, d // 4
    ids = np.arange(grid_h * grid_w)
    out = x.copy()
    for axis_pos, c0 in ((ids // grid_w, 0), (ids % grid_w, half)):
        ang = rope_angles(axis_pos, n_pairs, theta)             # [T_img, n_pairs]
        cos, sin = np.cos(ang), np.sin(ang)
        a = x[..., n_text:, c0:c0 + half:2]                     # even channels of the half
        b = x[..., n_text:, c0 + 1:c0 + half:2]                 # odd channels
        out[..., n_text:, c0:c0 + half:2] = a * cos - b * sin
        out[..., n_text:, c0 + 1:c0 + half:2] = a * sin + b * cos
    return out


def ssba_rope(q, k, v, *, grid_h, grid_w, tile, shift=(0, 0), n_text=0, gate="topk", keep=0,
              window=(1, 1), scale=None, theta=10000.0):
    """One SSBA call with the rotary step first: the rotated Q and K
    (rounded to bf16), then index and output on them.  Returns
    (q_rope, k_rope, index, out)."""
    kw = dict(grid_h=grid_h, grid_w=grid_w, n_text=n_text, theta=theta)
    qr = round_bf16(rope_2d(q, **kw))
    kr = round_bf16(rope_2d(k, **kw))
    idx, o = ssba(qr, kr, v, grid_h=grid_h, grid_w=grid_w, tile=tile, shift=shift, n_text=n_text,
                  gate=gate, keep=keep, window=window, scale=scale)
    return qr, kr, idx, o


def layer_shift(layer: int, tile: int):
    """Offset of layer l: (Bt/2, Bt/2) on even layers, (-Bt/2, -Bt/2) on odd
    layers (Section 2.2.2, with Bt/2 = 4 for the paper's 8x8 blocks)."""
    h = tile // 2
    return (h, h) if layer % 2 == 0 else (-h, -h)


def ssba_layers(layers, *, grid_h, grid_w, tile, shift=None, n_text=0, gate="topk",
                window=(1, 1), scale=None):
    """A stack of SSBA calls, one per layer (Section 2.2.2 alternation; the
    per-layer sparsity of the layer-importance-aware scheme; skipped layers of
    the depth-pruned model).

    ``layers``: sequence of dicts with ``q``, ``k``, ``v`` ([B, H, T, C]),
    ``keep`` (top-k gates) and optional ``skip``.  Layer l uses ``shift`` on
    even l and its negation on odd l (default: (Bt/2, Bt/2), the paper's
    rule).  Returns per layer (index, output), or None for a skipped layer.
    """
    base = (tile // 2, tile // 2) if shift is None else tuple(shift)
    out = []
    for l, layer in enumerate(layers):
        if layer.get("skip", False):
            out.append(None)
            continue
        sh = base if l % 2 == 0 else (-base[0], -base[1])
        out.append(ssba(layer["q"], layer["k"], layer["v"], grid_h=grid_h, grid_w=grid_w,
                        tile=tile, shift=sh, n_text=n_text, gate=gate,
                        keep=layer.get("keep", 0), window=window, scale=scale))
    return out


# --------------------------------------------------------------------------
# Backward pass of the attend step (gradients of Algorithm 1's attention
# with the gate held fixed: the kept lists carry no gradient).
# --------------------------------------------------------------------------
def transpose_index(index: np.ndarray) -> np.ndarray:
    """Key-block view of an index: entry [b, h, j] lists, ascending, the query
    blocks i whose kept list holds j (same canonical layout: count, ids, -1)."""
    b_n, h_n, tb = index.shape[:3]
    lists = []
    for b in range(b_n):
        per_h = []
        for h in range(h_n):
            seen = [[] for _ in range(tb)]
            for i in range(tb):
                for j in index[b, h, i, 1:1 + int(index[b, h, i, 0])]:
                    seen[int(j)].append(i)
            per_h.append([np.array(s, dtype=np.int64) for s in seen])
        lists.append(per_h)
    return pack_index(lists, tb)


def attention_backward(q, k, v, dout, index, *, grid_h, grid_w, tile, shift=(0, 0), n_text=0,
                       scale=None, heads=None, row_chunk=None):
    """Gradients of the SSBA attention output with respect to Q, K and V, fp64.

    With P = softmax(scale Q K^T + mask) over the token mask of the index
    (text rows and columns visible), and the upstream gradient dO:
      dV = P^T dO,  dP = dO V^T,  dS = P * (dP - rowsum(P * dP)),
      dQ = scale dS K,  dK = scale dS^T Q;
    also the natural-log log-sum-exp of each row's masked scaled logits.
    Returns (dq, dk, dv, lse); pairs outside ``heads`` are left NaN.

    ``row_chunk`` bounds memory at large T: the query rows are taken that
    many at a time (P, dP and dS of a row need only that row), and their
    terms of dV and dK are added up over the chunks.
    """
    b_n, h_n, t, c = q.shape
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(c)
    dq = np.full(q.shape, np.nan)
    dk = np.full(q.shape, np.nan)
    dv = np.full(q.shape, np.nan)
    lse = np.full((b_n, h_n, t), np.nan)
    pairs = [(b, h) for b in range(b_n) for h in range(h_n)] if heads is None else list(heads)
    step = t if not row_chunk else int(row_chunk)
    for b, h in pairs:
        qq, kk, vv, gg = (np.asarray(x[b, h], np.float64) for x in (q, k, v, dout))
        dk_bh = np.zeros((t, c))
        dv_bh = np.zeros((t, c))
        for r0 in range(0, t, step):
            rows = np.arange(r0, min(r0 + step, t))
            mask = token_mask_rows(index[b, h], rows, grid_h=grid_h, grid_w=grid_w, tile=tile,
                                   shift=shift, n_text=n_text)
            logits = np.where(mask, scale * (qq[rows] @ kk.T), -np.inf)
            m = logits.max(axis=-1, keepdims=True)
            e = np.exp(logits - m)
            s = e.sum(axis=-1, keepdims=True)
            p = e / s
            lse[b, h, rows] = (m + np.log(s))[:, 0]
            dp = gg[rows] @ vv.T
            ds = p * (dp - np.sum(p * dp, axis=-1, keepdims=True))
            dv_bh += p.T @ gg[rows]
            dq[b, h, rows] = scale * (ds @ kk)
            dk_bh += scale * (ds.T @ qq[rows])
        dk[b, h] = dk_bh
        dv[b, h] = dv_bh
    return dq, dk, dv, lse
