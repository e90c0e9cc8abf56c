"""Torch-facing binding of the SSBA forward library (libssba.so).

Thin marshalling layer over the C ABI in include/ssba.h: it checks tensors,
fills the descriptor, allocates the index and scratch buffers with torch and
passes raw device pointers plus the current HIP stream.  Every step of the
computation runs in the HIP kernels; importing this module fails if the
library is not built.

Tensors are [B, H, T, D] (any strides with a unit channel stride, shared by
Q, K, V and O), T = n_text + grid_h * grid_w, text rows first.
"""
from __future__ import annotations

import math
from typing import Optional, Tuple

import torch

from . import _lib

_lib.load()   # fail loudly at import if the HIP library is missing

__all__ = ["make_desc", "desc_for", "alloc_workspace", "build_index", "forward", "forward_dense",
           "forward_topk", "forward_topk_rope", "rope_pool_keys", "forward_layers", "forward_train", "backward",
           "attention", "read_status",
           "layer_shift",
           "keep_from_rho", "SsbaError"]

SsbaError = _lib.SsbaError
_GATES = {"topk": _lib.GATE_TOPK, "window": _lib.GATE_WINDOW, "dense": _lib.GATE_DENSE,
          "topk_shared": _lib.GATE_TOPK_SHARED}
_TOPK = (_lib.GATE_TOPK, _lib.GATE_TOPK_SHARED)
_DTYPES = {torch.bfloat16: _lib.DT_BF16, torch.float32: _lib.DT_F32}


def layer_shift(layer: int, tile: int) -> Tuple[int, int]:
    """Grid offset of DiT layer `layer`: (+tile/2, +tile/2) on even layers and
    (-tile/2, -tile/2) on odd ones (Section 2.2.2; +-4 for 8x8 blocks)."""
    h = tile // 2
    return (h, h) if layer % 2 == 0 else (-h, -h)


def keep_from_rho(n_tiles: int, rho: float) -> int:
    """Key blocks kept per query block when floor(T_b * rho) are dropped
    (Section 2.2.1, Top-k Gating)."""
    return n_tiles - int(math.floor(float(n_tiles) * float(rho)))


def make_desc(*, batch: int, heads: int, head_dim: int, grid: Tuple[int, int], tile: int,
              shift: Tuple[int, int] = (0, 0), n_text: int = 0, gate: str = "topk", keep: int = 0,
              window: Tuple[int, int] = (1, 1), dtype=torch.bfloat16, scale: Optional[float] = None,
              strides: Optional[Tuple[int, int, int]] = None) -> _lib.SsbaDesc:
    d = _lib.SsbaDesc()
    d.batch, d.heads, d.head_dim = int(batch), int(heads), int(head_dim)
    d.grid_h, d.grid_w, d.tile = int(grid[0]), int(grid[1]), int(tile)
    d.shift_y, d.shift_x = int(shift[0]), int(shift[1])
    d.n_text = int(n_text)
    d.gate = _GATES[gate]
    d.keep = int(keep)
    d.win_h, d.win_w = int(window[0]), int(window[1])
    d.dtype = _DTYPES[dtype]
    d.softmax_scale = float(scale) if scale is not None else 0.0
    sb, sh, st = strides if strides is not None else (0, 0, 0)
    d.stride_b, d.stride_h, d.stride_t = int(sb), int(sh), int(st)
    return d


def desc_for(q: torch.Tensor, **kw) -> _lib.SsbaDesc:
    """Descriptor for tensors shaped like `q` ([B, H, T, D])."""
    if q.dim() != 4:
        raise ValueError("expected a [B, H, T, D] tensor")
    b, h, t, dd = q.shape
    sb, sh, st, sc = q.stride()
    if sc != 1:
        raise ValueError("channel stride must be 1")
    desc = make_desc(batch=b, heads=h, head_dim=dd, dtype=q.dtype, strides=(sb, sh, st), **kw)
    if desc.n_text + desc.grid_h * desc.grid_w != t:
        raise ValueError(f"sequence length {t} != n_text + grid_h * grid_w")
    return desc


def _check_tensors(desc, *ts):
    ref = ts[0]
    for t in ts:
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise ValueError("SSBA tensors must be GPU tensors")
        if t.device != ref.device:
            raise ValueError("all tensors must be on one device")
        if t.dtype != ref.dtype or _DTYPES.get(t.dtype) != desc.dtype:
            raise ValueError("Q, K, V and O must share the descriptor's dtype")
        if t.shape != ref.shape or t.stride() != ref.stride():
            raise ValueError("Q, K, V and O must share shape and strides")


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _check_buffer(t: torch.Tensor, what: str, dtype=None) -> None:
    """A workspace buffer must be a contiguous GPU tensor (its size is checked
    by the library, which returns SSBA_ERR_WORKSPACE when it is short)."""
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous()
            and (dtype is None or t.dtype == dtype)):
        raise ValueError(f"{what} must be a contiguous GPU tensor" + (f" of {dtype}" if dtype else ""))


def alloc_workspace(desc, device) -> Tuple[torch.Tensor, torch.Tensor]:
    """Index (int32 [B, H, T_b, 1 + T_b]) and scratch buffers for `desc`."""
    ib, sb = _lib.workspace_size(desc)
    tb = desc.grid_h * desc.grid_w // (desc.tile * desc.tile)
    index = torch.empty((desc.batch, desc.heads, tb, tb + 1), dtype=torch.int32, device=device)
    assert index.numel() * 4 == ib
    scratch = torch.empty(((sb + 7) // 8,), dtype=torch.float64, device=device)
    return index, scratch


def build_index(q, k, desc, index=None, scratch=None):
    """Gate (top-k / shared top-k / window / dense) -> index.  Returns (index, scratch)."""
    if desc.gate in _TOPK:
        _check_tensors(desc, q, k)
        dev = q.device
    else:
        dev = q.device if isinstance(q, torch.Tensor) else torch.device("cuda", torch.cuda.current_device())
    if index is None or scratch is None:
        index, scratch = alloc_workspace(desc, dev)
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    qp = q.data_ptr() if desc.gate in _TOPK else None
    kp = k.data_ptr() if desc.gate in _TOPK else None
    _lib.check(_lib.build_index(desc, qp, kp, index.data_ptr(), scratch.data_ptr(), _stream(dev),
                                _nbytes(index), _nbytes(scratch)), "ssba_build_index")
    return index, scratch


def forward(q, k, v, index, desc, out=None):
    """SSBA attention of every row (text rows included) into `out`."""
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)
    _check_tensors(desc, q, k, v, out)
    _check_buffer(index, "index", torch.int32)
    _lib.check(_lib.forward(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), index.data_ptr(),
                            out.data_ptr(), _stream(q.device), _nbytes(index)), "ssba_forward")
    return out


def forward_dense(q, k, v, desc, out=None):
    """Dense attention over all T keys, same kernel family."""
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)
    _check_tensors(desc, q, k, v, out)
    _lib.check(_lib.forward_dense(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                  _stream(q.device)), "ssba_forward_dense")
    return out


def forward_topk(q, k, v, desc, index=None, scratch=None, out=None):
    """Top-k gate and attention in one call (gate fused into the attention
    kernel where the shape allows).  Returns (index, scratch, out); index and
    scratch hold exactly what build_index would have left there."""
    if desc.gate not in _TOPK:
        raise ValueError("forward_topk needs a top-k gate")
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)
    _check_tensors(desc, q, k, v, out)
    if index is None or scratch is None:
        index, scratch = alloc_workspace(desc, q.device)
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.forward_topk(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), index.data_ptr(),
                                 scratch.data_ptr(), out.data_ptr(), _stream(q.device), _nbytes(index),
                                 _nbytes(scratch)), "ssba_forward_topk")
    return index, scratch, out


def pool_keys(k, desc, scratch):
    """The pooling launch of the fused top-k form alone (ssba_pool_keys_ex):
    writes the pooled key sums into `scratch` (from alloc_workspace)."""
    if not (isinstance(k, torch.Tensor) and k.is_cuda and k.dtype == torch.bfloat16):
        raise ValueError("k must be a bf16 GPU tensor laid out as desc says")
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.pool_keys(desc, k.data_ptr(), scratch.data_ptr(), _stream(k.device), _nbytes(scratch)),
               "ssba_pool_keys")
    return scratch


def forward_gated(q, k, v, desc, index, scratch, out):
    """The gated attention launch of the fused top-k form alone
    (ssba_forward_gated_ex): `scratch` must hold what pool_keys wrote for
    this k.  pool_keys then forward_gated is exactly forward_topk."""
    _check_tensors(desc, q, k, v, out)
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.forward_gated(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), index.data_ptr(),
                                  scratch.data_ptr(), out.data_ptr(), _stream(q.device), _nbytes(index),
                                  _nbytes(scratch)), "ssba_forward_gated")
    return index, scratch, out


def _rope_outputs(q, k, q_rope, k_rope):
    mk = lambda t, like: torch.empty_strided(like.shape, like.stride(), dtype=like.dtype, device=like.device) \
        if t is None else t
    return mk(q_rope, q), mk(k_rope, k)


def rope_pool_keys(q, k, desc, scratch, q_rope=None, k_rope=None, theta=10000.0):
    """The rotary pre-pass alone (ssba_rope_pool_keys_ex): the rotated Q and
    K (2-D axial rotary embedding of the image rows, Algorithm 1's first
    step) and the pooled sums of the rotated keys in `scratch`.  Returns
    (q_rope, k_rope)."""
    q_rope, k_rope = _rope_outputs(q, k, q_rope, k_rope)
    _check_tensors(desc, q, k, q_rope, k_rope)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.rope_pool_keys(desc, q.data_ptr(), k.data_ptr(), q_rope.data_ptr(), k_rope.data_ptr(),
                                   float(theta), scratch.data_ptr(), _stream(q.device), _nbytes(scratch)),
               "ssba_rope_pool_keys")
    return q_rope, k_rope


def forward_topk_rope(q, k, v, desc, theta=10000.0, q_rope=None, k_rope=None, index=None, scratch=None,
                      out=None):
    """Algorithm 1 in one call (ssba_forward_topk_rope_ex): rotary step,
    pooling, gate and attention.  Returns (q_rope, k_rope, index, scratch,
    out); the results equal forward_topk on (q_rope, k_rope, v)."""
    q_rope, k_rope = _rope_outputs(q, k, q_rope, k_rope)
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)
    _check_tensors(desc, q, k, v, out, q_rope, k_rope)
    ib, sb = alloc_workspace(desc, q.device) if index is None or scratch is None else (index, scratch)
    index = ib if index is None else index
    scratch = sb if scratch is None else scratch
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.forward_topk_rope(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), q_rope.data_ptr(),
                                      k_rope.data_ptr(), float(theta), index.data_ptr(), scratch.data_ptr(),
                                      out.data_ptr(), _stream(q.device), _nbytes(index), _nbytes(scratch)),
               "ssba_forward_topk_rope")
    return q_rope, k_rope, index, scratch, out


def forward_layers(layers, desc, index=None, scratch=None):
    """A stack of SSBA layers in one call (ssba_forward_layers).

    `layers`: sequence of dicts with q, k, v, out ([B, H, T, D] tensors laid
    out as `desc` says), keep (top-k gates) and optional skip.  Layer l uses
    desc's offset on even l and its negation on odd l.  Returns (index,
    scratch): per-layer slices [L, B, H, T_b, 1 + T_b] and [L, stride]."""
    n = len(layers)
    ib, sb = _lib.layers_workspace_size(desc, n)
    arr = (_lib.SsbaLayer * n)()
    dev = None
    for l, layer in enumerate(layers):
        e = arr[l]
        e.skip = 1 if layer.get("skip", False) else 0
        e.keep = int(layer.get("keep", 0))
        if e.skip:
            continue
        _check_tensors(desc, layer["q"], layer["k"], layer["v"], layer["out"])
        dev = layer["q"].device
        e.q, e.k, e.v, e.o = (layer[x].data_ptr() for x in ("q", "k", "v", "out"))
    if dev is None:
        dev = torch.device("cuda", torch.cuda.current_device())
    tb = desc.grid_h * desc.grid_w // (desc.tile * desc.tile)
    if index is None:
        index = torch.empty((n, desc.batch, desc.heads, tb, tb + 1), dtype=torch.int32, device=dev)
    if scratch is None:
        scratch = torch.empty((n, sb // n // 8), dtype=torch.float64, device=dev)
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.forward_layers(desc, arr, index.data_ptr(), scratch.data_ptr(), _stream(dev),
                                   _nbytes(index), _nbytes(scratch)), "ssba_forward_layers")
    return index, scratch


def forward_train(q, k, v, index, desc, out=None, lse=None):
    """ssba_forward that also returns the per-row log-sum-exp (fp32 [B, H, T])
    the backward needs.  Returns (out, lse)."""
    if out is None:
        out = torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device)
    if lse is None:
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    _check_tensors(desc, q, k, v, out)
    if not (lse.is_cuda and lse.dtype == torch.float32 and lse.is_contiguous() and lse.shape == q.shape[:3]):
        raise ValueError("lse must be a contiguous fp32 GPU tensor of shape [B, H, T]")
    _check_buffer(index, "index", torch.int32)
    _lib.check(_lib.forward_train(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), index.data_ptr(),
                                  out.data_ptr(), lse.data_ptr(), _stream(q.device), _nbytes(index)),
               "ssba_forward_train")
    return out, lse


def backward(q, k, v, out, dout, lse, index, desc, dq=None, dk=None, dv=None, scratch=None):
    """Gradients (dq, dk, dv) of the SSBA attention for upstream gradient
    `dout`, with the gate held fixed (ssba_backward)."""
    mk = lambda t: torch.empty_strided(q.shape, q.stride(), dtype=q.dtype, device=q.device) if t is None else t
    dq, dk, dv = mk(dq), mk(dk), mk(dv)
    _check_tensors(desc, q, k, v, out, dout, dq, dk, dv)
    if scratch is None:
        sb = _lib.backward_workspace_size(desc)
        scratch = torch.empty(((sb + 7) // 8,), dtype=torch.float64, device=q.device)
    _check_buffer(index, "index", torch.int32)
    _check_buffer(scratch, "scratch")
    _lib.check(_lib.backward(desc, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), dout.data_ptr(),
                             lse.data_ptr(), index.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                             scratch.data_ptr(), _stream(q.device), _nbytes(index), _nbytes(scratch)),
               "ssba_backward")
    return dq, dk, dv


def read_status(desc, scratch) -> int:
    """Synchronize and return SSBA_OK or SSBA_ERR_NONFINITE from the last gate."""
    _check_buffer(scratch, "scratch")
    return _lib.read_device_status(desc, scratch.data_ptr(), _stream(scratch.device), _nbytes(scratch))


def attention(q, k, v, *, grid, tile, shift=None, layer=None, rho=None, keep=None, gate="topk",
              window=None, n_text=0, scale=None, return_text=True):
    """One SSBA layer call: gate, then attention.

    `layer` selects the alternating +-tile/2 shift; `rho` is converted to the
    kept-block count.  Returns O ([B, H, T, D]) or, with return_text=False,
    only its image rows (Algorithm 1's return value).
    """
    if shift is None:
        shift = layer_shift(layer, tile) if layer is not None else (0, 0)
    tb = (grid[0] // tile) * (grid[1] // tile)
    if gate in ("topk", "topk_shared") and keep is None:
        keep = keep_from_rho(tb, 0.75 if rho is None else rho)
    desc = desc_for(q, grid=grid, tile=tile, shift=shift, n_text=n_text, gate=gate,
                    keep=keep or 0, window=window or (1, 1), scale=scale)
    if gate in ("topk", "topk_shared"):
        _, _, o = forward_topk(q, k, v, desc)
    else:
        index, _ = build_index(q, k, desc)
        o = forward(q, k, v, index, desc)
    return o if return_text else o[:, :, n_text:]
