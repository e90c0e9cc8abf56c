"""Torch-facing binding of the multi-level Haar transform pair (include/ssba_haar.h).

Argument marshalling only: tensors are checked, output tensors allocated with
torch, and raw device pointers plus the current HIP stream are passed to the
HIP kernels in libssba.so.  Importing fails if the library is not built.

x: [N, C, H, W]; level l (1-based): [N, 4C, H >> l, W >> l], channel 4 c +
band with bands LL, HL, LH, HH; bf16 or fp32, contiguous.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import _lib

_lib.load()   # fail loudly at import if the HIP library is missing

__all__ = ["haar_desc", "dwt", "iwt"]

_DTYPES = {torch.bfloat16: _lib.DT_BF16, torch.float32: _lib.DT_F32}


def haar_desc(shape, levels: int, dtype) -> _lib.HaarDesc:
    d = _lib.HaarDesc()
    d.n, d.c, d.h, d.w = (int(v) for v in shape)
    d.levels = int(levels)
    d.dtype = _DTYPES[dtype]
    return d


def _check(t: torch.Tensor, shape, dtype, what: str) -> None:
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous() and t.dtype == dtype
            and tuple(t.shape) == tuple(shape)):
        raise ValueError(f"{what}: expected a contiguous {dtype} GPU tensor of shape {tuple(shape)}")


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def level_shape(x_shape, l: int):
    n, c, h, w = x_shape
    return (n, 4 * c, h >> l, w >> l)


def dwt(x: torch.Tensor, levels: int, out: Optional[Sequence[torch.Tensor]] = None) -> List[torch.Tensor]:
    """Forward multi-level transform; returns [W^(1), ..., W^(levels)]."""
    if x.dim() != 4:
        raise ValueError("expected x of shape [N, C, H, W]")
    d = haar_desc(x.shape, levels, x.dtype)
    _check(x, x.shape, x.dtype, "x")
    if out is None:
        out = [torch.empty(level_shape(x.shape, l), dtype=x.dtype, device=x.device) for l in range(1, levels + 1)]
    for l, t in enumerate(out, start=1):
        _check(t, level_shape(x.shape, l), x.dtype, f"level {l}")
    _lib.check(_lib.haar_dwt(d, x.data_ptr(), [t.data_ptr() for t in out], _stream(x.device)), "ssba_haar_dwt")
    return list(out)


def iwt(levels: Sequence[torch.Tensor], residuals: Optional[Sequence[Optional[torch.Tensor]]] = None,
        out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Inverse pyramid; residuals[l] (optional) is added to LL^(l), l = 0 the output."""
    w1 = levels[0]
    n, c4, h1, wd1 = w1.shape
    shape = (n, c4 // 4, 2 * h1, 2 * wd1)
    d = haar_desc(shape, len(levels), w1.dtype)
    for l, t in enumerate(levels, start=1):
        _check(t, level_shape(shape, l), w1.dtype, f"level {l}")
    res_ptrs = None
    if residuals is not None:
        if len(residuals) != len(levels):
            raise ValueError("one residual entry per level")
        res_ptrs = []
        for l, r in enumerate(residuals):
            if r is None:
                res_ptrs.append(None)
            else:
                _check(r, (n, c4 // 4, shape[2] >> l, shape[3] >> l), w1.dtype, f"residual {l}")
                res_ptrs.append(r.data_ptr())
    if out is None:
        out = torch.empty(shape, dtype=w1.dtype, device=w1.device)
    _check(out, shape, w1.dtype, "out")
    _lib.check(_lib.haar_iwt(d, [t.data_ptr() for t in levels], res_ptrs, out.data_ptr(), _stream(w1.device)),
               "ssba_haar_iwt")
    return out
