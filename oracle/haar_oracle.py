"""CPU oracle for the multi-level 2-D Haar transform pair -- TEST INFRASTRUCTURE ONLY.

Plain fp64 NumPy statement of the wavelet transforms of the Tiny DWT-Distilled
VAE (Section 2.3.1, "DWT-Enhanced Architecture"): a single 2-D Haar kernel
bank {LL, HL, LH, HH} applied level after level on the encoder side (the DWT
equation, W^(l) with 4C channels at H/2^l x W/2^l), and the decoder's inverse
pyramid (the IWT equation, each level's reconstruction plus a residual).  It
exists to check the HIP path: only the tests, the package smoke check and the
benchmark's CPU baseline may import it; it shares no code with the HIP path.

Readings (each also listed in the design notes):
  * the bank is the orthonormal Haar bank; for a 2 x 2 cell with a = x[2i, 2j],
    b = x[2i, 2j+1], c = x[2i+1, 2j], d = x[2i+1, 2j+1]:
        LL = (a + b + c + d) / 2      HL = (a - b + c - d) / 2
        LH = (a + b - c - d) / 2      HH = (a - b - c + d) / 2
    (HL is high-pass along the width, LH along the height);
  * level l transforms the unrounded LL band of level l - 1 (level 0 is the
    input); level l is stored as 4C channels, channel 4 c + band with bands in
    the order LL, HL, LH, HH;
  * the inverse rebuilds LL^(l-1) = IWT(LL^(l), HL^(l), LH^(l), HH^(l)) +
    Delta^(l-1) from the coarsest level down, reading only the coarsest LL and
    every level's detail bands; Delta is optional (zero gives perfect
    reconstruction); the finest reconstruction is the output.

Pins (tests/test_oracle_haar.py): a Kronecker-product matrix statement of the
same transform, perfect reconstruction, energy preservation, constant and
ramp images, a hand-computed cell.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np

BANDS = ("LL", "HL", "LH", "HH")


def dwt_level(x: np.ndarray) -> np.ndarray:
    """One level: ``x[..., H, W]`` -> ``[..., 4, H/2, W/2]`` (bands LL, HL, LH, HH)."""
    x = np.asarray(x, dtype=np.float64)
    a = x[..., 0::2, 0::2]
    b = x[..., 0::2, 1::2]
    c = x[..., 1::2, 0::2]
    d = x[..., 1::2, 1::2]
    return np.stack([(a + b + c + d) / 2, (a - b + c - d) / 2,
                     (a + b - c - d) / 2, (a - b - c + d) / 2], axis=-3)


def iwt_level(bands: np.ndarray) -> np.ndarray:
    """Inverse of one level: ``[..., 4, h, w]`` -> ``[..., 2h, 2w]``."""
    bands = np.asarray(bands, dtype=np.float64)
    ll, hl, lh, hh = (bands[..., k, :, :] for k in range(4))
    h, w = ll.shape[-2:]
    out = np.empty(ll.shape[:-2] + (2 * h, 2 * w))
    out[..., 0::2, 0::2] = (ll + hl + lh + hh) / 2
    out[..., 0::2, 1::2] = (ll - hl + lh - hh) / 2
    out[..., 1::2, 0::2] = (ll + hl - lh - hh) / 2
    out[..., 1::2, 1::2] = (ll - hl - lh + hh) / 2
    return out


def dwt(x: np.ndarray, levels: int) -> List[np.ndarray]:
    """Multi-level transform of ``x[N, C, H, W]``.

    Returns ``levels`` arrays; entry l - 1 is W^(l) of shape
    ``[N, 4C, H/2^l, W/2^l]`` (channel 4 c + band).  Level l transforms the
    unrounded LL band of level l - 1.
    """
    x = np.asarray(x, dtype=np.float64)
    n, c = x.shape[:2]
    out = []
    ll = x
    for _ in range(levels):
        w = dwt_level(ll)                                     # [N, C, 4, h, w]
        out.append(w.reshape(n, 4 * c, w.shape[-2], w.shape[-1]))
        ll = w[:, :, 0]
    return out


def iwt(levels: Sequence[np.ndarray], residuals: Optional[Sequence[Optional[np.ndarray]]] = None
        ) -> np.ndarray:
    """Inverse pyramid.  ``levels[l-1]`` is W^(l) as returned by `dwt`; only the
    coarsest level's LL band and every level's detail bands are read.
    ``residuals[l]`` (optional, shape of LL^(l), l = 0 .. L-1) is added to the
    reconstruction of LL^(l); ``residuals[0]`` to the output."""
    n_lv = len(levels)
    n, c4 = levels[0].shape[:2]
    c = c4 // 4
    cur = np.asarray(levels[-1], np.float64).reshape(n, c, 4, *levels[-1].shape[-2:])[:, :, 0]
    for l in range(n_lv, 0, -1):
        wl = np.asarray(levels[l - 1], np.float64).reshape(n, c, 4, *levels[l - 1].shape[-2:])
        bands = np.concatenate([cur[:, :, None], wl[:, :, 1:]], axis=2)
        cur = iwt_level(bands)
        if residuals is not None and residuals[l - 1] is not None:
            cur = cur + np.asarray(residuals[l - 1], np.float64)
    return cur
