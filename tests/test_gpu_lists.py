"""Forward parity on index lists of different lengths.  The gates produce
lists of one length (top-k) or of lengths fixed by the frame (window), but
the attention calls take any index whose counts lie in 0..T_b and whose ids
lie in 0..T_b-1.  Here the oracle's own top-k lists are cut to different
lengths on the host and given to both sides, so the kernels' per-block
chunk plans are uneven; every row is compared with the oracle (2e-2 max-abs
for bf16 inputs, 1e-5 for fp32).

A query block whose list is empty sees only the text keys; with no text
tokens it sees no key at all.  The oracle leaves such a row undefined (a
softmax over an empty set); the library writes zeros there, which
test_rows_without_visible_keys_are_zero checks on the GPU alone."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import preset, workload_from

from _parity import gpu_desc, inputs, oracle_index, oracle_kw, to64, tol

pytestmark = pytest.mark.gpu

CASES = [
    preset("tiny", n_text=9, heads=1),                                                # fp32 kernel
    workload_from(batch=1, heads=2, grid_h=16, grid_w=16, head_dim=64, tile=4, keep=5, shift=(2, 2),
                  n_text=11),                                                         # bf16, 4x4 blocks
    workload_from(batch=2, heads=1, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=6, shift=(4, 4),
                  n_text=20),                                                         # MFMA, 8x8, text
    workload_from(batch=1, heads=2, grid_h=48, grid_w=40, head_dim=128, tile=8, keep=7, shift=(3, 5)),
    workload_from(batch=1, heads=2, grid_h=48, grid_w=64, head_dim=128, tile=16, keep=5, shift=(-8, 5),
                  n_text=13),                                                         # MFMA, 16x16
]


def _ids(w):
    return f"{w.dtype}-{w.grid_h}x{w.grid_w}-D{w.head_dim}-b{w.tile}-k{w.keep}-t{w.n_text}"


def _cut(idx: np.ndarray, w, allow_empty: bool) -> np.ndarray:
    """Query block i keeps the first i mod (keep + 1) entries of its list
    (allow_empty) or the first 1 + i mod keep."""
    out = idx.copy()
    tb = w.n_tiles
    i = np.arange(tb)[None, :]
    out.reshape(-1, tb, tb + 1)[:, :, 0] = i % (w.keep + 1) if allow_empty else 1 + i % w.keep
    return out


@pytest.mark.parametrize("w", CASES, ids=_ids)
def test_forward_ragged_lists_against_oracle(w):
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    idx = _cut(oracle_index(w, q, k), w, allow_empty=w.n_text > 0)
    out = ssba.forward(qg, kg, vg, torch.from_numpy(idx).to("cuda"), gpu_desc(w, qg))
    torch.cuda.synchronize()
    ref = O.attention(to64(q), to64(k), to64(v), idx, **oracle_kw(w))
    got = out.float().cpu().double().numpy()
    assert np.isfinite(got).all()
    err = float(np.abs(got - ref).max())
    print(f"{_ids(w)}: max-abs {err:.3e}")
    assert err <= tol(w), f"max-abs {err:.3e}"


@pytest.mark.parametrize("w", [CASES[3], CASES[1].with_(n_text=0), preset("tiny", heads=1)], ids=_ids)
def test_rows_without_visible_keys_are_zero(w):
    """No text tokens and every third list empty: the rows of the empty
    blocks are exactly zero; every other row matches the oracle."""
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    idx = oracle_index(w, q, k).copy()
    tb = w.n_tiles
    lists = idx.reshape(-1, tb, tb + 1)
    empty = np.arange(tb) % 3 == 0
    lists[:, empty, 0] = 0
    out = ssba.forward(qg, kg, vg, torch.from_numpy(idx).to("cuda"), gpu_desc(w, qg))
    torch.cuda.synchronize()
    got = out.float().cpu().double().numpy()
    frame = O.frame_tiles(w.grid_h, w.grid_w, w.tile, w.shift[0], w.shift[1])   # [T_b, tile^2] token ids
    empty_rows = w.n_text + frame[empty].reshape(-1)
    assert (got[:, :, empty_rows] == 0).all()
    with np.errstate(invalid="ignore"):   # the empty rows: a softmax over no logits
        ref = O.attention(to64(q), to64(k), to64(v), idx, **oracle_kw(w))
    keep_rows = np.setdiff1d(np.arange(w.seq_len), empty_rows)
    assert np.isfinite(ref[:, :, keep_rows]).all()
    err = float(np.abs(got[:, :, keep_rows] - ref[:, :, keep_rows]).max())
    assert err <= tol(w), f"max-abs {err:.3e}"
