"""Limits and degenerate shapes on the GPU, against the oracle: the largest
block count the index supports (1024 blocks: a 128x128 grid of 4x4 tiles),
a grid that is a single block (every key kept), and a sequence shorter than
one 64-key chunk (the generic kernels)."""
import numpy as np
import pytest

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import workload_from

from _parity import (inputs, max_err, oracle_index, oracle_kw, run_gpu, sample_rows, to64, tol)

pytestmark = pytest.mark.gpu

CASES = [
    # 1024 blocks of 16 tokens, keep 100 (and 1): index bit-exact, sampled rows
    workload_from(name="max_blocks", batch=1, heads=1, grid_h=128, grid_w=128, head_dim=64, tile=4,
                  gate="topk", keep=100, shift=(2, -2), seed=21),
    workload_from(name="max_blocks_k1", batch=1, heads=1, grid_h=128, grid_w=128, head_dim=64, tile=4,
                  gate="topk", keep=1, shift=(2, 2), seed=22),
    # one block: the gate keeps it, attention is dense over the image (and text)
    workload_from(name="one_block", batch=2, heads=2, grid_h=8, grid_w=8, head_dim=64, tile=8,
                  n_text=3, gate="topk", keep=1, shift=(4, 4), seed=23),
    workload_from(name="one_block_f32", batch=1, heads=2, grid_h=16, grid_w=16, head_dim=128, tile=16,
                  gate="topk", keep=1, dtype="f32", seed=24),
    # 32 tokens in all: shorter than one 64-key chunk of the MFMA kernels
    workload_from(name="short_seq", batch=1, heads=3, grid_h=4, grid_w=8, head_dim=64, tile=4,
                  gate="topk", keep=1, shift=(1, 2), seed=25),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_limits_against_oracle(w):
    (q, k, v), (qg, kg, vg) = inputs(w)
    ref_index = oracle_index(w, q, k)
    index, out = run_gpu(w, qg, kg, vg)
    assert np.array_equal(index, ref_index)
    if w.n_tiles == 1:
        assert np.all(index[..., 0] == 1) and np.all(index[..., 1] == 0)
    rng = np.random.default_rng(w.seed)
    rows = np.arange(w.seq_len) if w.seq_len <= 4096 else sample_rows(w, rng)
    heads = [(b, h) for b in range(w.batch) for h in range(w.heads)]
    ref = O.attention(to64(q), to64(k), to64(v), ref_index, rows=rows, **oracle_kw(w))
    assert max_err(out, ref, heads, rows) <= tol(w)
