"""Mask exactness through identity values.  With V the identity on the key
columns c0 .. c0 + D - 1 (V[c0 + j][j] = 1, every other entry 0), row q of
the output is P[q, c0 .. c0 + D - 1], so ceil(T / D) calls return every
attention probability of the GPU path.  A masked (query, key) pair -- an
image key outside the query block's kept tiles -- must come out exactly 0
(skipped tiles contribute nothing), and every kept probability must equal
the oracle's within the output tolerance.  Covered: the fp32 kernel, the
bf16 MFMA kernels at head_dim 64 (with and without text rows) and 128 (8x8
and 16x16 tiles), and the call with the gate fused into the attention kernel
(8x8 tiles, head_dim 64 and 128)."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import make_qkv, preset, workload_from

from _parity import gpu_desc, oracle_index, oracle_kw, to64, tol

pytestmark = pytest.mark.gpu

CASES = [
    preset("tiny"),                                                   # fp32, 4x4 tiles, keep 4 of 16
    workload_from(name="mask64", batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8,
                  gate="topk", keep=4, shift=(4, 4), seed=3),          # MFMA, D 64, keep 4 of 16
    workload_from(name="mask64_text", batch=1, heads=1, grid_h=16, grid_w=16, head_dim=64, tile=8,
                  n_text=20, gate="topk", keep=2, shift=(-4, 4), seed=5),
    workload_from(name="mask128", batch=1, heads=1, grid_h=32, grid_w=32, head_dim=128, tile=16,
                  gate="topk", keep=2, shift=(8, 8), seed=7),          # MFMA, D 128, 16x16 tiles
    workload_from(name="mask128_t8", batch=1, heads=1, grid_h=24, grid_w=32, head_dim=128, tile=8,
                  n_text=7, gate="topk", keep=3, shift=(4, -4), seed=9),   # MFMA, D 128, 8x8 tiles
]


def _gpu_probabilities(w, qg, kg, fused: bool) -> np.ndarray:
    """P [B, H, T, T] of the GPU path, assembled from identity-value calls."""
    from paper_2605_15684_amd import ssba
    b, h, t, d = qg.shape
    desc = gpu_desc(w, qg)
    p = np.zeros((b, h, t, t))
    index = None
    for c0 in range(0, t, d):
        n = min(d, t - c0)
        v = torch.zeros_like(qg)
        v[:, :, c0 + torch.arange(n, device=qg.device), torch.arange(n, device=qg.device)] = 1
        if fused:
            index, _, out = ssba.forward_topk(qg, kg, v, desc)
        else:
            if index is None:
                index, _ = ssba.build_index(qg, kg, desc)
            out = ssba.forward(qg, kg, v, index, desc)
        torch.cuda.synchronize()
        p[:, :, :, c0:c0 + n] = out[..., :n].double().cpu().numpy()
    return p, index.cpu().numpy()


@pytest.mark.parametrize("fused", [False, True], ids=["two_calls", "fused_gate"])
@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_probabilities_exact_zero_when_masked(w, fused):
    if fused and (w.dtype != "bf16" or w.tile != 8):
        pytest.skip("the fused call falls back to the two calls for this shape")
    q, k, _ = make_qkv(w)
    qg, kg = q.to("cuda"), k.to("cuda")
    p_gpu, index = _gpu_probabilities(w, qg, kg, fused)
    ref_index = oracle_index(w, q, k)
    assert np.array_equal(index, ref_index)
    kw = oracle_kw(w)
    q64, k64 = to64(q), to64(k)
    t = w.seq_len
    scale = 1.0 / np.sqrt(w.head_dim)
    for b in range(w.batch):
        for h in range(w.heads):
            rows = np.arange(t)
            mask = O.token_mask_rows(ref_index[b, h], rows, grid_h=kw["grid_h"], grid_w=kw["grid_w"],
                                     tile=kw["tile"], shift=kw["shift"], n_text=kw["n_text"])
            # the oracle's probabilities: masked softmax applied to the identity
            p_ref = O.masked_attention_rows(q64[b, h], k64[b, h], np.eye(t), mask, scale)
            g = p_gpu[b, h]
            assert np.isfinite(g).all()
            assert np.all(g[~mask] == 0.0), "a masked pair has a nonzero probability"
            assert np.abs(g[mask] - p_ref[mask]).max() <= tol(w)
            # every row still sums to one over its kept keys
            assert np.abs(g.sum(axis=1) - 1.0).max() <= (0.02 if w.dtype == "bf16" else 1e-5)
