"""The rotary step fused into the pooling pre-pass (Algorithm 1 in full):
ssba_rope_pool_keys_ex and ssba_forward_topk_rope_ex against the oracle's
rotary step (2-D axial reading, fp64 rotation rounded to bf16) and against
the fused call on the rotated inputs.

Rotated Q and K are compared bit for bit: both sides rotate in fp64 with
every product rounded once; the device's and the host library's cos/sin
may differ in the last bit, which can change a bf16 result only when the
fp64 value lies within ~1e-16 (relative) of a rounding midpoint."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import preset
from _parity import BF16_TOL, gpu_desc, inputs, max_err, oracle_kw, sample_rows, to64

pytestmark = pytest.mark.gpu

CASES = [
    preset("grid64", heads=2, grid_h=16, grid_w=24, n_text=13, keep=5, shift=(4, 4)),
    preset("grid64", heads=3, grid_h=24, grid_w=16, n_text=0, keep=4, shift=(-4, -4), seed=3),
    preset("grid64", heads=2, head_dim=128, grid_h=32, grid_w=32, n_text=70, keep=7, shift=(4, 4), seed=4),
    preset("grid64", heads=1, grid_h=40, grid_w=48, n_text=64, keep=1, shift=(3, 5), seed=5),
]


def _oracle_rope(w, q, k, theta):
    kw = dict(grid_h=w.grid_h, grid_w=w.grid_w, n_text=w.n_text, theta=theta)
    return O.round_bf16(O.rope_2d(to64(q), **kw)), O.round_bf16(O.rope_2d(to64(k), **kw))


@pytest.mark.parametrize("theta", [10000.0, 500.0])
@pytest.mark.parametrize("w", CASES, ids=lambda w: f"{w.grid_h}x{w.grid_w}-D{w.head_dim}-t{w.n_text}")
def test_forward_topk_rope_against_oracle(w, theta):
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    qr, kr, index, _, out = ssba.forward_topk_rope(qg, kg, vg, desc, theta=theta)
    torch.cuda.synchronize()
    want_q, want_k = _oracle_rope(w, q, k, theta)
    assert np.array_equal(to64(qr), want_q)
    assert np.array_equal(to64(kr), want_k)
    want_idx = O.build_index(want_q, want_k, gate="topk", keep=w.keep, **oracle_kw(w))
    assert np.array_equal(index.cpu().numpy(), want_idx)
    heads = [(b, h) for b in range(w.batch) for h in range(w.heads)]
    rows = np.arange(w.seq_len)
    ref = O.attention(want_q, want_k, to64(v), want_idx, rows=rows, heads=heads, **oracle_kw(w))
    assert max_err(out, ref, heads, rows) <= BF16_TOL


def test_forward_topk_rope_equals_fused_call_on_rotated_inputs():
    from paper_2605_15684_amd import ssba
    w = CASES[0]
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    qr, kr, index, scratch, out = ssba.forward_topk_rope(qg, kg, vg, desc)
    idx2, scr2, out2 = ssba.forward_topk(qr, kr, vg, desc)
    torch.cuda.synchronize()
    assert torch.equal(index, idx2) and torch.equal(out, out2)
    assert ssba.read_status(desc, scratch) == 0
    # the pre-pass alone leaves the same pooled key sums as the pooling launch on the rotated keys
    _, s1 = ssba.alloc_workspace(desc, qg.device)
    _, s2 = ssba.alloc_workspace(desc, qg.device)
    s1.zero_()
    s2.zero_()
    ssba.rope_pool_keys(qg, kg, desc, s1)
    ssba.pool_keys(kr, desc, s2)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2)


def test_rope_in_place_equals_out_of_place():
    from paper_2605_15684_amd import ssba
    w = CASES[2]
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    qr, kr, idx, _, out = ssba.forward_topk_rope(qg, kg, vg, desc)
    q2, k2 = qg.clone(), kg.clone()
    qr2, kr2, idx2, _, out2 = ssba.forward_topk_rope(q2, k2, vg, desc, q_rope=q2, k_rope=k2)
    torch.cuda.synchronize()
    assert qr2.data_ptr() == q2.data_ptr()
    assert torch.equal(qr, q2) and torch.equal(kr, k2) and torch.equal(idx, idx2) and torch.equal(out, out2)


def test_forward_topk_rope_full_size_grid64():
    """All 16 heads at 64x64 tokens: rotated Q/K and the index over every
    element, the output on sampled rows of three heads."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64")
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    qr, kr, index, _, out = ssba.forward_topk_rope(qg, kg, vg, desc)
    torch.cuda.synchronize()
    want_q, want_k = _oracle_rope(w, q, k, 10000.0)
    assert np.array_equal(to64(qr), want_q) and np.array_equal(to64(kr), want_k)
    want_idx = O.build_index(want_q, want_k, gate="topk", keep=w.keep, **oracle_kw(w))
    assert np.array_equal(index.cpu().numpy(), want_idx)
    rng = np.random.default_rng(11)
    rows = sample_rows(w, rng)
    heads = [(0, 0), (0, 7), (0, 15)]
    ref = O.attention(want_q, want_k, to64(v), want_idx, rows=rows, heads=heads, **oracle_kw(w))
    assert max_err(out, ref, heads, rows) <= BF16_TOL


def test_rope_unsupported_shapes_and_bad_theta():
    from paper_2605_15684_amd import ssba, _lib
    w = preset("grid64", heads=1, grid_h=32, grid_w=32, tile=16, keep=3)
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    with pytest.raises(_lib.SsbaError):
        ssba.forward_topk_rope(qg, kg, vg, desc)          # 16x16 blocks
    w8 = w.with_(tile=8)
    desc8 = gpu_desc(w8, qg)
    with pytest.raises(_lib.SsbaError):
        ssba.forward_topk_rope(qg, kg, vg, desc8, theta=float("inf"))
