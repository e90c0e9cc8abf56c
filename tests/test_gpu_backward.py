"""GPU parity of the SSBA backward (gradients of the attend step with the gate
held fixed) and of the training forward's log-sum-exp, through the C ABI,
against the fp64 oracle.

Tolerance: for each gradient tensor, max |got - ref| <= GRAD_REL * max |ref|.
The kernels round P and dS to bf16 before their products and score with
Q scale log2(e) rounded to bf16 (each 2^-9 relative), and round the result to
bf16 (2^-9): a term carries at most about 3 * 2^-9 = 0.6 % relative error and
the sums do not amplify it, so 1 % of the tensor's scale bounds the result
(measured: at most 0.6 %).  The log-sum-exp of a row: its probabilities are
summed after rounding to bf16 (2^-9 relative, at most LSE_TOL = 0.002 in log
units), and each logit carries the rounding of Q scale log2(e) to bf16, at
most 2^-9 scale sum_c |q_c k_c| for key k; the log-sum-exp is a
probability-weighted mean of its logits' errors, so a row's bound is LSE_TOL
plus 2^-9 scale max over the row's visible keys of sum_c |q_c k_c|."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import preset, workload_from
from tests._parity import gpu_desc, inputs, oracle_index, oracle_kw, to64

pytestmark = pytest.mark.gpu

GRAD_REL = 1e-2
LSE_TOL = 2e-3


def _dout(w, seed=77):
    g = torch.Generator(device="cpu").manual_seed(seed)
    d = torch.randn((w.batch, w.heads, w.seq_len, w.head_dim), generator=g, dtype=torch.float32)
    return d.to(torch.bfloat16)


def _lse_bound(w, q, k, idx, heads, chunk=1024):
    """Per-row log-sum-exp bound (see the module docstring) for `heads`."""
    kw = oracle_kw(w)
    scale = 1.0 / np.sqrt(w.head_dim)
    out = {}
    for b, h in heads:
        qa, ka = np.abs(to64(q[b, h])), np.abs(to64(k[b, h]))
        bound = np.empty(w.seq_len)
        for r0 in range(0, w.seq_len, chunk):
            rows = np.arange(r0, min(r0 + chunk, w.seq_len))
            mask = O.token_mask_rows(idx[b, h], rows, **kw)
            mag = np.where(mask, qa[rows] @ ka.T, 0.0).max(axis=-1)
            bound[rows] = LSE_TOL + 2.0 ** -9 * scale * mag
        out[(b, h)] = bound
    return out


def _run(w, heads=None, row_chunk=None):
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, _ = ssba.build_index(qg, kg, desc)
    out, lse = ssba.forward_train(qg, kg, vg, index, desc)
    dout = _dout(w)
    dq, dk, dv = ssba.backward(qg, kg, vg, out, dout.to("cuda"), lse, index, desc)
    torch.cuda.synchronize()
    # The reference gradients use the oracle's own gate: the GPU index must
    # equal it bit for bit first, so a wrong gate cannot pass on both sides.
    want_idx = oracle_index(w, q, k)
    assert np.array_equal(index.cpu().numpy(), want_idx), "GPU index differs from the oracle's"
    ref = O.attention_backward(to64(q), to64(k), to64(v), to64(dout), want_idx,
                               heads=heads, row_chunk=row_chunk, **oracle_kw(w))
    pairs = heads or [(b, h) for b in range(w.batch) for h in range(w.heads)]
    return (dq, dk, dv, lse), ref + (_lse_bound(w, q, k, want_idx, pairs),)


def _check(got, ref, heads):
    errs, bad = {}, []
    for name, g, r in zip(("dq", "dk", "dv"), got[:3], ref[:3]):
        gg = g.float().cpu().double().numpy()
        for b, h in heads:
            assert np.isfinite(gg[b, h]).all()
            e = float(np.abs(gg[b, h] - r[b, h]).max())
            scale = float(np.abs(r[b, h]).max())
            errs[name] = max(errs.get(name, 0.0), e / scale)
            if e > GRAD_REL * scale:
                bad.append(f"{name} ({b},{h}): max-abs {e:.3e} vs scale {scale:.3e}")
    lg = got[3].cpu().double().numpy()
    le = max(float(np.abs(lg[b, h] - ref[3][b, h]).max()) for b, h in heads)
    over = max(float((np.abs(lg[b, h] - ref[3][b, h]) / ref[4][(b, h)]).max()) for b, h in heads)
    print(f"relative errors {errs}, lse max-abs {le:.2e}, largest share of its row bound {over:.3f}")
    assert not bad, "; ".join(bad)
    assert over <= 1.0, f"lse beyond its row bound (max-abs {le:.3e})"


CASES = [
    # one and two blocks per head (the key-side order over a single block)
    workload_from(batch=1, heads=2, grid_h=8, grid_w=8, head_dim=64, tile=8, keep=1, shift=(4, 4)),
    workload_from(batch=2, heads=1, grid_h=8, grid_w=16, head_dim=128, tile=8, keep=1, shift=(-4, 4), n_text=5),
    workload_from(batch=1, heads=2, grid_h=16, grid_w=16, head_dim=64, tile=8, keep=2, shift=(4, 4)),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=5, shift=(-4, -4), n_text=13),
    workload_from(batch=2, heads=1, grid_h=48, grid_w=40, head_dim=64, tile=8, keep=7, shift=(3, 5), n_text=77),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=128, tile=8, keep=6, shift=(4, 4), n_text=20),
    workload_from(batch=1, heads=1, grid_h=24, grid_w=24, head_dim=128, tile=8, keep=9, shift=(0, 0)),
    workload_from(batch=1, heads=2, grid_h=16, grid_w=16, head_dim=64, tile=8, keep=4, gate="dense"),
    # 16x16 blocks: each block is four 64-row chunks
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=16, keep=2, shift=(8, 8)),
    workload_from(batch=1, heads=2, grid_h=48, grid_w=64, head_dim=128, tile=16, keep=3, shift=(-8, 5),
                  n_text=13),
    workload_from(batch=2, heads=1, grid_h=64, grid_w=48, head_dim=64, tile=16, keep=5, shift=(3, -7),
                  n_text=77),
    workload_from(batch=1, heads=1, grid_h=32, grid_w=32, head_dim=128, tile=16, keep=4, gate="dense"),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: f"{w.grid_h}x{w.grid_w}-D{w.head_dim}-t{w.n_text}-k{w.keep}-{w.gate}")
def test_backward_small_against_oracle(w):
    got, ref = _run(w)
    _check(got, ref, [(b, h) for b in range(w.batch) for h in range(w.heads)])


RAGGED = [
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=6, shift=(4, 4), n_text=20),
    workload_from(batch=2, heads=1, grid_h=48, grid_w=40, head_dim=128, tile=8, keep=7, shift=(3, 5)),
    workload_from(batch=1, heads=2, grid_h=48, grid_w=64, head_dim=128, tile=16, keep=5, shift=(-8, 5),
                  n_text=13),
]


@pytest.mark.parametrize("w", RAGGED, ids=lambda w: f"{w.grid_h}x{w.grid_w}-D{w.head_dim}-b{w.tile}-t{w.n_text}")
def test_backward_ragged_lists_against_oracle(w):
    """Lists of different lengths (query block i keeps the first 1 + (i mod
    keep) blocks of its top-k list, so the key blocks are kept unevenly and
    the key side's longest-first order differs from block order): the
    training forward and the backward on that index, on every row, against
    the oracle on the same index."""
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    idx = oracle_index(w, q, k).copy()
    tb = w.n_tiles
    lists = idx.reshape(-1, tb, tb + 1)
    lists[:, :, 0] = 1 + np.arange(tb)[None, :] % w.keep
    index = torch.from_numpy(idx).to("cuda")
    out, lse = ssba.forward_train(qg, kg, vg, index, desc)
    dout = _dout(w)
    dq, dk, dv = ssba.backward(qg, kg, vg, out, dout.to("cuda"), lse, index, desc)
    torch.cuda.synchronize()
    ref = O.attention_backward(to64(q), to64(k), to64(v), to64(dout), idx, **oracle_kw(w))
    heads = [(b, h) for b in range(w.batch) for h in range(w.heads)]
    _check((dq, dk, dv, lse), ref + (_lse_bound(w, q, k, idx, heads),), heads)


def test_backward_full_size_sampled_heads():
    w = preset("grid64")
    heads = [(0, 0), (0, 7), (0, 15)]
    got, ref = _run(w, heads=heads)
    _check(got, ref, heads)


def test_backward_grid128_full_size_sampled_head():
    """The 128x128-token grid with 16x16 blocks and head_dim 128 (keep 7 of
    64), one head against the oracle (its rows taken 1024 at a time)."""
    w = preset("grid128")
    heads = [(0, 9)]
    got, ref = _run(w, heads=heads, row_chunk=1024)
    _check(got, ref, heads)


def test_backward_text_full_size_sampled_heads():
    # 16 heads: two per XCD, so the key side's rank-major numbering
    # interleaves heads, after the text groups.
    w = preset("grid64_text", batch=1, heads=16)
    heads = [(0, 0), (0, 9)]
    got, ref = _run(w, heads=heads)
    _check(got, ref, heads)


def test_zero_upstream_gradient_gives_zero_and_is_deterministic():
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2)
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, _ = ssba.build_index(qg, kg, desc)
    out, lse = ssba.forward_train(qg, kg, vg, index, desc)
    zero = torch.zeros_like(qg)
    dq, dk, dv = ssba.backward(qg, kg, vg, out, zero, lse, index, desc)
    torch.cuda.synchronize()
    assert bool((dq == 0).all() and (dk == 0).all() and (dv == 0).all())
    dout = _dout(w).to("cuda")
    a = ssba.backward(qg, kg, vg, out, dout, lse, index, desc)
    b = ssba.backward(qg, kg, vg, out, dout, lse, index, desc)
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(a, b))


def test_forward_train_output_equals_forward():
    from paper_2605_15684_amd import ssba
    w = preset("grid64_text", batch=1, heads=2)
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, _ = ssba.build_index(qg, kg, desc)
    o1 = ssba.forward(qg, kg, vg, index, desc)
    o2, _ = ssba.forward_train(qg, kg, vg, index, desc)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def _key_order_region(desc_w, scratch, tb):
    """The backward scratch's key-order region (int32 [B][H][T_b]), located by
    the layout ssba_backward_workspace_size documents."""
    up = lambda x: (x + 255) // 256 * 256
    bh = desc_w.batch * desc_w.heads
    off = 2 * up(4 * bh * desc_w.seq_len) + up(8 * bh * tb)
    raw = scratch.view(torch.uint8)[off:off + 4 * bh * tb].cpu()
    return raw.view(torch.int32).numpy().reshape(bh, tb)


@pytest.mark.parametrize("w,truncate", [
    (preset("grid64", heads=2), False),
    (preset("grid64", heads=2), True),
    (workload_from(batch=2, heads=1, grid_h=64, grid_w=48, head_dim=64, tile=16, keep=5, shift=(3, -7),
                   n_text=77), True),
], ids=["grid64", "grid64-ragged-lists", "16x16-text-ragged-lists"])
def test_key_side_order_is_longest_first(w, truncate):
    """The key-side kernel takes each head's key blocks in descending order of
    the number of lists that keep them, ties by block id; the order is left
    in the scratch.  With ragged lists (list i cut to 1 + i mod keep
    entries) the counts see only each list's first n entries.  A second run
    on a fresh scratch gives the same gradients."""
    from paper_2605_15684_amd import _lib, ssba
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, _ = ssba.build_index(qg, kg, desc)
    tb = (w.grid_h // w.tile) * (w.grid_w // w.tile)
    if truncate:
        host = index.cpu().numpy().reshape(-1, tb, tb + 1).copy()
        host[:, :, 0] = 1 + np.arange(tb)[None, :] % w.keep
        index = torch.from_numpy(host.reshape(index.shape)).to("cuda")
    out, lse = ssba.forward_train(qg, kg, vg, index, desc)
    dout = _dout(w).to("cuda")
    sb = _lib.backward_workspace_size(desc)
    scratch = torch.full(((sb + 7) // 8,), -1.0, dtype=torch.float64, device="cuda")
    first = ssba.backward(qg, kg, vg, out, dout, lse, index, desc, scratch=scratch)
    torch.cuda.synchronize()
    got = _key_order_region(w, scratch, tb)
    lists = index.cpu().numpy().reshape(-1, tb, tb + 1)
    for bh in range(lists.shape[0]):
        cnt = np.zeros(tb, dtype=np.int64)
        for i in range(tb):
            n = min(max(int(lists[bh, i, 0]), 0), tb)
            np.add.at(cnt, lists[bh, i, 1:1 + n], 1)
        want = sorted(range(tb), key=lambda j: (-cnt[j], j))
        assert got[bh].tolist() == want, f"head {bh}"
    again = ssba.backward(qg, kg, vg, out, dout, lse, index, desc)
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(first, again))
