"""Pins for the oracle's attention backward (gradients of Algorithm 1's
attend step with the gate held fixed): central finite differences of the
oracle's own forward, torch autograd for the dense case and for an explicit
boolean mask, a library log-sum-exp, and a brute-force index transpose."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O

KW = dict(grid_h=4, grid_w=4, tile=2, shift=(1, 1), n_text=2)


def _tiny(seed, keep=2, gate="topk"):
    rng = np.random.default_rng(seed)
    q, k, v, g = (rng.standard_normal((1, 1, 18, 4)) for _ in range(4))
    idx = O.build_index(q, k, gate=gate, keep=keep, **KW)
    return q, k, v, g, idx


@pytest.mark.parametrize("seed,keep", [(0, 2), (1, 1), (2, 4)])
def test_gradients_match_finite_differences(seed, keep):
    q, k, v, g, idx = _tiny(seed, keep)
    dq, dk, dv, _ = O.attention_backward(q, k, v, g, idx, **KW)

    def loss(qq, kk, vv):
        return float(np.sum(O.attention(qq, kk, vv, idx, **KW) * g))

    eps = 1e-6
    rng = np.random.default_rng(seed + 10)
    for name, x, grad in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(12):
            pos = tuple(int(rng.integers(s)) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[pos] += eps
            xm[pos] -= eps
            args = {"q": (q, k, v), "k": (q, k, v), "v": (q, k, v)}[name]
            ap = [xp if a is x else a for a in args]
            am = [xm if a is x else a for a in args]
            fd = (loss(*ap) - loss(*am)) / (2 * eps)
            assert abs(fd - grad[pos]) <= 1e-6 * max(1.0, abs(fd)), (name, pos, fd, grad[pos])


def _torch_grads(q, k, v, g, mask, scale):
    qt, kt, vt = (torch.tensor(x[0, 0], dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    logits = scale * qt @ kt.T
    logits = logits.masked_fill(~torch.tensor(mask), float("-inf"))
    out = torch.softmax(logits, dim=-1) @ vt
    out.backward(torch.tensor(g[0, 0]))
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy(), torch.logsumexp(logits, -1).detach().numpy()


@pytest.mark.parametrize("gate", ["dense", "topk"])
def test_gradients_match_torch_autograd(gate):
    q, k, v, g, idx = _tiny(5, keep=2, gate=gate)
    dq, dk, dv, lse = O.attention_backward(q, k, v, g, idx, **KW)
    mask = O.token_mask_rows(idx[0, 0], np.arange(18), **KW)
    if gate == "dense":
        assert mask.all()
    tq, tk, tv, tl = _torch_grads(q, k, v, g, mask, 0.5)
    np.testing.assert_allclose(dq[0, 0], tq, atol=1e-12)
    np.testing.assert_allclose(dk[0, 0], tk, atol=1e-12)
    np.testing.assert_allclose(dv[0, 0], tv, atol=1e-12)
    np.testing.assert_allclose(lse[0, 0], tl, atol=1e-12)


def test_transpose_index_bruteforce():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((2, 2, 64, 8))
    k = rng.standard_normal((2, 2, 64, 8))
    idx = O.build_index(q, k, grid_h=8, grid_w=8, tile=2, shift=(1, 0), keep=5)
    tr = O.transpose_index(idx)
    for b in range(2):
        for h in range(2):
            for j in range(16):
                want = [i for i in range(16) if j in idx[b, h, i, 1:1 + idx[b, h, i, 0]].tolist()]
                n = tr[b, h, j, 0]
                assert n == len(want) and tr[b, h, j, 1:1 + n].tolist() == want
                assert (tr[b, h, j, 1 + n:] == -1).all()
    assert tr[..., 0].sum() == idx[..., 0].sum()


@pytest.mark.parametrize("chunk", [1, 5, 7])
def test_row_chunks_give_the_whole_rows_result(chunk):
    """Taking the query rows a few at a time changes only the order in which
    dK and dV add their row terms (fp64): the gradients agree with the
    all-rows result to rounding, and the finite-difference pins above hold
    for the chunked form through that agreement."""
    q, k, v, g, idx = _tiny(9, keep=2)
    whole = O.attention_backward(q, k, v, g, idx, **KW)
    part = O.attention_backward(q, k, v, g, idx, row_chunk=chunk, **KW)
    for a, b in zip(whole, part):
        np.testing.assert_allclose(b, a, rtol=1e-12, atol=1e-12)
