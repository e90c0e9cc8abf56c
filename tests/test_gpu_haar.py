"""GPU parity of the multi-level Haar transform pair (Section 2.3.1, the DWT
and IWT equations) against the fp64 oracle, through the C ABI.

Tolerances: fp32 tensors max-abs 1e-5; bf16 tensors one bf16 rounding of the
fp64 value (relative 2^-8) plus 1e-6 -- the kernels compute in fp32 and round
each stored value once."""
import numpy as np
import pytest
import torch

from oracle import haar_oracle as H

pytestmark = pytest.mark.gpu


def _inputs(shape, dtype, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn(shape, generator=g, dtype=torch.float32).to(dtype)
    return x, x.to("cuda")


def _close(got: torch.Tensor, ref: np.ndarray, dtype) -> float:
    g = got.detach().float().cpu().double().numpy()
    err = np.abs(g - ref)
    if dtype == torch.float32:
        assert err.max() <= 1e-5, err.max()
    else:
        assert (err <= 2.0 ** -8 * np.abs(ref) + 1e-6).all(), float((err - 2.0 ** -8 * np.abs(ref)).max())
    return float(err.max())


CASES = [((2, 3, 16, 24), 1), ((2, 3, 16, 24), 2), ((2, 3, 16, 24), 3), ((1, 5, 8, 40), 3),
         ((3, 2, 32, 8), 2), ((1, 7, 24, 72), 3), ((1, 1, 2, 8), 1)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape,levels", CASES, ids=[f"{s}-L{l}" for s, l in CASES])
def test_dwt_and_iwt_small(shape, levels, dtype):
    from paper_2605_15684_amd import haar
    x, xg = _inputs(shape, dtype, seed=sum(shape) + levels)
    lv = haar.dwt(xg, levels)
    torch.cuda.synchronize()
    ref = H.dwt(x.double().numpy(), levels)
    for got, want in zip(lv, ref):
        _close(got, want, dtype)
    # the inverse of the stored levels, against the oracle's inverse of the same values
    stored = [t.double().cpu().numpy() for t in lv]
    y = haar.iwt(lv)
    torch.cuda.synchronize()
    _close(y, H.iwt(stored), dtype)
    if dtype == torch.float32:
        assert float((y.cpu() - x).abs().max()) <= 1e-5      # perfect reconstruction


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_iwt_with_residuals(dtype):
    from paper_2605_15684_amd import haar
    shape, levels = (2, 3, 16, 32), 3
    x, xg = _inputs(shape, dtype, seed=5)
    lv = haar.dwt(xg, levels)
    res = []
    for l in range(levels):
        r, rg = _inputs((2, 3, 16 >> l, 32 >> l), dtype, seed=40 + l)
        res.append(rg if l != 1 else None)                    # one level without a residual
    y = haar.iwt(lv, res)
    torch.cuda.synchronize()
    want = H.iwt([t.double().cpu().numpy() for t in lv],
                 [None if r is None else r.double().cpu().numpy() for r in res])
    _close(y, want, dtype)


def test_full_size_sampled_planes():
    """The benchmark shape ([4, 128, 512, 512] bf16, 3 levels): every output of
    six planes against the oracle, the round trip on all planes."""
    from paper_2605_15684_amd import haar
    shape, levels = (4, 128, 512, 512), 3
    x, xg = _inputs(shape, torch.bfloat16, seed=1)
    lv = haar.dwt(xg, levels)
    y = haar.iwt(lv)
    torch.cuda.synchronize()
    for n, c in ((0, 0), (0, 127), (1, 63), (2, 64), (3, 1), (3, 126)):
        ref = H.dwt(x[n:n + 1, c:c + 1].double().numpy(), levels)
        for l, (got, want) in enumerate(zip(lv, ref)):
            _close(got[n:n + 1, 4 * c:4 * c + 4], want, torch.bfloat16)
    # round trip through bf16-stored bands: within the bf16 rounding of each level
    err = (y.float() - xg.float()).abs().max().item()
    assert err <= 0.05, err


def test_stream_ordering_and_no_overrun():
    """Outputs land exactly in their tensors: guard bands around each level
    stay untouched."""
    from paper_2605_15684_amd import haar
    shape, levels = (1, 2, 16, 16), 3
    x, xg = _inputs(shape, torch.float32, seed=9)
    outs, views = [], []
    for l in range(1, levels + 1):
        n = 1 * 8 * (16 >> l) * (16 >> l)
        buf = torch.full((n + 128,), 123.0, device="cuda")
        outs.append(buf)
        views.append(buf[64:64 + n].view(1, 8, 16 >> l, 16 >> l))
    haar.dwt(xg, levels, out=views)
    torch.cuda.synchronize()
    for buf in outs:
        assert bool((buf[:64] == 123.0).all()) and bool((buf[-64:] == 123.0).all())
