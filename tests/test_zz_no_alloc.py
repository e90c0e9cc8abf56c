"""ssba_forward_topk_noalloc (scratch from the library's fixed device array,
for callers that cannot allocate) against ssba_forward_topk with a caller
scratch buffer: index rows and outputs identical, on two calls in a row, the
second with a smaller input.  (Descriptors whose scratch would exceed the
array are rejected before any launch: tests/test_abi.py.)"""
import numpy as np
import pytest
import torch

from paper_2605_15684_amd import _lib
from paper_2605_15684_amd.inputs import preset, workload_from

from _parity import gpu_desc, inputs, oracle_index

pytestmark = pytest.mark.gpu


def _noalloc(w):
    from paper_2605_15684_amd import ssba
    (q, k, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    ib, _ = _lib.workspace_size(desc)
    index = torch.full((ib // 4,), -7, dtype=torch.int32, device="cuda")
    out = torch.full_like(qg, float("nan"))
    st = _lib.forward_topk_noalloc(desc, qg.data_ptr(), kg.data_ptr(), vg.data_ptr(), index.data_ptr(),
                                   out.data_ptr(), torch.cuda.current_stream().cuda_stream, ib)
    _lib.check(st, "ssba_forward_topk_noalloc")
    ref_index, _, ref_out = ssba.forward_topk(qg, kg, vg, desc)
    torch.cuda.synchronize()
    got_index = index.view(ref_index.shape)
    assert torch.equal(got_index, ref_index)
    assert np.array_equal(got_index.cpu().numpy(), oracle_index(w, q, k))
    assert torch.equal(out, ref_out)


def test_noalloc_matches_forward_topk_twice_second_smaller():
    _noalloc(preset("grid64"))                      # 1 MB of scratch
    _noalloc(workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=5,
                           shift=(-4, -4), n_text=13))   # smaller, with a ragged text tail
