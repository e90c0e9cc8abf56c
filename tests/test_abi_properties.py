"""Property checks of the C ABI's host layer over many generated descriptors
(no GPU, nothing launched): every accepted descriptor's workspace sizes
follow the documented formulas, the layer-stack sizes are whole multiples of
one call's, and the size-checked entry points accept exactly those sizes and
reject one byte less with SSBA_ERR_WORKSPACE before any launch (the buffer
pointers are never dereferenced on that path)."""
import os

import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from paper_2605_15684_amd import _lib

FAKE = 0x100000


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2605_15684_amd import build
        build.build()
    return _lib.load()


@st.composite
def descriptors(draw):
    tile = draw(st.sampled_from([4, 8, 16]))
    ny = draw(st.integers(1, 8))
    nx = draw(st.integers(1, 8))
    tb = ny * nx
    gate = draw(st.sampled_from([_lib.GATE_TOPK, _lib.GATE_WINDOW, _lib.GATE_DENSE, _lib.GATE_TOPK_SHARED]))
    win_h = draw(st.sampled_from([w for w in range(1, ny + 1) if ny % w == 0]))
    win_w = draw(st.sampled_from([w for w in range(1, nx + 1) if nx % w == 0]))
    d = _lib.SsbaDesc()
    kw = dict(batch=draw(st.integers(1, 4)), heads=draw(st.integers(1, 8)),
              head_dim=draw(st.sampled_from([64, 128])), grid_h=ny * tile, grid_w=nx * tile, tile=tile,
              shift_y=draw(st.integers(-40, 40)), shift_x=draw(st.integers(-40, 40)),
              n_text=draw(st.integers(0, 300)), gate=gate, keep=draw(st.integers(1, tb)),
              win_h=win_h, win_w=win_w, dtype=draw(st.sampled_from([_lib.DT_BF16, _lib.DT_F32])),
              softmax_scale=0.0, stride_b=0, stride_h=0, stride_t=0)
    for k, v in kw.items():
        setattr(d, k, v)
    return d, tb


def _expected(d, tb):
    pairs = d.batch * d.heads
    index = 4 * pairs * tb * (1 + tb)
    flags = 4 * pairs * tb
    if d.gate == _lib.GATE_TOPK:
        scratch = 16 * pairs * tb * d.head_dim + flags
    elif d.gate == _lib.GATE_TOPK_SHARED:
        scratch = 16 * pairs * tb * d.head_dim + 8 * pairs * tb * tb + flags
    else:
        scratch = flags
    return index, scratch


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(descriptors())
def test_workspace_sizes_follow_the_formulas(lib, dt):
    d, tb = dt
    assert _lib.workspace_size(d) == _expected(d, tb)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(descriptors(), st.integers(1, 6))
def test_layer_stack_sizes_are_whole_slices(lib, dt, n_layers):
    d, tb = dt
    ib, sb = _lib.workspace_size(d)
    lib_, lsb = _lib.layers_workspace_size(d, n_layers)
    assert lib_ == n_layers * ib
    assert lsb == n_layers * ((sb + 255) // 256 * 256)


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(descriptors())
def test_one_byte_short_is_rejected_before_launch(lib, dt):
    d, _ = dt
    ib, sb = _lib.workspace_size(d)
    W = _lib.SSBA_ERR_WORKSPACE
    assert _lib.build_index(d, FAKE, FAKE, FAKE, FAKE, None, ib - 1, sb) == W
    assert _lib.build_index(d, FAKE, FAKE, FAKE, FAKE, None, ib, sb - 1) == W
    assert _lib.forward(d, FAKE, FAKE, FAKE, FAKE, FAKE, None, ib - 1) == W
    if d.gate in (_lib.GATE_TOPK, _lib.GATE_TOPK_SHARED):
        assert _lib.forward_topk(d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, ib - 1, sb) == W
        assert _lib.forward_topk(d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, ib, sb - 1) == W
