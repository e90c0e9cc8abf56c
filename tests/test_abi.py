"""Host-side checks of the C ABI (no GPU needed, nothing is launched): the
library loads, exports every function include/ssba.h declares, sizes its
workspace as documented and rejects bad descriptors before any launch."""
import ctypes
import glob
import os
import re

import pytest

from paper_2605_15684_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2605_15684_amd import build
        build.build()
    return _lib.load()


def _declared_functions():
    text = "\n".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssba_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert set(names) == set(_lib.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_status_strings(lib):
    assert lib.ssba_abi_version() == 3
    seen = set()
    for s in range(7):
        txt = _lib.status_str(s)
        assert txt and txt != "unknown status"
        seen.add(txt)
    assert len(seen) == 7
    assert _lib.status_str(99) == "unknown status"


def _desc(**kw):
    d = _lib.SsbaDesc()
    base = dict(batch=1, heads=16, head_dim=64, grid_h=64, grid_w=64, tile=8, shift_y=4, shift_x=4,
                n_text=0, gate=_lib.GATE_TOPK, keep=10, win_h=1, win_w=1, dtype=_lib.DT_BF16,
                softmax_scale=0.0, stride_b=0, stride_h=0, stride_t=0)
    base.update(kw)
    for k, v in base.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("kw,index_bytes,scratch_bytes", [
    ({}, 4 * 16 * 64 * 65, 16 * 16 * 64 * 64 + 4 * 16 * 64),
    ({"gate": _lib.GATE_WINDOW, "win_h": 2, "win_w": 2}, 4 * 16 * 64 * 65, 4 * 16 * 64),
    ({"gate": _lib.GATE_DENSE, "batch": 2, "heads": 24, "n_text": 256}, 4 * 48 * 64 * 65, 4 * 48 * 64),
    ({"grid_h": 128, "grid_w": 128, "tile": 16, "head_dim": 128, "keep": 7},
     4 * 16 * 64 * 65, 16 * 16 * 64 * 128 + 4 * 16 * 64),
    ({"grid_h": 16, "grid_w": 16, "tile": 4, "heads": 2, "keep": 4, "dtype": _lib.DT_F32},
     4 * 2 * 16 * 17, 16 * 2 * 16 * 64 + 4 * 2 * 16),
    ({"gate": _lib.GATE_TOPK_SHARED}, 4 * 16 * 64 * 65, 16 * 16 * 64 * 64 + 8 * 16 * 64 * 64 + 4 * 16 * 64),
])
def test_workspace_sizes(lib, kw, index_bytes, scratch_bytes):
    assert _lib.workspace_size(_desc(**kw)) == (index_bytes, scratch_bytes)


@pytest.mark.parametrize("kw,status", [
    ({"batch": 0}, _lib.SSBA_ERR_SHAPE),
    ({"heads": -1}, _lib.SSBA_ERR_SHAPE),
    ({"n_text": -3}, _lib.SSBA_ERR_SHAPE),
    ({"grid_h": 60}, _lib.SSBA_ERR_SHAPE),
    ({"head_dim": 96}, _lib.SSBA_ERR_UNSUPPORTED),
    ({"tile": 32}, _lib.SSBA_ERR_UNSUPPORTED),
    ({"grid_h": 512, "grid_w": 512}, _lib.SSBA_ERR_UNSUPPORTED),   # 4096 blocks > 1024
    ({"dtype": 7}, _lib.SSBA_ERR_ARG),
    ({"gate": 9}, _lib.SSBA_ERR_ARG),
    ({"keep": 0}, _lib.SSBA_ERR_ARG),
    ({"keep": 65}, _lib.SSBA_ERR_ARG),
    ({"gate": _lib.GATE_WINDOW, "win_h": 3, "win_w": 1}, _lib.SSBA_ERR_ARG),
    ({"gate": _lib.GATE_WINDOW, "win_h": 0, "win_w": 1}, _lib.SSBA_ERR_ARG),
    ({"softmax_scale": float("nan")}, _lib.SSBA_ERR_ARG),
    ({"stride_b": 1, "stride_h": 1, "stride_t": 32}, _lib.SSBA_ERR_SHAPE),
    ({"stride_b": 64 * 4096 * 16, "stride_h": 64 * 4096, "stride_t": 68}, _lib.SSBA_ERR_UNSUPPORTED),
])
def test_bad_descriptors_rejected_before_launch(lib, kw, status):
    d = _desc(**kw)
    ib, sb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.ssba_workspace_size(ctypes.byref(d), ctypes.byref(ib), ctypes.byref(sb)) == status
    # Every entry point validates the descriptor first; pointers are never touched.
    assert _lib.build_index(d, None, None, None, None, None) == status
    assert _lib.forward(d, None, None, None, None, None, None) == status
    assert _lib.forward_dense(d, None, None, None, None, None) == status


def test_null_pointers_rejected(lib):
    d = _desc()
    assert _lib.build_index(d, None, None, None, None, None) == _lib.SSBA_ERR_ARG
    assert _lib.forward(d, None, None, None, None, None, None) == _lib.SSBA_ERR_ARG
    assert _lib.forward_dense(d, None, None, None, None, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_workspace_size(None, None, None) == _lib.SSBA_ERR_ARG
    out = ctypes.c_int(0)
    assert lib.ssba_read_device_status(ctypes.byref(d), None, ctypes.byref(out), None) == _lib.SSBA_ERR_ARG


def test_misaligned_pointers_rejected(lib):
    d = _desc()
    # bf16 attention needs 16-byte aligned bases; rejected before any launch.
    assert _lib.forward(d, 0x1002, 0x2000, 0x3000, 0x4000, 0x5000, None) == _lib.SSBA_ERR_ARG
    assert _lib.build_index(d, 0x1000, 0x2000, 0x3002, 0x4000, None) == _lib.SSBA_ERR_ARG


@pytest.mark.parametrize("kw,dense,name", [
    ({}, False, "k_attn_mfma<64, 3, false, false>"),
    ({}, True, "k_attn_mfma<64, 3, true, false>"),
    ({"n_text": 256, "batch": 2, "heads": 24}, False, "k_attn_mfma<64, 3, false, false>"),
    ({"grid_h": 128, "grid_w": 128, "tile": 16, "head_dim": 128, "keep": 7}, False, "k_attn_mfma<128, 4, false, false>"),
    ({"grid_h": 128, "grid_w": 128, "tile": 16, "head_dim": 128, "keep": 7}, True, "k_attn_mfma<128, 3, true, false>"),
    ({"grid_h": 64, "grid_w": 64, "tile": 16, "keep": 4}, False, "k_attn_mfma<64, 4, false, false>"),
    ({"grid_h": 16, "grid_w": 16, "tile": 4, "keep": 4, "dtype": _lib.DT_F32}, False, "k_attn_f32<64>"),
    ({"grid_h": 32, "grid_w": 32, "tile": 4, "keep": 4}, False, "k_attn_bf16<64, 2>"),
])
def test_forward_kernel_names(lib, kw, dense, name):
    assert _lib.forward_kernel(_desc(**kw), dense) == name


@pytest.mark.parametrize("kw,name", [
    ({}, "k_attn_mfma<64, 3, false, true>"),
    ({"n_text": 256, "batch": 2, "heads": 24}, "k_attn_mfma<64, 3, false, true>"),
    ({"head_dim": 128}, "k_attn_mfma<128, 3, false, true>"),
    ({"grid_h": 128, "grid_w": 128, "tile": 16, "head_dim": 128, "keep": 7}, "k_attn_mfma<128, 4, false, false>"),
    ({"grid_h": 16, "grid_w": 16, "tile": 4, "keep": 4, "dtype": _lib.DT_F32}, "k_attn_f32<64>"),
])
def test_forward_topk_kernel_names(lib, kw, name):
    assert _lib.forward_kernel(_desc(**kw), mode=2) == name


def test_forward_topk_rejects_other_gates_before_launch(lib):
    d = _desc(gate=_lib.GATE_WINDOW, win_h=2, win_w=2)
    buf = ctypes.c_void_p(256)   # never dereferenced: the descriptor is rejected first
    assert lib.ssba_forward_topk(ctypes.byref(d), buf, buf, buf, buf, buf, buf, None) == _lib.SSBA_ERR_ARG
    assert _lib.forward_kernel(d, mode=2) is None
    assert _lib.forward_kernel(_desc(), mode=3) is None


def test_forward_kernel_name_of_invalid_descriptor(lib):
    assert _lib.forward_kernel(_desc(keep=0)) is None
    assert _lib.forward_kernel(_desc(keep=0), dense=True) == "k_attn_mfma<64, 3, true, false>"
    assert _lib.forward_kernel(_desc(head_dim=96)) is None


@pytest.mark.parametrize("kw", [{}, {"gate": _lib.GATE_WINDOW, "win_h": 2, "win_w": 2},
                                {"gate": _lib.GATE_TOPK_SHARED, "keep": 0}, {"keep": 0, "heads": 3}])
def test_layers_workspace_size(lib, kw):
    d = _desc(**kw)
    one = _desc(**dict(kw, keep=1)) if "keep" in kw else d
    ib1, sb1 = _lib.workspace_size(one)
    for n in (1, 2, 24):
        ib, sb = _lib.layers_workspace_size(d, n)
        assert ib == n * ib1
        assert sb == n * ((sb1 + 255) // 256 * 256)


def test_layers_bad_arguments_rejected_before_launch(lib):
    d = _desc()
    fake = 1 << 20                                   # aligned, never dereferenced: rejected first
    layers = (_lib.SsbaLayer * 3)()
    for e in layers:
        e.q = e.k = e.v = e.o = fake
        e.keep = 10
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 0, fake, fake, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_forward_layers(ctypes.byref(d), None, 3, fake, fake, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_forward_layers(None, layers, 3, fake, fake, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 3, None, fake, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 3, fake, None, None) == _lib.SSBA_ERR_ARG
    layers[2].keep = 65                              # keep beyond T_b in the last layer
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 3, fake, fake, None) == _lib.SSBA_ERR_ARG
    layers[2].skip = 1                               # ... unless that layer is skipped: then a null
    layers[1].q = None                               # q in layer 1 is still caught
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 3, fake, fake, None) == _lib.SSBA_ERR_ARG
    layers[1].q = fake + 8                           # misaligned bf16 rows
    assert lib.ssba_forward_layers(ctypes.byref(d), layers, 3, fake, fake, None) == _lib.SSBA_ERR_ARG
    bad = _desc(grid_h=60)
    layers[1].q = fake
    assert lib.ssba_forward_layers(ctypes.byref(bad), layers, 3, fake, fake, None) == _lib.SSBA_ERR_SHAPE


def test_shared_gate_names_two_call_kernel(lib):
    """The shared gate runs the two calls inside ssba_forward_topk: mode 2
    names the ungated attention kernel."""
    assert _lib.forward_kernel(_desc(gate=_lib.GATE_TOPK_SHARED), mode=2) == "k_attn_mfma<64, 3, false, false>"
    assert _lib.forward_kernel(_desc(), mode=2) == "k_attn_mfma<64, 3, false, true>"


def _hdesc(**kw):
    d = _lib.HaarDesc()
    base = dict(n=1, c=128, h=512, w=512, levels=3, dtype=_lib.DT_BF16)
    base.update(kw)
    for k, v in base.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("kw,status", [
    ({"n": 0}, _lib.SSBA_ERR_SHAPE), ({"c": -1}, _lib.SSBA_ERR_SHAPE),
    ({"h": 12}, _lib.SSBA_ERR_SHAPE),                   # not a multiple of 2^3
    ({"w": 20}, _lib.SSBA_ERR_SHAPE),                   # not a multiple of 8
    ({"levels": 0}, _lib.SSBA_ERR_UNSUPPORTED), ({"levels": 4}, _lib.SSBA_ERR_UNSUPPORTED),
    ({"dtype": 5}, _lib.SSBA_ERR_ARG),
])
def test_haar_bad_descriptors_rejected_before_launch(lib, kw, status):
    d = _hdesc(**kw)
    fake = 1 << 20
    assert _lib.haar_dwt(d, fake, [fake] * 3, None) == status
    assert _lib.haar_iwt(d, [fake] * 3, None, fake, None) == status
    assert _lib.haar_kernel_name(d, False) is None


def test_haar_null_and_misaligned_pointers_rejected(lib):
    d = _hdesc()
    fake = 1 << 20
    assert _lib.haar_dwt(d, None, [fake] * 3, None) == _lib.SSBA_ERR_ARG
    assert _lib.haar_dwt(d, fake, [fake, None, fake], None) == _lib.SSBA_ERR_ARG
    assert _lib.haar_dwt(d, fake + 2, [fake] * 3, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_haar_dwt(ctypes.byref(d), fake, None, None) == _lib.SSBA_ERR_ARG
    assert _lib.haar_iwt(d, [fake] * 3, None, None, None) == _lib.SSBA_ERR_ARG
    assert _lib.haar_iwt(d, [fake, fake, fake + 8], None, fake, None) == _lib.SSBA_ERR_ARG
    assert _lib.haar_iwt(d, [fake] * 3, [None, fake + 4, None], fake, None) == _lib.SSBA_ERR_ARG
    assert lib.ssba_haar_dwt(None, fake, None, None) == _lib.SSBA_ERR_ARG


def test_haar_kernel_names(lib):
    assert _lib.haar_kernel_name(_hdesc(), False) == "k_haar_dwt<unsigned short, 3>"
    assert _lib.haar_kernel_name(_hdesc(levels=1, dtype=_lib.DT_F32), True) == "k_haar_iwt<float, 1>"


@pytest.mark.parametrize("kw", [{"tile": 16, "grid_h": 256, "grid_w": 256, "keep": 7},   # 256 blocks
                                {"tile": 4, "grid_h": 32, "grid_w": 32, "keep": 4},
                                {"dtype": _lib.DT_F32, "tile": 4, "grid_h": 16, "grid_w": 16, "keep": 4},
                                {"grid_h": 128, "grid_w": 128}])      # 256 blocks
def test_backward_unsupported_shapes_rejected_before_launch(lib, kw):
    d = _desc(**kw)
    fake = 1 << 20
    assert _lib.backward(d, *([fake] * 11), None) == _lib.SSBA_ERR_UNSUPPORTED


def test_backward_arguments_rejected_before_launch(lib):
    d = _desc()
    fake = 1 << 20
    args = [fake] * 11                           # q k v o dout lse index dq dk dv scratch
    for i in range(11):
        bad = list(args)
        bad[i] = None
        assert _lib.backward(d, *bad, None) == _lib.SSBA_ERR_ARG
    bad = list(args)
    bad[10] = fake + 16                          # scratch must be 256-byte aligned
    assert _lib.backward(d, *bad, None) == _lib.SSBA_ERR_ARG
    assert _lib.forward_train(d, fake, fake, fake, fake, fake, None, None) == _lib.SSBA_ERR_ARG
    assert _lib.forward_train(_desc(dtype=_lib.DT_F32), *([fake] * 6), None) == _lib.SSBA_ERR_UNSUPPORTED


def test_backward_workspace_size(lib):
    d = _desc(batch=2, heads=3, n_text=10)
    rows = 2 * 3 * (10 + 4096)
    up = lambda x: (x + 255) // 256 * 256
    assert _lib.backward_workspace_size(d) == 2 * up(4 * rows) + up(8 * 2 * 3 * 64) + up(4 * 2 * 3 * 64)


def test_probe_rejects_bad_arguments(lib):
    sink = ctypes.c_void_p(16)   # never dereferenced: every call below fails its checks first
    assert _lib.probe_mfma(0, 10, sink, None) == _lib.SSBA_ERR_ARG
    assert _lib.probe_mfma(4, 0, sink, None) == _lib.SSBA_ERR_ARG
    assert _lib.probe_mfma(4, (1 << 20) + 1, sink, None) == _lib.SSBA_ERR_ARG
    assert _lib.probe_mfma(4, 10, None, None) == _lib.SSBA_ERR_ARG


def test_short_workspace_rejected_before_launch(lib):
    """The _ex entry points return SSBA_ERR_WORKSPACE, before anything is
    launched, when index or scratch is one byte short of what the workspace
    queries report (no device is touched: the check precedes every launch)."""
    fake = ctypes.c_void_p(0x100000)
    d = _desc()
    ib, sb = _lib.workspace_size(d)
    W = _lib.SSBA_ERR_WORKSPACE
    assert _lib.build_index(d, fake, fake, fake, fake, None, ib - 1, sb) == W
    assert _lib.build_index(d, fake, fake, fake, fake, None, ib, sb - 1) == W
    assert _lib.forward(d, fake, fake, fake, fake, fake, None, ib - 1) == W
    assert _lib.forward_topk(d, fake, fake, fake, fake, fake, fake, None, ib - 1, sb) == W
    assert _lib.forward_topk(d, fake, fake, fake, fake, fake, fake, None, ib, sb - 1) == W
    assert _lib.forward_train(d, fake, fake, fake, fake, fake, fake, None, ib - 1) == W
    bsb = _lib.backward_workspace_size(d)
    assert _lib.backward(d, *([fake] * 11), None, ib - 1, bsb) == W
    assert _lib.backward(d, *([fake] * 11), None, ib, bsb - 1) == W
    out = ctypes.c_int(0)
    assert lib.ssba_read_device_status_ex(ctypes.byref(d), fake, sb - 1, ctypes.byref(out), None) == W
    # the layer stack needs n_layers slices of each
    layers = (_lib.SsbaLayer * 3)()
    for e in layers:
        e.q = e.k = e.v = e.o = 0x100000
        e.keep = 10
    lib_, lsb = _lib.layers_workspace_size(d, 3)
    assert _lib.forward_layers(d, layers, fake, fake, None, lib_ - 1, lsb) == W
    assert _lib.forward_layers(d, layers, fake, fake, None, lib_, lsb - 1) == W
    # the argument checks still come first
    assert _lib.forward_topk(d, None, fake, fake, fake, fake, fake, None, 0, 0) == _lib.SSBA_ERR_ARG
    bad = _desc(keep=0)
    assert _lib.build_index(bad, fake, fake, fake, fake, None, 0, 0) == _lib.SSBA_ERR_ARG


def test_noalloc_rejects_scratch_beyond_its_array(lib):
    """ssba_forward_topk_noalloc returns SSBA_ERR_WORKSPACE, before touching a
    device, when the descriptor's scratch exceeds the fixed array, and
    SSBA_ERR_ARG for a gate without scratch sums."""
    fake = 0x100000
    d = _desc(batch=8, heads=32, head_dim=128)
    _, sb = _lib.workspace_size(d)
    assert sb > _lib.NOALLOC_SCRATCH_BYTES
    assert _lib.forward_topk_noalloc(d, fake, fake, fake, fake, fake, None, 1 << 30) == _lib.SSBA_ERR_WORKSPACE
    w = _desc(gate=_lib.GATE_WINDOW, win_h=2, win_w=2)
    assert _lib.forward_topk_noalloc(w, fake, fake, fake, fake, fake, None, 1 << 30) == _lib.SSBA_ERR_ARG
    assert lib.ssba_forward_topk_noalloc(None, fake, fake, fake, fake, 1 << 30, fake, None) == _lib.SSBA_ERR_ARG


def test_split_fused_launches_checked_before_launch(lib):
    """ssba_pool_keys_ex and ssba_forward_gated_ex (the two launches of the
    fused top-k form) reject, before anything is launched, shapes the gated
    kernel does not take (SSBA_ERR_UNSUPPORTED), missing or misaligned
    buffers (SSBA_ERR_ARG) and short workspaces (SSBA_ERR_WORKSPACE)."""
    fake = 0x100000
    d = _desc()
    ib, sb = _lib.workspace_size(d)
    U, A, W = _lib.SSBA_ERR_UNSUPPORTED, _lib.SSBA_ERR_ARG, _lib.SSBA_ERR_WORKSPACE
    for other in (_desc(tile=16), _desc(gate=_lib.GATE_TOPK_SHARED),
                  _desc(dtype=_lib.DT_F32)):
        assert _lib.pool_keys(other, fake, fake, None, 1 << 30) == U
        assert _lib.forward_gated(other, fake, fake, fake, fake, fake, fake, None, 1 << 30, 1 << 30) == U
    assert _lib.pool_keys(d, None, fake, None, sb) == A
    assert _lib.pool_keys(d, fake, None, None, sb) == A
    assert _lib.pool_keys(d, fake + 2, fake, None, sb) == A
    assert _lib.pool_keys(d, fake, fake, None, sb - 1) == W
    for i in range(6):   # q, k, v, index, scratch, o in turn missing
        ptrs = [fake] * 6
        ptrs[i] = None
        assert _lib.forward_gated(d, *ptrs, None, ib, sb) == A
    assert _lib.forward_gated(d, fake, fake, fake, fake, fake, fake + 8, None, ib, sb) == A
    assert _lib.forward_gated(d, fake, fake, fake, fake, fake, fake, None, ib - 1, sb) == W
    assert _lib.forward_gated(d, fake, fake, fake, fake, fake, fake, None, ib, sb - 1) == W
    bad = _desc(keep=0)
    assert _lib.pool_keys(bad, fake, fake, None, sb) == A


def test_rope_calls_checked_before_launch(lib):
    """ssba_rope_pool_keys_ex and ssba_forward_topk_rope_ex reject
    unsupported shapes, missing or misaligned buffers, short workspaces and a
    non-finite frequency base before anything is launched."""
    fake = 0x100000
    d = _desc()
    ib, sb = _lib.workspace_size(d)
    U, A, W = _lib.SSBA_ERR_UNSUPPORTED, _lib.SSBA_ERR_ARG, _lib.SSBA_ERR_WORKSPACE
    for other in (_desc(tile=16), _desc(gate=_lib.GATE_TOPK_SHARED), _desc(dtype=_lib.DT_F32)):
        assert _lib.rope_pool_keys(other, fake, fake, fake, fake, 0.0, fake, None, 1 << 30) == U
        assert _lib.forward_topk_rope(other, fake, fake, fake, fake, fake, 0.0, fake, fake, fake, None,
                                      1 << 30, 1 << 30) == U
    for i in range(4):   # q, k, q_rope, k_rope in turn missing
        ptrs = [fake] * 4
        ptrs[i] = None
        assert _lib.rope_pool_keys(d, *ptrs, 0.0, fake, None, sb) == A
        ptrs[i] = fake + 8
        assert _lib.rope_pool_keys(d, *ptrs, 0.0, fake, None, sb) == A
    assert _lib.rope_pool_keys(d, fake, fake, fake, fake, 0.0, fake, None, sb - 1) == W
    for theta in (float("nan"), float("inf"), -float("inf")):
        assert _lib.rope_pool_keys(d, fake, fake, fake, fake, theta, fake, None, sb) == A
        assert _lib.forward_topk_rope(d, fake, fake, fake, fake, fake, theta, fake, fake, fake, None, ib, sb) == A
    assert _lib.forward_topk_rope(d, fake, fake, fake, fake, fake, 0.0, fake, fake, fake, None, ib - 1, sb) == W
    assert _lib.forward_topk_rope(d, fake, fake, None, fake, fake, 0.0, fake, fake, fake, None, ib, sb) == A
    assert _lib.forward_topk_rope(d, fake, fake, fake, None, fake, 0.0, fake, fake, fake, None, ib, sb) == A
