"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on
the same seeded inputs.  Index lists must match bit for bit; outputs within
2e-2 max-abs for bf16 inputs and 1e-5 for fp32."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O
from paper_2605_15684_amd.inputs import (PRESETS, SWEEP_TOPK_KEEP, SWEEP_WINDOW, Workload, make_qkv,
                                         preset, workload_from)

from _parity import (BF16_TOL, F32_TOL, gpu_desc, inputs, max_err, oracle_index, oracle_kw,
                      run_gpu, sample_rows, to64, tol)  # noqa: F401

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- index --
INDEX_CASES = [
    preset("tiny"), preset("tiny", shift=(-2, -2)),
    preset("tiny", gate="window", window=(1, 1), shift=(0, 0)),
    preset("tiny", gate="window", window=(1, 1), shift=(2, 2)),
    preset("tiny", gate="window", window=(2, 4), shift=(1, -3)),
    preset("tiny", gate="dense"), preset("tiny", keep=1), preset("tiny", keep=16),
    preset("grid64"), preset("grid64", shift=(-4, -4)),
    preset("grid64_text"), preset("grid128"),
] + [preset("sweep64", keep=k) for k in SWEEP_TOPK_KEEP.values()] \
  + [preset("sweep64", gate="window", window=w) for w in SWEEP_WINDOW.values()]


@pytest.mark.parametrize("w", INDEX_CASES, ids=lambda w: f"{w.name}-{w.gate}-k{w.keep}-w{w.window}-s{w.shift}")
def test_index_bit_exact(w):
    (q, k, _), (qg, kg, _) = inputs(w)
    from paper_2605_15684_amd import ssba
    desc = gpu_desc(w, qg)
    index, scratch = ssba.build_index(qg, kg, desc)
    got = index.cpu().numpy()
    want = oracle_index(w, q, k)
    assert got.dtype == want.dtype == np.int32 and got.shape == want.shape
    assert np.array_equal(got, want)
    assert ssba.read_status(desc, scratch) == 0
    if w.gate == "topk":
        assert (got[..., 0] == w.keep).all()


# ------------------------------------------------------- small, full output --
SMALL = [
    preset("tiny"),                                                  # fp32, 4x4 blocks
    preset("tiny", shift=(-2, -2)),
    preset("tiny", gate="window", window=(1, 1), shift=(0, 0)),
    preset("tiny", gate="window", window=(1, 1), shift=(2, 2)),
    preset("tiny", gate="dense"),
    preset("tiny", n_text=7, heads=1),                               # fp32 ragged text
    preset("tiny", head_dim=128, tile=8, keep=2, shift=(4, 4)),      # fp32 D128, 8x8
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=4, shift=(4, 4)),
    workload_from(batch=2, heads=1, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=5, shift=(-4, -4),
                  n_text=77),                                        # ragged text tail
    workload_from(batch=1, heads=2, grid_h=32, grid_w=16, head_dim=64, tile=8, keep=1, shift=(3, -5),
                  n_text=64),
    workload_from(batch=1, heads=2, grid_h=64, grid_w=64, head_dim=128, tile=16, keep=3, shift=(8, 8),
                  heavy_key_rows=40),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=128, tile=8, keep=6, shift=(4, 4),
                  n_text=13),
    workload_from(batch=1, heads=2, grid_h=64, grid_w=32, head_dim=64, tile=16, keep=2, shift=(-8, 8)),
    workload_from(batch=1, heads=2, grid_h=16, grid_w=16, head_dim=64, tile=4, keep=5, shift=(2, 2)),
    workload_from(batch=1, heads=1, grid_h=16, grid_w=32, head_dim=128, tile=4, keep=7, shift=(1, 2),
                  n_text=20),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, gate="window",
                  window=(2, 2), shift=(4, 4)),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, gate="dense", n_text=5),
]


def _ids(w: Workload):
    return f"{w.name}-{w.dtype}-D{w.head_dim}-B{w.tile}-{w.gate}{w.keep}-t{w.n_text}-s{w.shift}"


@pytest.mark.parametrize("w", SMALL, ids=_ids)
def test_output_small_full(w):
    (q, k, v), (qg, kg, vg) = inputs(w)
    index, out = run_gpu(w, qg, kg, vg)
    want_idx = oracle_index(w, q, k)
    assert np.array_equal(index, want_idx)
    ref = O.attention(to64(q), to64(k), to64(v), want_idx, **oracle_kw(w))
    got = out.float().cpu().double().numpy()
    err = np.abs(got - ref).max()
    assert np.isfinite(got).all()
    assert err <= tol(w), f"max-abs {err:.3e}"


@pytest.mark.parametrize("w", [preset("tiny"), preset("tiny", n_text=9, heads=1),
                               workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64,
                                             tile=8, n_text=70),
                               workload_from(batch=1, heads=1, grid_h=32, grid_w=32, head_dim=128,
                                             tile=16, n_text=3)], ids=_ids)
def test_dense_path_small(w):
    (q, k, v), (qg, kg, vg) = inputs(w)
    _, out = run_gpu(w, qg, kg, vg, dense=True)
    idx = O.build_index(to64(q), to64(k), gate="dense", **oracle_kw(w))
    ref = O.attention(to64(q), to64(k), to64(v), idx, **oracle_kw(w))
    err = np.abs(out.float().cpu().double().numpy() - ref).max()
    assert err <= tol(w), f"max-abs {err:.3e}"


# -------------------------------------------- full size, sampled outputs --
FULL = [preset("grid64"), preset("grid64", shift=(-4, -4)), preset("grid64_text"), preset("grid128"),
        preset("sweep64")]


@pytest.mark.parametrize("w", FULL, ids=_ids)
def test_output_full_size_sampled(w):
    (q, k, v), (qg, kg, vg) = inputs(w)
    index, out = run_gpu(w, qg, kg, vg)
    want_idx = oracle_index(w, q, k)
    assert np.array_equal(index, want_idx)
    rng = np.random.default_rng(123)
    heads = [(0, 0), (w.batch - 1, w.heads - 1), (int(rng.integers(w.batch)), int(rng.integers(w.heads)))]
    rows = sample_rows(w, rng)
    ref = O.attention(to64(q), to64(k), to64(v), want_idx, rows=rows, heads=heads, **oracle_kw(w))
    err = max_err(out, ref, heads, rows)
    assert err <= BF16_TOL, f"max-abs {err:.3e}"


@pytest.mark.parametrize("w", [preset("grid64"), preset("grid64_text")], ids=_ids)
def test_dense_path_full_size_sampled(w):
    (q, k, v), (qg, kg, vg) = inputs(w)
    _, out = run_gpu(w, qg, kg, vg, dense=True)
    rng = np.random.default_rng(7)
    heads = [(0, 0), (w.batch - 1, w.heads - 1)]
    rows = sample_rows(w, rng)
    idx = O.build_index(to64(q[:1, :1]), to64(k[:1, :1]), gate="dense", **oracle_kw(w))
    idx = np.broadcast_to(idx, (w.batch, w.heads) + idx.shape[2:])
    ref = O.attention(to64(q), to64(k), to64(v), idx, rows=rows, heads=heads, **oracle_kw(w))
    assert max_err(out, ref, heads, rows) <= BF16_TOL


# -------------------------------------------------------------- properties --
def test_rows_sum_to_one_via_ones_values():
    w = preset("grid64_text", batch=1, heads=2)
    (q, k, _), (qg, kg, _) = inputs(w)
    vg = torch.ones_like(qg)
    _, out = run_gpu(w, qg, kg, vg)
    assert (out.float() - 1.0).abs().max().item() <= BF16_TOL / 4


def test_deterministic_and_stride_independent():
    w = preset("grid64_text", batch=1, heads=4)
    (_, _, _), (qg, kg, vg) = inputs(w)
    i1, o1 = run_gpu(w, qg, kg, vg)
    i2, o2 = run_gpu(w, qg, kg, vg)
    assert np.array_equal(i1, i2) and torch.equal(o1, o2)
    # Same data stored as [B, T, H, D] and viewed as [B, H, T, D].
    qs, ks, vs = (t.transpose(1, 2).contiguous().transpose(1, 2) for t in (qg, kg, vg))
    assert qs.stride() != qg.stride()
    i3, o3 = run_gpu(w, qs, ks, vs)
    assert np.array_equal(i1, i3) and torch.equal(o1, o3.contiguous())


def test_nonfinite_input_sets_status():
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2)
    (_, _, _), (qg, kg, _) = inputs(w)
    desc = gpu_desc(w, qg)
    _, scratch = ssba.build_index(qg, kg, desc)
    assert ssba.read_status(desc, scratch) == 0
    kg2 = kg.clone()
    kg2[0, 1, 100, 5] = float("nan")
    _, scratch = ssba.build_index(qg, kg2, desc)
    assert ssba.read_status(desc, scratch) == 5


def test_permutation_within_a_block():
    w = preset("grid64", heads=2)
    (q, k, v), (qg, kg, vg) = inputs(w)
    tiles = O.frame_tiles(w.grid_h, w.grid_w, w.tile, *w.shift)
    rng = np.random.default_rng(0)
    perm = np.arange(w.t_img)
    for t in range(tiles.shape[0]):
        perm[tiles[t]] = tiles[t][rng.permutation(tiles.shape[1])]
    p = torch.tensor(perm, device="cuda")
    i1, o1 = run_gpu(w, qg, kg, vg)
    i2, o2 = run_gpu(w, qg, kg[:, :, p], vg[:, :, p])
    assert np.array_equal(i1, i2)
    assert (o1.float() - o2.float()).abs().max().item() <= BF16_TOL
    i3, o3 = run_gpu(w, qg[:, :, p], kg, vg)
    assert np.array_equal(i1, i3)
    assert (o3.float() - o1[:, :, p].float()).abs().max().item() <= BF16_TOL


def test_half_block_offsets_agree():
    w = preset("grid64", heads=2)
    (_, _, _), (qg, kg, vg) = inputs(w)
    _, a = run_gpu(w.with_(shift=(4, 4)), qg, kg, vg)
    _, b = run_gpu(w.with_(shift=(-4, -4)), qg, kg, vg)
    assert (a.float() - b.float()).abs().max().item() <= BF16_TOL


def test_zero_sparsity_equals_dense_path():
    w = preset("grid64", heads=2, keep=64)
    (_, _, _), (qg, kg, vg) = inputs(w)
    _, a = run_gpu(w, qg, kg, vg)
    _, b = run_gpu(w, qg, kg, vg, dense=True)
    assert (a.float() - b.float()).abs().max().item() <= BF16_TOL


def test_attention_convenience_call():
    from paper_2605_15684_amd import ssba
    w = preset("grid64_text", batch=1, heads=2)
    (q, k, v), (qg, kg, vg) = inputs(w)
    img = ssba.attention(qg, kg, vg, grid=(64, 64), tile=8, layer=0, keep=10, n_text=256,
                         return_text=False)
    assert img.shape == (1, 2, 4096, 64)
    _, full = run_gpu(w, qg, kg, vg)
    assert torch.equal(img, full[:, :, 256:])


def test_graph_replay_matches_eager():
    """A step (gate + attention) captured in a HIP graph and replayed several
    times, with eager work on other inputs in between, equals the eager step
    bit for bit on every replay."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64_text", batch=1, heads=4)
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, scratch = ssba.alloc_workspace(desc, qg.device)
    out = torch.empty_like(qg)

    def step():
        ssba.build_index(qg, kg, desc, index, scratch)
        ssba.forward(qg, kg, vg, index, desc, out)

    step()
    torch.cuda.synchronize()
    ref_index, ref_out = index.clone(), out.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    other = torch.randn_like(qg)
    for rep in range(4):
        index.fill_(-7)
        out.zero_()
        _, eager_other = run_gpu(w, other, kg, vg)     # unrelated eager work in between
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(index, ref_index), rep
        assert torch.equal(out, ref_out), rep
        assert eager_other.shape == out.shape


TOPK_CASES = [
    preset("grid64", heads=4),
    preset("grid64", heads=2, shift=(-4, -4)),
    preset("grid64_text", batch=1, heads=4),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=64, head_dim=128, tile=8, keep=5, shift=(4, -4),
                  n_text=77),
    workload_from(batch=2, heads=3, grid_h=48, grid_w=40, head_dim=64, tile=8, keep=7, shift=(3, 5),
                  n_text=13),
    preset("grid128", heads=2),                                  # 16x16 blocks: two-call route
    preset("tiny"),                                              # fp32: two-call route
]
# Few blocks per head in the gated kernel: one block, two blocks both kept
# (with text), sixteen blocks all kept.
FEW_BLOCKS = [
    workload_from(batch=1, heads=2, grid_h=8, grid_w=8, head_dim=64, tile=8, keep=1, shift=(4, 4)),
    workload_from(batch=2, heads=1, grid_h=8, grid_w=16, head_dim=128, tile=8, keep=2, shift=(-4, 4),
                  n_text=5),
    workload_from(batch=1, heads=2, grid_h=32, grid_w=32, head_dim=64, tile=8, keep=16, shift=(4, 4)),
]
TOPK_CASES += FEW_BLOCKS


@pytest.mark.parametrize("w", TOPK_CASES, ids=_ids)
def test_forward_topk_equals_build_index_then_forward(w):
    """The fused gate writes bit-identical index rows and status flags, and the
    attention output equals the two-call output bit for bit."""
    from paper_2605_15684_amd import ssba
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index2, scratch2 = ssba.build_index(qg, kg, desc)
    out2 = ssba.forward(qg, kg, vg, index2, desc)
    index1, scratch1 = ssba.alloc_workspace(desc, qg.device)
    index1.fill_(-5)
    _, _, out1 = ssba.forward_topk(qg, kg, vg, desc, index1, scratch1)
    torch.cuda.synchronize()
    assert torch.equal(index1, index2)
    assert ssba.read_status(desc, scratch1) == ssba.read_status(desc, scratch2) == 0
    assert torch.equal(out1, out2)


@pytest.mark.parametrize("w", TOPK_CASES[:5] + FEW_BLOCKS, ids=_ids)
def test_pool_keys_then_forward_gated_equals_forward_topk(w):
    """The fused form's two launches called one at a time give the fused
    call's index rows, status flags and output bit for bit; the index is the
    oracle's."""
    from paper_2605_15684_amd import ssba
    (q, k, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index1, scratch1, out1 = ssba.forward_topk(qg, kg, vg, desc)
    index2, scratch2 = ssba.alloc_workspace(desc, qg.device)
    index2.fill_(-5)
    out2 = torch.full_like(out1, float("nan"))
    ssba.pool_keys(kg, desc, scratch2)
    ssba.forward_gated(qg, kg, vg, desc, index2, scratch2, out2)
    torch.cuda.synchronize()
    assert torch.equal(index1, index2) and torch.equal(out1, out2)
    assert ssba.read_status(desc, scratch2) == 0
    assert np.array_equal(index2.cpu().numpy(), oracle_index(w, q, k))


@pytest.mark.parametrize("w", FEW_BLOCKS, ids=_ids)
def test_forward_topk_few_blocks_against_oracle(w):
    """The fused call with one, two and sixteen blocks per head: index bit
    exact and every output row within tolerance of the oracle."""
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    index, _, out = ssba.forward_topk(qg, kg, vg, gpu_desc(w, qg))
    torch.cuda.synchronize()
    want_idx = oracle_index(w, q, k)
    assert np.array_equal(index.cpu().numpy(), want_idx)
    ref = O.attention(to64(q), to64(k), to64(v), want_idx, **oracle_kw(w))
    err = float(np.abs(out.float().cpu().double().numpy() - ref).max())
    assert err <= tol(w), f"max-abs {err:.3e}"


def test_forward_topk_full_size_against_oracle():
    from paper_2605_15684_amd import ssba
    w = preset("grid64")
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index, _, out = ssba.forward_topk(qg, kg, vg, desc)
    torch.cuda.synchronize()
    want_idx = oracle_index(w, q, k)
    assert np.array_equal(index.cpu().numpy(), want_idx)
    rng = np.random.default_rng(7)
    heads = [(0, 0), (0, w.heads - 1), (0, int(rng.integers(w.heads)))]
    rows = sample_rows(w, rng)
    ref = O.attention(to64(q), to64(k), to64(v), want_idx, rows=rows, heads=heads, **oracle_kw(w))
    err = max_err(out, ref, heads, rows)
    assert err <= BF16_TOL, f"max-abs {err:.3e}"


def test_forward_topk_nonfinite_sets_status():
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2)
    (_, _, _), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    kg2 = kg.clone()
    kg2[0, 1, 100, 5] = float("nan")
    _, scratch, _ = ssba.forward_topk(qg, kg2, vg, desc)
    assert ssba.read_status(desc, scratch) == 5


# ------------------------------------------------ head-shared top-k gate --
SHARED_CASES = [
    preset("grid64", heads=4, gate="topk_shared"),
    preset("grid64_text", batch=2, heads=3, gate="topk_shared"),
    preset("grid128", heads=3, gate="topk_shared"),                       # D 128, 16x16 blocks
    workload_from(batch=1, heads=5, grid_h=128, grid_w=128, head_dim=64, tile=8, keep=30,
                  shift=(-4, 4), gate="topk_shared"),                      # T_b 256
    workload_from(batch=2, heads=2, grid_h=48, grid_w=40, head_dim=64, tile=8, keep=7, shift=(3, 5),
                  n_text=13, gate="topk_shared"),                          # T_b 30
    preset("tiny", gate="topk_shared"),                                    # fp32
]


@pytest.mark.parametrize("w", SHARED_CASES, ids=_ids)
def test_shared_gate_index_bit_exact(w):
    (q, k, _), (qg, kg, _) = inputs(w)
    from paper_2605_15684_amd import ssba
    desc = gpu_desc(w, qg)
    index, scratch = ssba.build_index(qg, kg, desc)
    got = index.cpu().numpy()
    want = oracle_index(w, q, k)
    assert np.array_equal(got, want)
    assert (got == got[:, :1]).all()              # every head holds the same lists
    assert ssba.read_status(desc, scratch) == 0


@pytest.mark.parametrize("w", SHARED_CASES[:2] + SHARED_CASES[-1:], ids=_ids)
def test_shared_gate_forward_topk_and_output(w):
    """forward_topk with the shared gate equals build_index + forward, and the
    output matches the oracle on every row (small) or sampled rows."""
    from paper_2605_15684_amd import ssba
    (q, k, v), (qg, kg, vg) = inputs(w)
    desc = gpu_desc(w, qg)
    index2, _ = ssba.build_index(qg, kg, desc)
    out2 = ssba.forward(qg, kg, vg, index2, desc)
    index1, _, out1 = ssba.forward_topk(qg, kg, vg, desc)
    torch.cuda.synchronize()
    assert torch.equal(index1, index2) and torch.equal(out1, out2)
    want_idx = oracle_index(w, q, k)
    rng = np.random.default_rng(3)
    heads = [(b, h) for b in range(w.batch) for h in range(w.heads)][:4]
    rows = sample_rows(w, rng)
    ref = O.attention(to64(q), to64(k), to64(v), want_idx, rows=rows, heads=heads, **oracle_kw(w))
    assert max_err(out1, ref, heads, rows) <= tol(w)


def test_shared_gate_nonfinite_sets_status():
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=3, gate="topk_shared")
    (_, _, _), (qg, kg, _) = inputs(w)
    desc = gpu_desc(w, qg)
    kg2 = kg.clone()
    kg2[0, 2, 700, 1] = float("inf")
    _, scratch = ssba.build_index(qg, kg2, desc)
    assert ssba.read_status(desc, scratch) == 5


# ------------------------------------------------------------ layer stack --
def _layer_stack(w, keeps, skips, seed0=11):
    """Per-layer seeded inputs (seed seed0 + l) of workload w."""
    layers = []
    for l, (kp, sk) in enumerate(zip(keeps, skips)):
        (q, k, v), (qg, kg, vg) = inputs(w.with_(seed=seed0 + l))
        out = torch.full_like(qg, 7.0)
        layers.append(dict(q=qg, k=kg, v=vg, out=out, keep=kp, skip=sk, cpu=(q, k, v)))
    return layers


@pytest.mark.parametrize("gate,window", [("topk", (1, 1)), ("topk_shared", (1, 1)), ("window", (2, 2)),
                                         ("dense", (1, 1))])
def test_layer_stack_equals_per_layer_calls(gate, window):
    """ssba_forward_layers == one call per layer with the layer's offset
    (negated on odd layers) and keep; skipped layers leave their output
    untouched; static gates reuse one index per offset parity."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2, n_text=0, gate=gate, window=window, shift=(4, 4))
    keeps = [10, 16, 4, 10, 7]
    skips = [False, False, True, False, False]
    layers = _layer_stack(w, keeps, skips)
    desc = gpu_desc(w, layers[0]["q"])
    index, scratch = ssba.forward_layers(layers, desc)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        if L["skip"]:
            assert bool((L["out"] == 7.0).all())
            continue
        sh = (4, 4) if l % 2 == 0 else (-4, -4)
        wl = w.with_(shift=sh, keep=keeps[l])
        dl = gpu_desc(wl, L["q"])
        if gate in ("topk", "topk_shared"):
            idx1, _, out1 = ssba.forward_topk(L["q"], L["k"], L["v"], dl)
            assert torch.equal(index[l], idx1)
        else:
            idx1, _ = ssba.build_index(None, None, dl)
            out1 = ssba.forward(L["q"], L["k"], L["v"], idx1, dl)
        torch.cuda.synchronize()
        assert torch.equal(L["out"], out1), f"layer {l}"
        if gate in ("topk", "topk_shared"):
            dl_status = gpu_desc(wl, L["q"])
            assert ssba.read_status(dl_status, scratch[l]) == 0


@pytest.mark.parametrize("gate,window", [("window", (2, 2)), ("topk_shared", (1, 1))])
def test_layer_stack_16x16_blocks_d128(gate, window):
    """The layer driver's one attention launch over several layers with
    16x16 blocks at head_dim 128 (the 128x128-grid kernels): every layer's
    output equals one call per layer."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2, head_dim=128, tile=16, n_text=0, gate=gate, window=window, shift=(8, 8))
    keeps = [5, 9, 3, 16]
    skips = [False, True, False, False]
    layers = _layer_stack(w, keeps, skips, seed0=50)
    desc = gpu_desc(w, layers[0]["q"])
    index, scratch = ssba.forward_layers(layers, desc)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        if L["skip"]:
            assert bool((L["out"] == 7.0).all())
            continue
        wl = w.with_(shift=(8, 8) if l % 2 == 0 else (-8, -8), keep=keeps[l])
        dl = gpu_desc(wl, L["q"])
        if gate == "topk_shared":
            idx1, _ = ssba.build_index(L["q"], L["k"], dl)
            assert torch.equal(index[l], idx1), f"layer {l}"
        else:
            idx1, _ = ssba.build_index(None, None, dl)
        out1 = ssba.forward(L["q"], L["k"], L["v"], idx1, dl)
        torch.cuda.synchronize()
        assert torch.equal(L["out"], out1), f"layer {l}"


def test_layer_stack_topk_d128():
    """The batched pooling and gated attention launches at head_dim 128
    (8x8 blocks, text tokens): every layer equals one fused call."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2, head_dim=128, grid_h=32, grid_w=48, n_text=20, shift=(4, 4))
    keeps = [3, 11, 24, 1]
    skips = [False, False, True, False]
    layers = _layer_stack(w, keeps, skips, seed0=70)
    desc = gpu_desc(w, layers[0]["q"])
    index, scratch = ssba.forward_layers(layers, desc)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        if L["skip"]:
            assert bool((L["out"] == 7.0).all())
            continue
        wl = w.with_(shift=(4, 4) if l % 2 == 0 else (-4, -4), keep=keeps[l])
        dl = gpu_desc(wl, L["q"])
        idx1, _, out1 = ssba.forward_topk(L["q"], L["k"], L["v"], dl)
        torch.cuda.synchronize()
        assert torch.equal(index[l], idx1), f"layer {l}"
        assert torch.equal(L["out"], out1), f"layer {l}"
        assert ssba.read_status(dl, scratch[l]) == 0


def test_layer_stack_beyond_one_prepass_launch():
    """A stack longer than one batched pooling launch takes (32 layers), with
    skipped layers and text tokens: every layer's index, status and output
    equal one fused call per layer."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=1, grid_h=32, grid_w=32, n_text=13, shift=(4, 4))
    n = 37
    keeps = [1 + (5 * l) % 16 for l in range(n)]
    skips = [l % 6 == 5 for l in range(n)]
    layers = _layer_stack(w, keeps, skips, seed0=100)
    desc = gpu_desc(w, layers[0]["q"])
    index, scratch = ssba.forward_layers(layers, desc)
    torch.cuda.synchronize()
    for l, L in enumerate(layers):
        if L["skip"]:
            assert bool((L["out"] == 7.0).all())
            continue
        wl = w.with_(shift=(4, 4) if l % 2 == 0 else (-4, -4), keep=keeps[l])
        dl = gpu_desc(wl, L["q"])
        idx1, _, out1 = ssba.forward_topk(L["q"], L["k"], L["v"], dl)
        torch.cuda.synchronize()
        assert torch.equal(index[l], idx1), f"layer {l}"
        assert torch.equal(L["out"], out1), f"layer {l}"
        assert ssba.read_status(dl, scratch[l]) == 0


def test_layer_stack_against_oracle_and_status():
    """Three layers at the 64x64 size against the oracle's layer stack
    (sampled rows), with a NaN in layer 1 reported by that layer's scratch
    slice only."""
    from paper_2605_15684_amd import ssba
    w = preset("grid64", heads=2)
    keeps, skips = [10, 12, 8], [False, False, False]
    layers = _layer_stack(w, keeps, skips, seed0=21)
    layers[1]["k"][0, 1, 333, 7] = float("nan")
    desc = gpu_desc(w, layers[0]["q"])
    index, scratch = ssba.forward_layers(layers, desc)
    torch.cuda.synchronize()
    statuses = [ssba.read_status(desc, scratch[l]) for l in range(3)]
    assert statuses == [0, 5, 0]
    ol = [dict(q=to64(L["cpu"][0]), k=to64(L["cpu"][1]), v=to64(L["cpu"][2]), keep=L["keep"])
          for L in layers]
    for l in (0, 2):   # the NaN layer is only checked through its status
        sh = O.layer_shift(l, w.tile)
        want_idx = O.build_index(ol[l]["q"], ol[l]["k"], gate="topk", keep=keeps[l], grid_h=w.grid_h,
                                 grid_w=w.grid_w, tile=w.tile, shift=sh, n_text=0)
        assert np.array_equal(index[l].cpu().numpy(), want_idx)
        rng = np.random.default_rng(l)
        wl = w.with_(shift=sh)
        rows = sample_rows(wl, rng, n_random=32)
        heads = [(0, 0), (0, 1)]
        ref = O.attention(ol[l]["q"], ol[l]["k"], ol[l]["v"], want_idx, rows=rows, heads=heads,
                          **oracle_kw(wl))
        assert max_err(layers[l]["out"], ref, heads, rows) <= BF16_TOL
