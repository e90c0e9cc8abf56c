"""Pins for the oracle's affinity and gates (Section 2.2.1: affinity
S = q_b k_b^T, Top-k Gating with k = floor(T_b * rho); window and dense
controls).  Checks: a matmul library call, constructed inputs whose kept sets
follow by reasoning, exhaustive per-row ordering, ties, and the sparsity the
paper prints in Table 2."""
import os

import numpy as np
import pytest

from oracle import ssba_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tile_map(grid, tile, sy, sx):
    nx = grid // tile
    out = np.empty(grid * grid, dtype=np.int64)
    for y in range(grid):
        for x in range(grid):
            y2, x2 = (y + sy) % grid, (x + sx) % grid
            out[y * grid + x] = (y2 // tile) * nx + x2 // tile
    return out


def test_affinity_matches_matmul():
    rng = np.random.default_rng(0)
    qb = rng.standard_normal((2, 3, 16, 32))
    kb = rng.standard_normal((2, 3, 16, 32))
    np.testing.assert_allclose(O.affinity(qb, kb), qb @ np.swapaxes(kb, -1, -2),
                               rtol=1e-12, atol=1e-12)


def test_affinity_orientation_and_frame_constructed():
    """Query block i pools to a_i * e0 (a_i = +1 even, -1 odd), key block j to
    (j + 1) * e0 (token level, in the shifted frame).  Row i of S is then
    a_i * (j + 1) * Bt^4: even rows keep the largest j, odd rows the smallest.
    A transposed S, an unshifted frame or a flipped ranking fails this."""
    grid, tile, sy, sx, keep, c = 16, 4, 2, -2, 3, 4
    tb = (grid // tile) ** 2
    tmap = _tile_map(grid, tile, sy, sx)
    q = np.zeros((1, 1, grid * grid, c))
    k = np.zeros((1, 1, grid * grid, c))
    for tok in range(grid * grid):
        t = tmap[tok]
        q[0, 0, tok, 0] = 1.0 if t % 2 == 0 else -1.0
        k[0, 0, tok, 0] = float(t + 1)
    idx = O.build_index(q, k, grid_h=grid, grid_w=grid, tile=tile, shift=(sy, sx),
                        gate="topk", keep=keep)
    for i in range(tb):
        want = list(range(tb - keep, tb)) if i % 2 == 0 else list(range(keep))
        assert idx[0, 0, i, 0] == keep
        assert idx[0, 0, i, 1:1 + keep].tolist() == want
        assert (idx[0, 0, i, 1 + keep:] == -1).all()


def _check_row(s_row, kept, keep):
    tb = s_row.size
    assert len(kept) == keep and list(kept) == sorted(kept)
    dropped = sorted(set(range(tb)) - set(kept))
    for a in kept:
        for b in dropped:
            assert s_row[a] > s_row[b] or (s_row[a] == s_row[b] and a < b)


@pytest.mark.parametrize("tb,keep", [(16, 4), (16, 1), (16, 16), (64, 10), (64, 7), (9, 5)])
def test_topk_row_exhaustive(tb, keep):
    rng = np.random.default_rng(tb * 100 + keep)
    for _ in range(50):
        s = rng.standard_normal(tb)
        s[rng.integers(0, tb, 3)] = s[rng.integers(0, tb)]          # inject ties
        _check_row(s, O.gate_topk_row(s, keep), keep)


def test_topk_ties_keep_lowest_indices():
    s = np.full(16, 0.25)
    assert O.gate_topk_row(s, 5).tolist() == [0, 1, 2, 3, 4]
    z = np.array([0.0, -0.0, 0.0, -0.0, -1.0, 1.0])
    assert O.gate_topk_row(z, 3).tolist() == [0, 1, 5]                # +0 == -0


def test_topk_keep_one_is_argmax():
    rng = np.random.default_rng(11)
    for _ in range(100):
        s = np.round(rng.standard_normal(12), 1)
        assert O.gate_topk_row(s, 1).tolist() == [int(np.argmax(s))]


def test_topk_constant_key_blocks_keep_first():
    """K constant inside every block and equal across blocks -> every S row is
    constant -> the kept set is the first `keep` blocks."""
    grid, tile = 16, 4
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 2, grid * grid, 8))
    k = np.tile(rng.standard_normal(8), (1, 2, grid * grid, 1))
    idx = O.build_index(q, k, grid_h=grid, grid_w=grid, tile=tile, shift=(2, 2), keep=6)
    assert (idx[..., 1:7] == np.arange(6)).all() and (idx[..., 0] == 6).all()


def test_paper_sparsity_fraction():
    line = [l for l in open(os.path.join(GOLDEN, "paper_sparsity.txt")) if not l.startswith("#")][0]
    cfg = dict(kv.split("=") for kv in line.split())
    grid, block = int(cfg["grid"]), int(cfg["block"])
    assert grid * grid == int(cfg["tokens"])
    tb = (grid // block) ** 2
    assert tb == int(cfg["n_blocks"])
    keep = O.keep_from_rho(tb, float(cfg["rho"]))
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 1, grid * grid, 64))
    k = rng.standard_normal((1, 1, grid * grid, 64))
    idx = O.build_index(q, k, grid_h=grid, grid_w=grid, tile=block, shift=(4, 4), keep=keep)
    masked = 1.0 - idx[..., 0].sum() / float(tb * tb)
    assert round(100.0 * masked, 2) == float(cfg["sparsity_percent"])


@pytest.mark.parametrize("tb,rho,keep", [(64, 0.84375, 10), (64, 0.84, 11), (64, 0.9, 7),
                                         (64, 0.0, 64), (64, 0.75, 16), (64, 0.9375, 4)])
def test_keep_from_rho(tb, rho, keep):
    assert O.keep_from_rho(tb, rho) == keep


def test_window_gate_special_cases():
    ny, nx = 4, 6
    diag = O.gate_window(ny, nx, 1, 1)
    assert all(l.tolist() == [i] for i, l in enumerate(diag))
    full = O.gate_window(ny, nx, ny, nx)
    assert all(l.tolist() == list(range(ny * nx)) for l in full)
    w = O.gate_window(ny, nx, 2, 3)
    g = np.zeros((ny * nx, ny * nx), bool)
    for i, l in enumerate(w):
        g[i, l] = True
        assert len(l) == 6
    assert (g == g.T).all() and (g @ g.astype(int) > 0).sum() == g.sum()   # equivalence classes


def test_index_layout_dense_and_window():
    q = np.zeros((2, 1, 64, 4))
    idx = O.build_index(q, q, grid_h=8, grid_w=8, tile=4, gate="dense")
    assert idx.shape == (2, 1, 4, 5) and idx.dtype == np.int32
    assert (idx[..., 0] == 4).all() and (idx[..., 1:] == np.arange(4)).all()
    idx = O.build_index(q, q, grid_h=8, grid_w=8, tile=4, gate="window", window=(1, 2))
    assert idx[0, 0, 0].tolist() == [2, 0, 1, -1, -1]
    assert idx[0, 0, 3].tolist() == [2, 2, 3, -1, -1]
    with pytest.raises(ValueError):
        O.build_index(q, q, grid_h=8, grid_w=8, tile=4, gate="topk", keep=0)


# --------------------------------------------------------------------------
# Head-shared gate (the gate variant whose score is the sum over heads of the
# per-head affinities) and the layer stack (Section 2.2.2 alternation).
# --------------------------------------------------------------------------
def _int_bruteforce_shared(q, k, grid, tile, shift, keep, n_text=0):
    """Pure-integer reference: pooled sums, products and sums are exact, so
    any order gives the same S; kept lists by sorting (-S, j)."""
    b_n, h_n, _, c_n = q.shape
    tmap = _tile_map(grid, tile, shift[0], shift[1])
    tb = (grid // tile) ** 2
    out = []
    for b in range(b_n):
        s = [[0] * tb for _ in range(tb)]
        for h in range(h_n):
            qb = [[0] * c_n for _ in range(tb)]
            kb = [[0] * c_n for _ in range(tb)]
            for tok in range(grid * grid):
                t = int(tmap[tok])
                for c in range(c_n):
                    qb[t][c] += int(q[b, h, n_text + tok, c])
                    kb[t][c] += int(k[b, h, n_text + tok, c])
            for i in range(tb):
                for j in range(tb):
                    s[i][j] += sum(qb[i][c] * kb[j][c] for c in range(c_n))
        out.append([sorted(sorted(range(tb), key=lambda j: (-s[i][j], j))[:keep]) for i in range(tb)])
    return out


@pytest.mark.parametrize("shift,keep,n_text", [((2, 2), 4, 0), ((-2, -2), 5, 3), ((1, 3), 1, 0)])
def test_shared_gate_integer_bruteforce(shift, keep, n_text):
    grid, tile = 8, 2
    rng = np.random.default_rng(keep * 7 + n_text)
    q = rng.integers(-3, 4, size=(2, 3, n_text + grid * grid, 4)).astype(np.float64)
    k = rng.integers(-3, 4, size=(2, 3, n_text + grid * grid, 4)).astype(np.float64)
    idx = O.build_index(q, k, grid_h=grid, grid_w=grid, tile=tile, shift=shift, n_text=n_text,
                        gate="topk_shared", keep=keep)
    ref = _int_bruteforce_shared(q, k, grid, tile, shift, keep, n_text)
    for b in range(2):
        for h in range(3):
            for i in range(16):
                assert idx[b, h, i, 0] == keep
                assert idx[b, h, i, 1:1 + keep].tolist() == ref[b][i]
                assert (idx[b, h, i, 1 + keep:] == -1).all()


def test_shared_gate_one_head_equals_per_head_gate():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((2, 1, 256, 8))
    k = rng.standard_normal((2, 1, 256, 8))
    kw = dict(grid_h=16, grid_w=16, tile=4, shift=(2, 2), keep=5)
    assert (O.build_index(q, k, gate="topk_shared", **kw) == O.build_index(q, k, gate="topk", **kw)).all()


def test_shared_affinity_adds_heads_in_order():
    """Three heads whose per-head scores are 1, 2^-53 and 2^-53: left to
    right the two tiny terms each round away (1 + 2^-53 = 1 in fp64, ties to
    even); any other order would keep them (2^-52 + 1 is exact)."""
    s = np.zeros((1, 3, 1, 1))
    s[0, :, 0, 0] = [1.0, 2.0 ** -53, 2.0 ** -53]
    assert O.shared_affinity(s)[0, 0, 0] == 1.0


def test_layer_stack_alternates_shift_and_skips():
    grid, tile = 16, 4
    rng = np.random.default_rng(9)
    mk = lambda: rng.standard_normal((1, 2, grid * grid, 8))
    layers = [dict(q=mk(), k=mk(), v=mk(), keep=k) for k in (3, 6, 2)]
    layers[1]["skip"] = True
    res = O.ssba_layers(layers, grid_h=grid, grid_w=grid, tile=tile)
    assert res[1] is None
    for l in (0, 2):
        sh = O.layer_shift(l, tile)
        ref = O.ssba(layers[l]["q"], layers[l]["k"], layers[l]["v"], grid_h=grid, grid_w=grid,
                     tile=tile, shift=sh, keep=layers[l]["keep"])
        assert (res[l][0] == ref[0]).all() and np.array_equal(res[l][1], ref[1])
    # an odd layer takes the negated offset: (-2, -2) here
    layers[1]["skip"] = False
    res = O.ssba_layers(layers, grid_h=grid, grid_w=grid, tile=tile)
    ref = O.build_index(layers[1]["q"], layers[1]["k"], grid_h=grid, grid_w=grid, tile=tile,
                        shift=(-2, -2), keep=6)
    assert (res[1][0] == ref).all()
