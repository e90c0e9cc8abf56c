"""Pins of the oracle's rotary step (Algorithm 1, first step; 2-D axial
reading) and of its bf16 rounding, against facts that do not restate the
oracle's formula: a hand-worked case, complex arithmetic, the rotation's
invariants, the relative-position property of rotary embeddings and torch's
own bf16 conversion."""
import numpy as np
import pytest
import torch

from oracle import ssba_oracle as O


def _rng(seed=0):
    return np.random.default_rng(seed)


def test_hand_worked_d4():
    # D 4: one pair per half, angle = position (theta**0 = 1).  Token (y 1, x 2)
    # of a 4 x 6 grid, vector (1, 0, 1, 0) -> (cos 1, sin 1, cos 2, sin 2).
    x = np.zeros((1, 1, 24, 4))
    x[..., 0] = 1.0
    x[..., 2] = 1.0
    r = O.rope_2d(x, grid_h=4, grid_w=6)
    assert np.allclose(r[0, 0, 1 * 6 + 2], [0.5403023058681398, 0.8414709848078965,
                                            -0.4161468365471424, 0.9092974268256817], atol=1e-15)
    # (0, 1, 0, 1) at the same token -> (-sin 1, cos 1, -sin 2, cos 2)
    y = np.zeros((1, 1, 24, 4))
    y[..., 1] = 1.0
    y[..., 3] = 1.0
    r = O.rope_2d(y, grid_h=4, grid_w=6)
    assert np.allclose(r[0, 0, 8], [-0.8414709848078965, 0.5403023058681398,
                                    -0.9092974268256817, -0.4161468365471424], atol=1e-15)


def test_row_drives_first_half_column_second():
    # A token in row 0 keeps its first half; a token in column 0 keeps its second.
    x = _rng(1).standard_normal((1, 1, 8 * 8, 16))
    r = O.rope_2d(x, grid_h=8, grid_w=8)
    row0 = np.arange(8)            # y = 0, x = 0..7
    col0 = np.arange(0, 64, 8)     # x = 0, y = 0..7
    assert np.array_equal(r[0, 0, row0, :8], x[0, 0, row0, :8])
    assert np.array_equal(r[0, 0, col0, 8:], x[0, 0, col0, 8:])
    assert not np.allclose(r[0, 0, row0[1:], 8:], x[0, 0, row0[1:], 8:])
    assert not np.allclose(r[0, 0, col0[1:], :8], x[0, 0, col0[1:], :8])


def test_equals_complex_multiplication():
    # Pair (a, b) of a half as a + ib times exp(i * pos * theta**(-i/(D/4))),
    # with numpy's complex exponential.
    gh, gw, d, theta = 6, 10, 32, 500.0
    x = _rng(2).standard_normal((2, 3, gh * gw, d))
    r = O.rope_2d(x, grid_h=gh, grid_w=gw, theta=theta)
    ids = np.arange(gh * gw)
    for pos, c0 in ((ids // gw, 0), (ids % gw, d // 2)):
        z = x[..., c0:c0 + d // 2:2] + 1j * x[..., c0 + 1:c0 + d // 2:2]
        freq = np.power(theta, -np.arange(d // 4) / (d // 4))
        w = z * np.exp(1j * np.outer(pos, freq))
        assert np.allclose(r[..., c0:c0 + d // 2:2], w.real, atol=1e-13)
        assert np.allclose(r[..., c0 + 1:c0 + d // 2:2], w.imag, atol=1e-13)


def test_pair_norms_kept_and_text_untouched():
    n_text, gh, gw, d = 5, 4, 4, 16
    x = _rng(3).standard_normal((1, 2, n_text + gh * gw, d))
    r = O.rope_2d(x, grid_h=gh, grid_w=gw, n_text=n_text)
    assert np.array_equal(r[..., :n_text, :], x[..., :n_text, :])
    n0 = x[..., 0::2] ** 2 + x[..., 1::2] ** 2
    n1 = r[..., 0::2] ** 2 + r[..., 1::2] ** 2
    assert np.allclose(n0, n1, rtol=1e-13)


def test_relative_position_property():
    # <R(p) q, R(p') k> depends on p - p' only: moving both tokens by the same
    # (dy, dx) leaves every query-key dot product unchanged.
    gh, gw, d = 12, 12, 64
    rng = _rng(4)
    q, k = rng.standard_normal(d), rng.standard_normal(d)

    def dot(p1, p2):
        x = np.zeros((1, 1, gh * gw, d))
        x[0, 0, p1[0] * gw + p1[1]] = q
        y = np.zeros((1, 1, gh * gw, d))
        y[0, 0, p2[0] * gw + p2[1]] = k
        rq = O.rope_2d(x, grid_h=gh, grid_w=gw)[0, 0, p1[0] * gw + p1[1]]
        rk = O.rope_2d(y, grid_h=gh, grid_w=gw)[0, 0, p2[0] * gw + p2[1]]
        return float(rq @ rk)

    base = dot((2, 3), (5, 1))
    for dy, dx in ((1, 0), (0, 4), (6, 7), (-2, 2)):
        assert dot((2 + dy, 3 + dx), (5 + dy, 1 + dx)) == pytest.approx(base, abs=1e-11)
    assert dot((2, 3), (5, 2)) != pytest.approx(base, abs=1e-6)   # a different offset differs


def test_round_bf16_matches_torch_on_fp32_values():
    # For fp64 values that are fp32 numbers, torch's fp32 -> bf16 conversion
    # (round to nearest even) is the same single rounding.
    rng = _rng(5)
    f32 = (rng.standard_normal(20000) * np.exp2(rng.integers(-20, 20, 20000))).astype(np.float32)
    # exact ties: 8 significant bits plus a half
    ties = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 3.0 + 2.0 ** -7], np.float32)
    f32 = np.concatenate([f32, ties])
    want = torch.from_numpy(f32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.round_bf16(f32.astype(np.float64)), want)


def test_round_bf16_direct_from_fp64():
    # A value just above a bf16 midpoint rounds up, although the nearest fp32
    # is the midpoint itself (which would round to even, down): one rounding.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert np.float32(x) == np.float32(1.0 + 2.0 ** -8)
    assert O.round_bf16(np.array([x]))[0] == 1.0 + 2.0 ** -7
    assert O.round_bf16(np.array([0.0, -0.0, 1.5, -3.0]))[2] == 1.5


def test_ssba_rope_is_ssba_on_rounded_rotations():
    gh = gw = 16
    rng = _rng(6)
    q, k, v = (torch.from_numpy(rng.standard_normal((1, 2, gh * gw, 64))).to(torch.bfloat16)
               .double().numpy() for _ in range(3))
    qr, kr, idx, o = O.ssba_rope(q, k, v, grid_h=gh, grid_w=gw, tile=4, shift=(2, 2), keep=5)
    assert np.array_equal(O.round_bf16(qr), qr) and np.array_equal(O.round_bf16(kr), kr)
    idx2, o2 = O.ssba(qr, kr, v, grid_h=gh, grid_w=gw, tile=4, shift=(2, 2), keep=5)
    assert np.array_equal(idx, idx2) and np.array_equal(o, o2)
    assert not np.array_equal(qr, q)
