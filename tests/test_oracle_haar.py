"""Pins for the Haar oracle (Section 2.3.1: the 2-D Haar kernel bank applied
level after level, and the inverse pyramid).  Checks: the transform written
as a Kronecker product of 1-D orthonormal Haar matrices (an independent
statement), perfect reconstruction, energy preservation, images whose bands
follow by reasoning, and a hand-computed cell."""
import numpy as np
import pytest

from oracle import haar_oracle as H


def _haar_1d(n: int) -> np.ndarray:
    """Rows 0..n/2-1: pair sums / sqrt(2); rows n/2..n-1: pair differences / sqrt(2)."""
    m = np.zeros((n, n))
    for i in range(n // 2):
        m[i, 2 * i] = m[i, 2 * i + 1] = 1 / np.sqrt(2)
        m[n // 2 + i, 2 * i] = 1 / np.sqrt(2)
        m[n // 2 + i, 2 * i + 1] = -1 / np.sqrt(2)
    return m


@pytest.mark.parametrize("h,w", [(2, 2), (4, 6), (8, 8), (6, 10)])
def test_one_level_equals_kronecker_matrices(h, w):
    """Y = A_h X A_w^T with 1-D Haar matrices: the quadrant (low rows, low
    cols) is LL, (low rows, high cols) HL (high-pass along the width), (high
    rows, low cols) LH, (high rows, high cols) HH."""
    rng = np.random.default_rng(h * 31 + w)
    x = rng.standard_normal((h, w))
    y = _haar_1d(h) @ x @ _haar_1d(w).T
    got = H.dwt_level(x)
    hh, ww = h // 2, w // 2
    np.testing.assert_allclose(got[0], y[:hh, :ww], atol=1e-13)
    np.testing.assert_allclose(got[1], y[:hh, ww:], atol=1e-13)
    np.testing.assert_allclose(got[2], y[hh:, :ww], atol=1e-13)
    np.testing.assert_allclose(got[3], y[hh:, ww:], atol=1e-13)


def test_hand_cell():
    x = np.array([[1.0, 2.0], [3.0, 5.0]])
    got = H.dwt_level(x)[:, 0, 0]
    assert got.tolist() == [5.5, -1.5, -2.5, 0.5]
    assert H.iwt_level(got[:, None, None]).tolist() == x.tolist()


@pytest.mark.parametrize("levels", [1, 2, 3])
def test_perfect_reconstruction_and_energy(levels):
    rng = np.random.default_rng(levels)
    x = rng.standard_normal((2, 3, 16, 24))
    w = H.dwt(x, levels)
    for l, wl in enumerate(w, start=1):
        assert wl.shape == (2, 12, 16 >> l, 24 >> l)
    np.testing.assert_allclose(H.iwt(w), x, atol=1e-12)
    # Orthonormal bank: the coarsest level plus every finer level's details
    # carry the input's energy.
    energy = np.sum(w[-1] ** 2)
    for wl in w[:-1]:
        energy += np.sum(wl.reshape(2, 3, 4, *wl.shape[-2:])[:, :, 1:] ** 2)
    assert np.isclose(energy, np.sum(x ** 2), rtol=1e-12)


def test_constant_and_ramps_land_in_the_expected_bands():
    const = np.full((1, 1, 8, 8), 3.0)
    w = H.dwt(const, 3)
    for l, wl in enumerate(w, start=1):
        b = wl.reshape(1, 1, 4, *wl.shape[-2:])
        assert np.all(b[:, :, 0] == 3.0 * 2 ** l)        # LL doubles per level
        assert np.all(b[:, :, 1:] == 0)
    xs = np.tile(np.arange(8.0), (8, 1))                  # ramp along the width
    b = H.dwt_level(xs)
    assert np.all(b[1] == -1.0) and np.all(b[2] == 0) and np.all(b[3] == 0)
    ys = xs.T.copy()                                      # ramp along the height
    b = H.dwt_level(ys)
    assert np.all(b[2] == -1.0) and np.all(b[1] == 0) and np.all(b[3] == 0)
    cb = (np.indices((8, 8)).sum(axis=0) % 2) * 2.0 - 1.0  # checkerboard
    b = H.dwt_level(cb)
    assert np.all(b[3] == -2.0) and np.all(b[:3] == 0)


def test_levels_transform_the_unrounded_ll_and_residuals_add():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((1, 2, 8, 8))
    w = H.dwt(x, 2)
    ll1 = w[0].reshape(1, 2, 4, 4, 4)[:, :, 0]
    np.testing.assert_array_equal(w[1], H.dwt(ll1, 1)[0])
    r0 = rng.standard_normal((1, 2, 8, 8))
    r1 = rng.standard_normal((1, 2, 4, 4))
    got = H.iwt(w, [r0, r1])
    # residual of level 1 enters the LL that the finest level inverts
    w1 = w[0].reshape(1, 2, 4, 4, 4).copy()
    w1[:, :, 0] = ll1 + r1
    want = H.iwt_level(w1) + r0
    np.testing.assert_allclose(got, want, atol=1e-12)


def test_reading_of_the_band_subscript_matches_the_stated_shape():
    """The DWT equation writes level l as the Haar bank applied to W^(l-1)_c
    with c = {LL, HL, LH}, and gives W^(l) 4C channels at H/2^l x W/2^l for
    every l with one C.  Reading: level l transforms the LL band of level
    l - 1 (the Mallat pyramid); c names the bands the encoder keeps from each
    level (all four are stored).  Pinned two ways:
      * the pyramid written with 1-D Haar matrices -- level 2 is the
        Kronecker transform of level 1's low/low quadrant -- equals the
        oracle's level 2, band by band;
      * the shapes: the oracle's level l has 4C channels for every l, while
        transforming the three bands {LL, HL, LH} of level 1 would give 12C
        channels at level 2, which the stated shape rules out."""
    rng = np.random.default_rng(11)
    c, h, w_ = 2, 16, 16
    x = rng.standard_normal((1, c, h, w_))
    lv = H.dwt(x, 3)
    for l, wl in enumerate(lv, start=1):
        assert wl.shape == (1, 4 * c, h >> l, w_ >> l)
    for ch in range(c):
        y1 = _haar_1d(h) @ x[0, ch] @ _haar_1d(w_).T                 # level 1, quadrant form
        ll1 = y1[: h // 2, : w_ // 2]
        y2 = _haar_1d(h // 2) @ ll1 @ _haar_1d(w_ // 2).T            # level 2 from LL only
        q = h // 4
        got = lv[1][0, 4 * ch: 4 * ch + 4]
        np.testing.assert_allclose(got[0], y2[:q, :q], atol=1e-12)   # LL
        np.testing.assert_allclose(got[1], y2[:q, q:], atol=1e-12)   # HL
        np.testing.assert_allclose(got[2], y2[q:, :q], atol=1e-12)   # LH
        np.testing.assert_allclose(got[3], y2[q:, q:], atol=1e-12)   # HH
    # The other reading: the bank applied to the three kept bands of level 1.
    kept = lv[0].reshape(1, c, 4, h // 2, w_ // 2)[:, :, :3].reshape(1, 3 * c, h // 2, w_ // 2)
    other = H.dwt(kept, 1)[0]
    assert other.shape[1] == 12 * c != 4 * c
