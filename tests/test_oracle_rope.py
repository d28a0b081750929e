"""Pins for the oracle's rotary encoding (Sec. 3.3: keys keep the rotation of
their original position).  Each check comes from the mathematics of a
rotation, not from re-typing the oracle's formula."""
import numpy as np
import pytest

from oracle import rope


def test_position_zero_is_identity():
    x = np.random.default_rng(0).standard_normal((5, 3, 64))
    np.testing.assert_array_equal(rope.rotate(x, np.zeros(5, np.int64), 1e6), x)


def test_hand_worked_rotate_half_d4():
    # D = 4, theta = 100: pair 0 rotates by pos, pair 1 by pos / 10 (= pos*100^(-1/2)).
    # x = e_0 -> (cos p, 0, sin p, 0); x = e_1 -> (0, cos(p/10), 0, sin(p/10)).
    p = 3
    e0 = np.array([1.0, 0, 0, 0])
    e1 = np.array([0, 1.0, 0, 0])
    np.testing.assert_allclose(rope.rotate(e0, np.array(p), 100.0),
                               [np.cos(3), 0, np.sin(3), 0], atol=1e-15)
    np.testing.assert_allclose(rope.rotate(e1, np.array(p), 100.0),
                               [0, np.cos(0.3), 0, np.sin(0.3)], atol=1e-15)
    # the upper half rotates the other way round: e_2 -> (-sin p, 0, cos p, 0)
    e2 = np.array([0, 0, 1.0, 0])
    np.testing.assert_allclose(rope.rotate(e2, np.array(p), 100.0),
                               [-np.sin(3), 0, np.cos(3), 0], atol=1e-15)


def test_matches_complex_multiplication():
    # rotate-half is multiplication of z_i = x_i + i x_{i+D/2} by exp(i pos theta^(-2i/D))
    rng = np.random.default_rng(1)
    D, theta = 128, 1e6
    x = rng.standard_normal((7, D))
    pos = rng.integers(0, 80_000, 7)
    z = x[:, :D // 2] + 1j * x[:, D // 2:]
    freq = np.array([theta ** (-(2.0 * i) / D) for i in range(D // 2)])
    zr = z * np.exp(1j * pos[:, None] * freq[None, :])
    want = np.concatenate([zr.real, zr.imag], axis=1)
    # angles reach ~8e4 rad, where a 1-ulp frequency difference moves the result by ~1e-11
    np.testing.assert_allclose(rope.rotate(x, pos, theta), want, rtol=0, atol=1e-10)


def test_pair_norms_preserved():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((9, 4, 128))
    y = rope.rotate(x, rng.integers(0, 10_000, 9), 1e6)
    nx = x[..., :64] ** 2 + x[..., 64:] ** 2
    ny = y[..., :64] ** 2 + y[..., 64:] ** 2
    np.testing.assert_allclose(nx, ny, rtol=1e-13)


def test_composition_adds_positions():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((6, 64))
    a, b = rng.integers(0, 5000, 6), rng.integers(0, 5000, 6)
    np.testing.assert_allclose(rope.rotate(rope.rotate(x, a, 1e4), b, 1e4),
                               rope.rotate(x, a + b, 1e4), atol=1e-11)


def test_dot_product_depends_only_on_offset():
    # the relative-position property that makes kept keys valid without re-encoding
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    d1 = rope.rotate(q, np.array(900), 1e6) @ rope.rotate(k, np.array(850), 1e6)
    d2 = rope.rotate(q, np.array(50_050), 1e6) @ rope.rotate(k, np.array(50_000), 1e6)
    assert d1 == pytest.approx(d2, abs=1e-9)


def test_frequencies():
    f = rope.inverse_frequencies(128, 1e6)
    assert f[0] == 1.0
    assert f[-1] == pytest.approx(1e6 ** (-126 / 128), rel=1e-14)
    assert np.all(np.diff(f) < 0)
