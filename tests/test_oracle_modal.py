"""Pins of the oracle's modal filter, the implicit filter of order M of the
appendix "Filter Generation": k[c, t] = Re sum_m R[c, m] lambda[c, m]^t with
lambda = exp(a + i theta).  Checked against printed values (a halving real
pole, a quarter-turn pole), the geometric-series sum computed with numpy's
complex arithmetic, the second-order recurrence every damped cosine obeys,
conjugate-pair symmetry, linearity in the residues and mode relabelling."""
import math

import numpy as np
import pytest

import oracle


def test_real_pole_halves():
    """theta = 0: the imaginary residue drops out and lambda^t = 2^-t."""
    k = oracle.modal_filter([[math.log(0.5)]], [[0.0]], [[3.0]], [[7.0]], 6)
    assert np.allclose(k[0], [3.0, 1.5, 0.75, 0.375, 0.1875, 0.09375], rtol=1e-15, atol=0)


def test_quarter_turn_pole():
    """|lambda| = 1, theta = pi/2, R = 1 - 2i: Re((1 - 2i) i^t) = 1, 2, -1, -2, ..."""
    k = oracle.modal_filter([[0.0]], [[math.pi / 2]], [[1.0]], [[-2.0]], 8)
    assert np.allclose(k[0], [1, 2, -1, -2, 1, 2, -1, -2], rtol=0, atol=1e-14)


def _params(seed, C, M):
    rng = np.random.default_rng(seed)
    a = -np.exp(rng.uniform(np.log(1e-3), np.log(0.3), (C, M)))
    th = rng.uniform(0.0, np.pi, (C, M))
    return a, th, rng.standard_normal((C, M)), rng.standard_normal((C, M))


def test_geometric_series_sum():
    """sum_{t < L} Re(R lambda^t) = Re(R (1 - lambda^L) / (1 - lambda)), per mode and summed."""
    a, th, re, im = _params(1, 3, 5)
    L = 300
    k = oracle.modal_filter(a, th, re, im, L)
    lam = np.exp(a + 1j * th)
    R = re + 1j * im
    expect = np.real(R * (1 - lam ** L) / (1 - lam)).sum(axis=1)
    assert np.allclose(k.sum(axis=1), expect, rtol=1e-11, atol=1e-12)


def test_second_order_recurrence():
    """One mode is a damped cosine: k[t + 2] = 2 |lambda| cos(theta) k[t + 1] - |lambda|^2 k[t]."""
    a, th, re, im = _params(2, 4, 1)
    k = oracle.modal_filter(a, th, re, im, 200)
    r = np.exp(a)
    lhs = k[:, 2:]
    rhs = 2 * r * np.cos(th) * k[:, 1:-1] - r * r * k[:, :-2]
    assert np.allclose(lhs, rhs, rtol=1e-10, atol=1e-13)


def test_conjugate_pair():
    """Re(R lambda^t) is unchanged by conjugating both pole and residue."""
    a, th, re, im = _params(3, 2, 4)
    k1 = oracle.modal_filter(a, th, re, im, 64)
    k2 = oracle.modal_filter(a, -th, re, -im, 64)
    assert np.allclose(k1, k2, rtol=1e-13, atol=1e-14)


def test_linear_in_residues_and_mode_order():
    a, th, re, im = _params(4, 3, 6)
    re2, im2 = np.random.default_rng(5).standard_normal((2, 3, 6))
    k = lambda r, i: oracle.modal_filter(a, th, r, i, 50)
    assert np.allclose(k(2 * re - re2, 2 * im - im2), 2 * k(re, im) - k(re2, im2), rtol=1e-12, atol=1e-13)
    perm = np.array([3, 0, 5, 1, 4, 2])
    kp = oracle.modal_filter(a[:, perm], th[:, perm], re[:, perm], im[:, perm], 50)
    assert np.allclose(kp, k(re, im), rtol=1e-12, atol=1e-13)


def test_long_filter_phase_is_exact():
    """At t = 2^20 the phase t * theta of an fp32 angle is exact in double:
    theta = 2 pi / 2^10 rounded to fp32, sampled every 2^10 steps, returns to
    the same point of the circle as t * theta mod 2 pi says."""
    th = float(np.float32(2 * np.pi / 1024))
    L = (1 << 20) + 1
    k = oracle.modal_filter([[0.0]], [[th]], [[1.0]], [[0.0]], L)[0]
    t = np.arange(0, L, 1 << 16)
    expect = np.cos(np.mod(t.astype(np.float64) * th, 2 * np.pi))
    assert np.allclose(k[t], expect, rtol=0, atol=1e-12)


def test_argument_checks():
    with pytest.raises(ValueError):
        oracle.modal_filter(np.zeros((2, 3)), np.zeros((2, 4)), np.zeros((2, 3)), np.zeros((2, 3)), 8)
