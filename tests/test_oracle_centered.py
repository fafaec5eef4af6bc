"""Pins of the oracle's centered mode: the kernel on the double grid of the
paper's non-circular convolution (section 3.2.1, "Support for circular and
non-circular convolutions": the kernel is evaluated on (2 L_d - 1) points per
axis and the input zero-padded to that size).  kc index L_d - 1 is the zero
displacement:

    y[n] = x2[n] * (sum_m kc[n - m + (L - 1)] u[m] + D[c] u[n]),  u = x1 v.

Checked against scipy's N-D linear convolution (a library routine outside
the oracle), between the oracle's two evaluations, against the causal
("linear") mode for a kernel that vanishes at negative displacements, for the
centre impulse, and for the mirror symmetry of the definition."""
import numpy as np
import pytest
from scipy import signal

import oracle


def _case(B, C, grid, seed):
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    x1, x2, v = (rng.standard_normal(shape) for _ in range(3))
    kc = rng.standard_normal(oracle.kernel_shape(shape, "centered"))
    D = rng.standard_normal(C)
    return x1, x2, v, kc, D


def _scipy_reference(x1, x2, v, kc, D):
    B, C = x1.shape[:2]
    grid = x1.shape[2:]
    y = np.empty_like(x1)
    for b in range(B):
        for c in range(C):
            u = x1[b, c] * v[b, c]
            full = signal.convolve(u, kc[b, c], mode="full", method="direct")
            sl = tuple(slice(L - 1, 2 * L - 1) for L in grid)
            y[b, c] = x2[b, c] * (full[sl] + D[c] * u)
    return y


@pytest.mark.parametrize("grid", [(1,), (2,), (5,), (16,), (3, 4), (8, 8), (2, 3, 4), (4, 4, 4)])
def test_direct_matches_scipy_convolution(grid):
    x1, x2, v, kc, D = _case(2, 3, grid, 11 + sum(grid))
    ref = _scipy_reference(x1, x2, v, kc, D)
    got = oracle.conv_direct(x1, x2, v, kc, D, "centered")
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("grid", [(1,), (2,), (16,), (64,), (4, 8), (16, 16), (2, 4, 8), (8, 8, 8)])
def test_fft_matches_direct(grid):
    x1, x2, v, kc, D = _case(2, 2, grid, 21 + sum(grid))
    a = oracle.conv_direct(x1, x2, v, kc, D, "centered")
    b = oracle.conv_fft(x1, x2, v, kc, D, "centered")
    assert np.max(np.abs(a - b)) <= 1e-11 * max(1.0, np.max(np.abs(a)))


@pytest.mark.parametrize("grid", [(8,), (4, 8), (2, 4, 4)])
def test_points_match_lines(grid):
    x1, x2, v, kc, D = _case(2, 3, grid, 5)
    full = oracle.conv_direct(x1, x2, v, kc, D, "centered")
    idx = np.random.default_rng(1).choice(full.size, size=17, replace=False)
    pts = oracle.conv_direct_points(x1, x2, v, kc, D, idx, "centered")
    assert np.allclose(pts, full.ravel()[idx], rtol=0, atol=0)


@pytest.mark.parametrize("grid", [(8,), (4, 8), (2, 4, 4)])
def test_causal_kernel_reduces_to_linear_mode(grid):
    """kc zero wherever some displacement is negative, kc[L - 1 + m] = k[m]:
    the centered call equals the linear-mode call with k."""
    x1, x2, v, _, D = _case(2, 2, grid, 31)
    k = np.random.default_rng(2).standard_normal(x1.shape)
    kc = np.zeros(oracle.kernel_shape(x1.shape, "centered"))
    kc[(slice(None), slice(None)) + tuple(slice(L - 1, 2 * L - 1) for L in grid)] = k
    for fn in (oracle.conv_direct, oracle.conv_fft):
        a = fn(x1, x2, v, kc, D, "centered")
        b = fn(x1, x2, v, k, D, "linear")
        assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("grid", [(8,), (4, 8), (2, 4, 4)])
def test_centre_impulse(grid):
    """kc = delta at the zero displacement: y = x2 (1 + D) u."""
    x1, x2, v, _, D = _case(1, 3, grid, 41)
    kc = np.zeros(oracle.kernel_shape(x1.shape, "centered"))
    kc[(slice(None), slice(None)) + tuple(L - 1 for L in grid)] = 1.0
    want = x2 * x1 * v * (1.0 + D.reshape((1, -1) + (1,) * len(grid)))
    for fn in (oracle.conv_direct, oracle.conv_fft):
        assert np.allclose(fn(x1, x2, v, kc, D, "centered"), want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("grid", [(8,), (4, 8), (2, 4, 4)])
def test_mirror_symmetry(grid):
    """Reversing u, x2 and kc along every axis reverses the output (all
    displacements change sign together)."""
    x1, x2, v, kc, D = _case(1, 2, grid, 51)
    axes = tuple(range(2, 2 + len(grid)))
    a = oracle.conv_fft(x1, x2, v, kc, D, "centered")
    b = oracle.conv_fft(np.flip(x1, axes), np.flip(x2, axes), np.flip(v, axes), np.flip(kc, axes), D, "centered")
    assert np.allclose(np.flip(b, axes), a, rtol=1e-11, atol=1e-11)


def test_kernel_shape_is_checked():
    x1, x2, v, kc, D = _case(1, 1, (4,), 0)
    with pytest.raises(ValueError):
        oracle.conv_direct(x1, x2, v, x1, D, "centered")  # k on the L grid
    with pytest.raises(ValueError):
        oracle.backward_fft(x1, x2, v, kc, D, x1, "centered")
