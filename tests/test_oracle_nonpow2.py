"""Pins of the oracle on grids whose extents are not powers of two (linear and
centered modes): the transform runs on the smallest power of two >= 2L - 1,
which holds every displacement between two grid points, so the result is the
plain linear convolution.  Checked against scipy's N-D convolution, between
the oracle's direct and FFT evaluations, and for the backward."""
import numpy as np
import pytest
from scipy import signal

import oracle


def _case(B, C, grid, seed, mode):
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    x1, x2, v = (rng.standard_normal(shape) for _ in range(3))
    k = rng.standard_normal(oracle.kernel_shape(shape, mode))
    D = rng.standard_normal(C)
    return x1, x2, v, k, D


@pytest.mark.parametrize("grid", [(3,), (7,), (12,), (3, 5), (14, 14), (3, 6, 5)])
def test_linear_matches_scipy(grid):
    x1, x2, v, k, D = _case(2, 2, grid, 1 + sum(grid), "linear")
    got = oracle.conv_fft(x1, x2, v, k, D, "linear")
    sl = tuple(slice(0, L) for L in grid)
    for b in range(2):
        for c in range(2):
            u = x1[b, c] * v[b, c]
            full = signal.convolve(u, k[b, c], mode="full", method="direct")
            want = x2[b, c] * (full[sl] + D[c] * u)
            assert np.allclose(got[b, c], want, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("mode", ["linear", "centered"])
@pytest.mark.parametrize("grid", [(5,), (9,), (100,), (6, 10), (14, 14), (5, 3, 7)])
def test_fft_matches_direct(mode, grid):
    x1, x2, v, k, D = _case(2, 3, grid, 11 + sum(grid), mode)
    a = oracle.conv_direct(x1, x2, v, k, D, mode)
    b = oracle.conv_fft(x1, x2, v, k, D, mode)
    assert np.max(np.abs(a - b)) <= 1e-11 * max(1.0, np.max(np.abs(a)))


@pytest.mark.parametrize("grid", [(7,), (6, 10), (3, 5, 6)])
def test_backward_fft_matches_direct(grid):
    x1, x2, v, k, D = _case(2, 2, grid, 21 + sum(grid), "linear")
    gy = np.random.default_rng(3).standard_normal(x1.shape)
    a = oracle.backward_direct(x1, x2, v, k, D, gy, "linear")
    b = oracle.backward_fft(x1, x2, v, k, D, gy, "linear")
    for ga, gb in zip(a, b):
        assert np.max(np.abs(ga - gb)) <= 1e-10 * max(1.0, np.max(np.abs(ga)))


def test_circular_fft_needs_powers_of_two():
    x1, x2, v, k, D = _case(1, 1, (6,), 0, "circular")
    with pytest.raises(RuntimeError):
        oracle.conv_fft(x1, x2, v, k, D, "circular")


@pytest.mark.parametrize("grid", [(3,), (6,), (12,), (3, 5), (14, 14), (5, 6, 7)])
def test_circular_direct_matches_numpy_fft(grid):
    """The circular mode on any extents (the direct sums) against numpy's
    FFT of the same length: circular convolution = ifftn(fftn(u) fftn(k))."""
    x1, x2, v, k, D = _case(2, 2, grid, 41 + sum(grid), "circular")
    got = oracle.conv_direct(x1, x2, v, k, D, "circular")
    ax = tuple(range(2, 2 + len(grid)))
    u = x1 * v
    conv = np.real(np.fft.ifftn(np.fft.fftn(u, axes=ax) * np.fft.fftn(k, axes=ax), axes=ax))
    want = x2 * (conv + D.reshape((1, 2) + (1,) * len(grid)) * u)
    assert np.allclose(got, want, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("grid", [(6,), (3, 5)])
def test_circular_backward_direct_matches_numpy_fft(grid):
    """Circular gradients on any extents against numpy FFT correlations:
    gu = ifft(conj(K) H) + D h, gk = ifft(conj(U) H)."""
    x1, x2, v, k, D = _case(1, 2, grid, 51 + sum(grid), "circular")
    gy = np.random.default_rng(9).standard_normal(x1.shape)
    gx1, gx2, gv, gk, gD = oracle.backward_direct(x1, x2, v, k, D, gy, "circular")
    ax = tuple(range(2, 2 + len(grid)))
    F = lambda a: np.fft.fftn(a, axes=ax)
    iF = lambda a: np.real(np.fft.ifftn(a, axes=ax))
    u, h = x1 * v, gy * x2
    Dc = D.reshape((1, 2) + (1,) * len(grid))
    gu = iF(np.conj(F(k)) * F(h)) + Dc * h
    assert np.allclose(gx1, gu * v, rtol=1e-11, atol=1e-11)
    assert np.allclose(gv, gu * x1, rtol=1e-11, atol=1e-11)
    assert np.allclose(gk, iF(np.conj(F(u)) * F(h)), rtol=1e-11, atol=1e-11)
    assert np.allclose(gx2, gy * (iF(F(u) * F(k)) + Dc * u), rtol=1e-11, atol=1e-11)
    assert np.allclose(gD, (h * u).sum(axis=(0,) + ax), rtol=1e-11, atol=1e-11)
