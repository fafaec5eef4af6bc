"""Pins of the oracle's backward (gradients through y), CPU only.

The forward output y is linear in each of x1, v, x2, k and D separately, so
the loss <gy, y> is too: a central difference with a unit step along any
direction d equals the directional derivative <grad, d> exactly, up to
rounding.  That ties both backward evaluations (explicit sums, FFT) to the
forward definition (explicit sums), which is pinned on its own in
test_oracle_pins.py.
"""
import numpy as np
import pytest

import oracle

NAMES = ("x1", "x2", "v", "k", "D")
SHAPES = [
    ((2, 3, 8), "linear"), ((2, 3, 8), "circular"),
    ((1, 2, 4, 8), "linear"), ((2, 1, 8, 4), "circular"),
    ((1, 2, 4, 4, 2), "linear"), ((1, 1, 2, 4, 4), "circular"),
    ((2, 2, 5, 3), "linear"), ((1, 2, 3, 5), "circular"), ((1, 1, 3, 2, 5), "linear"),
]


def _inputs(shape, seed):
    rng = np.random.default_rng(seed)
    x1, x2, v, k, gy = (rng.standard_normal(shape) for _ in range(5))
    D = rng.standard_normal(shape[1])
    return [x1, x2, v, k, D], gy, rng


def _pow2(shape):
    return all(s >= 1 and (s & (s - 1)) == 0 for s in shape[2:])


@pytest.mark.parametrize("shape,mode", SHAPES)
def test_backward_matches_finite_differences(shape, mode):
    args, gy, rng = _inputs(shape, 7)
    grads = dict(zip(NAMES, oracle.backward_direct(*args, gy, mode)))

    def loss(a):
        return float(np.sum(gy * oracle.conv_direct(*a, mode)))

    for i, name in enumerate(NAMES):
        d = rng.standard_normal(args[i].shape)
        ap, am = list(args), list(args)
        ap[i] = args[i] + d
        am[i] = args[i] - d
        fd = (loss(ap) - loss(am)) / 2.0
        an = float(np.sum(grads[name] * d))
        assert abs(fd - an) <= 1e-11 * max(1.0, abs(an)), (name, fd, an)


@pytest.mark.parametrize("shape,mode", [s for s in SHAPES if _pow2(s[0])])
def test_backward_fft_equals_direct(shape, mode):
    args, gy, _ = _inputs(shape, 11)
    for a, b in zip(oracle.backward_direct(*args, gy, mode), oracle.backward_fft(*args, gy, mode)):
        assert np.max(np.abs(a - b)) <= 1e-12 * max(1.0, np.max(np.abs(a)))


@pytest.mark.parametrize("mode", ["linear", "circular"])
def test_backward_impulse_kernel(mode):
    """k = unit impulse at index 0: z = (1 + D) u, so gu = (1 + D) h."""
    shape = (2, 3, 4, 8)
    args, gy, _ = _inputs(shape, 3)
    x1, x2, v, k, D = args
    k = np.zeros(shape)
    k[:, :, 0, 0] = 1.0
    gx1, gx2, gv, gk, gD = oracle.backward_fft(x1, x2, v, k, D, gy, mode)
    h = gy * x2
    gu = (1.0 + D[None, :, None, None]) * h
    u = x1 * v
    np.testing.assert_allclose(gx1, gu * v, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gv, gu * x1, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gx2, gy * (1.0 + D[None, :, None, None]) * u, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gD, np.sum(h * u, axis=(0, 2, 3)), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mode", ["linear", "circular"])
def test_backward_kernel_gradient_is_signal_gradient_of_swapped_call(mode):
    """k * u = u * k: the gradient for k equals the gradient for the signal
    of the call with the two roles exchanged (v = 1, D = 0)."""
    shape = (2, 2, 8, 4)
    args, gy, _ = _inputs(shape, 5)
    x1, x2, v, k, D = args
    zero = np.zeros_like(D)
    ones = np.ones(shape)
    gk = oracle.backward_direct(x1, x2, v, k, zero, gy, mode)[3]
    gx1_swapped = oracle.backward_direct(k, x2, ones, x1 * v, zero, gy, mode)[0]
    np.testing.assert_allclose(gk, gx1_swapped, rtol=1e-12, atol=1e-12)
