"""Pins of the oracle's centred-mode backward (the direct sums): each gradient
against the exact change of the oracle's centred forward along a random
direction (the operation is linear in each input when the others are held,
so <gy, f(t + d) - f(t)> = <g_t, d> holds to rounding), and against the
linear-mode backward when the centred kernel has no negative displacements
(then the two forwards agree, and so must gx1, gx2, gv and the causal half of
gk).  Extents that are not powers of two included."""
import numpy as np
import pytest

import oracle


def _case(shape, seed):
    rng = np.random.default_rng(seed)
    x1, x2, v, gy = (rng.standard_normal(shape) for _ in range(4))
    k = rng.standard_normal(oracle.kernel_shape(shape, "centered")) * 0.3
    D = rng.standard_normal(shape[1])
    return x1, x2, v, k, D, gy


@pytest.mark.parametrize("shape", [(2, 3, 7), (1, 2, 5, 6), (1, 2, 3, 4, 5), (2, 2, 8)])
def test_gradients_are_directional_derivatives(shape):
    x1, x2, v, k, D, gy = _case(shape, sum(shape))
    gx1, gx2, gv, gk, gD = oracle.backward_direct(x1, x2, v, k, D, gy, "centered")
    f = lambda *a: oracle.conv_direct(*a, "centered")
    y = f(x1, x2, v, k, D)
    rng = np.random.default_rng(1)
    for name, grad in (("x1", gx1), ("x2", gx2), ("v", gv), ("k", gk), ("D", gD)):
        args = dict(x1=x1, x2=x2, v=v, k=k, D=D)
        d = rng.standard_normal(args[name].shape)
        args[name] = args[name] + d
        lhs = np.sum(gy * (f(args["x1"], args["x2"], args["v"], args["k"], args["D"]) - y))
        rhs = np.sum(grad * d)
        assert abs(lhs - rhs) <= 1e-10 * max(1.0, abs(rhs)), name


@pytest.mark.parametrize("shape", [(2, 3, 9), (1, 2, 4, 6), (1, 1, 3, 3, 4)])
def test_causal_kernel_matches_linear_mode(shape):
    x1, x2, v, k, D, gy = _case(shape, 7 + sum(shape))
    grid = shape[2:]
    kc = np.zeros_like(k)
    causal = (slice(None), slice(None)) + tuple(slice(L - 1, None) for L in grid)
    kc[causal] = k[causal]
    kl = np.ascontiguousarray(k[causal])  # index i of kl is displacement i
    c = oracle.backward_direct(x1, x2, v, kc, D, gy, "centered")
    lin = oracle.backward_direct(x1, x2, v, kl, D, gy, "linear")
    for a, b in zip(c[:3], lin[:3]):
        assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    assert np.allclose(c[3][causal], lin[3], rtol=1e-12, atol=1e-12)
    assert np.allclose(c[4], lin[4], rtol=1e-12, atol=1e-12)


def test_fft_backward_rejects_centered():
    x1, x2, v, k, D, gy = _case((1, 1, 4), 3)
    with pytest.raises(ValueError):
        oracle.backward_fft(x1, x2, v, k, D, gy, "centered")
