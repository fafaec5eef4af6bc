"""Pins of the oracle's HyenaND operator, Eq. (HyenaND) of section 3.2:

    y = RMSNorm(Sigmoid(vin) * (k conv RMSNorm(l2(q) * SiLU(kin)) + D * .)),

both norms across the C channels of every (sample, grid point).  Checked
through properties the definition fixes: invariance of the l2 norm to a
positive scale of q and of the output norm to a joint scale of (k, D); odd
symmetry in q; unit channel RMS of the output; a constant gate cancelling;
the SiLU limit; point-wise behaviour and channel equivariance with an impulse
kernel; and closed forms for one and two channels."""
import numpy as np
import pytest

import oracle


def _case(B, C, grid, seed, mode="linear"):
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    q, kin, vin = (rng.standard_normal(shape) for _ in range(3))
    k = rng.standard_normal(oracle.kernel_shape(shape, mode)) * 0.3
    D = rng.standard_normal(C)
    w_in = 1.0 + 0.2 * rng.standard_normal(C)
    w_out = 1.0 + 0.2 * rng.standard_normal(C)
    return q, kin, vin, k, D, w_in, w_out


def _impulse(shape, mode="linear"):
    k = np.zeros(oracle.kernel_shape(shape, mode))
    grid = shape[2:]
    idx = tuple(L - 1 for L in grid) if mode == "centered" else (0,) * len(grid)
    k[(slice(None), slice(None)) + idx] = 1.0
    return k


MODES = ["linear", "circular", "centered"]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("grid", [(16,), (4, 8), (2, 4, 4)])
def test_scale_of_q_cancels(mode, grid):
    q, kin, vin, k, D, wi, wo = _case(2, 5, grid, 1, mode)
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-12, 1e-6, mode)
    b = oracle.operator(7.5 * q, kin, vin, k, D, wi, wo, 1e-12, 1e-6, mode)
    assert np.allclose(a, b, rtol=1e-11, atol=1e-12)


def test_scale_of_q_cancels_through_the_l2_norm():
    """With a large eps_rms the RMSNorm no longer removes a scale of its
    input, so only the l2 normalisation of q makes the output invariant."""
    q, kin, vin, k, D, wi, wo = _case(1, 4, (8,), 11)
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-12, 1.0)
    b = oracle.operator(0.01 * q, kin, vin, k, D, wi, wo, 1e-12, 1.0)
    assert np.allclose(a, b, rtol=1e-11, atol=1e-12)
    c = oracle.operator(q, 0.01 * kin, vin, k, D, wi, wo, 1e-12, 1.0)  # no such invariance in kin
    assert not np.allclose(a, c, rtol=1e-3)


@pytest.mark.parametrize("mode", MODES)
def test_odd_in_q(mode):
    q, kin, vin, k, D, wi, wo = _case(2, 4, (4, 8), 2, mode)
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-6, 1e-6, mode)
    b = oracle.operator(-q, kin, vin, k, D, wi, wo, 1e-6, 1e-6, mode)
    assert np.allclose(a, -b, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("mode", MODES)
def test_joint_scale_of_kernel_and_shortcut_cancels(mode):
    q, kin, vin, k, D, wi, wo = _case(2, 4, (8, 4), 3, mode)
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-6, 0.0, mode)
    b = oracle.operator(q, kin, vin, 3.25 * k, 3.25 * D, wi, wo, 1e-6, 0.0, mode)
    assert np.allclose(a, b, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("mode", MODES)
def test_unit_channel_rms(mode):
    q, kin, vin, k, D, wi, _ = _case(2, 6, (16,), 4, mode)
    y = oracle.operator(q, kin, vin, k, D, wi, np.ones(6), 1e-6, 0.0, mode)
    rms = np.sqrt(np.mean(y * y, axis=1))
    assert np.allclose(rms, 1.0, rtol=1e-12)


def test_constant_gate_cancels():
    q, kin, _, k, D, wi, wo = _case(1, 4, (4, 4), 5)
    zero = np.zeros_like(q)
    a = oracle.operator(q, kin, zero, k, D, wi, wo, 1e-6, 0.0)          # Sigmoid = 1/2
    b = oracle.operator(q, kin, zero + 40.0, k, D, wi, wo, 1e-6, 0.0)   # Sigmoid = 1
    assert np.allclose(a, b, rtol=1e-11, atol=1e-12)


def test_silu_limit_switches_the_input_off():
    q, kin, vin, k, D, wi, wo = _case(1, 3, (8,), 6)
    y = oracle.operator(q, np.full_like(kin, -60.0), vin, k, D, wi, wo, 1e-6, 1e-6)
    assert np.max(np.abs(y)) < 1e-10


@pytest.mark.parametrize("mode", MODES)
def test_impulse_kernel_acts_per_point(mode):
    """With k an impulse at the zero displacement the operator acts on every
    grid point on its own: permuting the points permutes the output."""
    q, kin, vin, _, D, wi, wo = _case(2, 3, (16,), 7, mode)
    k = _impulse(q.shape, mode)
    perm = np.random.default_rng(0).permutation(16)
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-6, 1e-6, mode)
    b = oracle.operator(q[..., perm], kin[..., perm], vin[..., perm], k, D, wi, wo, 1e-6, 1e-6, mode)
    assert np.allclose(a[..., perm], b, rtol=1e-12, atol=1e-13)


def test_channel_permutation_equivariance():
    q, kin, vin, k, D, wi, wo = _case(2, 5, (4, 4), 8)
    perm = np.array([3, 0, 4, 1, 2])
    a = oracle.operator(q, kin, vin, k, D, wi, wo, 1e-6, 1e-6)
    b = oracle.operator(q[:, perm], kin[:, perm], vin[:, perm], k[:, perm], D[perm], wi[perm], wo[perm], 1e-6, 1e-6)
    assert np.allclose(a[:, perm], b, rtol=1e-12, atol=1e-13)


def test_one_channel_closed_form():
    """C = 1, no epsilons, impulse kernel: both norms reduce to signs, and
    SiLU has the sign of its argument, so y = w_out sign(q kin w_in (1 + D))."""
    rng = np.random.default_rng(9)
    shape = (2, 1, 32)
    q, kin, vin = (rng.standard_normal(shape) for _ in range(3))
    D = np.array([0.7])
    wi, wo = np.array([-1.3]), np.array([2.5])
    y = oracle.operator(q, kin, vin, _impulse(shape), D, wi, wo, 0.0, 0.0)
    assert np.allclose(y, wo[0] * np.sign(q * kin * wi[0] * (1.0 + D[0])), rtol=1e-12)


def test_two_channel_worked_example():
    """C = 2, q = (1, 1), kin = (1, 2), an open gate and an impulse kernel, no
    shortcut, unit weights, no epsilons: y = a / rms(a) with a = (SiLU(1),
    SiLU(2)) / sqrt(2); SiLU(1) = 0.7310585786300049, SiLU(2) =
    1.7615941559557646 (x times the logistic function)."""
    shape = (1, 2, 1)
    q = np.ones(shape)
    kin = np.array([1.0, 2.0]).reshape(shape)
    vin = np.full(shape, 40.0)
    y = oracle.operator(q, kin, vin, _impulse(shape), np.zeros(2), np.ones(2), np.ones(2), 0.0, 0.0)
    a = np.array([0.7310585786300049, 1.7615941559557646])
    assert np.allclose(y.ravel(), a / np.sqrt(np.mean(a * a)), rtol=1e-12)
