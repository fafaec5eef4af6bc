"""Pins of the oracle's kernel synthesis: the HyenaND kernel K(x) = w(c) *
f_theta(c; z(x)) of section 3.2.1 (Eq. (kernel), a SIREN over the normalised
grid coordinates), section 3.2.2 (Eq. (film), per-sample FiLM of every hidden
layer) and the appendix on masking (Eq. (mask), the per-axis Gaussian window;
the exponential window of the original Hyena).

Checked through values fixed by the definition: the grid coordinates of every
pad mode against printed sines and against numpy's linspace, the window
against printed exponentials, closed forms for one hidden unit and for a
constant hidden layer, a cyclic-shift layer that exposes a transposed weight
matrix, FiLM's position (after the sine: the output is affine in beta with
one layer), the FiLM identity, odd symmetry, invariance to a relabelling of
the hidden units, and linearity in the output weights."""
import math

import numpy as np
import pytest

import oracle


def _one_unit(shape, mode, omega0=1.0, w1=1.0, bias=None, alpha=0.0):
    """J = 1, Hf = 1, Wout = 1, exponential window alpha (0: w = 1)."""
    nd = len(shape) - 2
    C = shape[1]
    return oracle.kernel_synth(shape, [omega0], np.full((nd, 1), w1), None, np.ones((1, C)),
                               np.full(C, alpha), bias=None if bias is None else [[bias]],
                               window_kind="exponential", pad_mode=mode)


# sin(1/4), sin(1/3), sin(1/2), sin(2/3), sin(1)
S14, S13, S12, S23, S1 = 0.24740395925452294, 0.3271946967961522, 0.479425538604203, 0.618369803069737, \
    0.8414709848078965


@pytest.mark.parametrize("mode,L,expect", [
    ("centered", 3, [-S1, -S12, 0.0, S12, S1]),         # displacements -2..2 over 2
    ("linear", 3, [0.0, S12, S1]),                       # 0, 1, 2 over 2
    ("circular", 4, [0.0, S13, S23, -S13]),              # 0, 1, 2, -1 over 3
    ("circular", 5, [0.0, S14, S12, -S12, -S14]),        # 0, 1, 2, -2, -1 over 4
])
def test_coordinates_printed(mode, L, expect):
    k = _one_unit((1, 1, L), mode)
    assert np.allclose(k[0], expect, rtol=0, atol=1e-15)


def test_single_point_axis_has_coordinate_zero():
    k = _one_unit((1, 1, 1), "centered", bias=0.5)
    assert k.shape == (1, 1) and abs(k[0, 0] - S12) < 1e-15


@pytest.mark.parametrize("mode", ["linear", "circular", "centered"])
def test_one_unit_closed_form_2d(mode):
    """k = w * sin(omega0 (r W1) + b) on the 2D grid, coordinates built from
    numpy's linspace over each axis' displacements."""
    L0, L1 = 6, 5
    om, w1, b, sig = 2.5, np.array([[0.7], [-1.3]]), 0.4, np.array([[0.8], [0.35]])
    k = oracle.kernel_synth((1, 1, L0, L1), [om], w1, None, np.ones((1, 1)), sig, bias=[[b]], pad_mode=mode)

    def coords(L):
        if mode == "centered":
            return np.linspace(-1.0, 1.0, 2 * L - 1)
        if mode == "linear":
            return np.linspace(0.0, 1.0, L)
        d = np.arange(L)
        return np.where(d <= L // 2, d, d - L) / (L - 1)

    r0, r1 = np.meshgrid(coords(L0), coords(L1), indexing="ij")
    ref = np.exp(-0.5 * ((r0 / sig[0, 0]) ** 2 + (r1 / sig[1, 0]) ** 2)) * np.sin(om * (r0 * w1[0, 0] + r1 * w1[1, 0]) + b)
    assert np.allclose(k[0], ref, rtol=1e-14, atol=1e-15)


def test_gaussian_window_printed():
    """W1 = 0 and bias pi/2: every hidden unit is sin(pi/2) = 1, so
    k = w_c(r) * sum_i Wout[i, c]; centered (3, 2) grid, sigma = (1, 1/2)."""
    shape = (1, 2, 3, 2)
    Hf = 3
    Wout = np.array([[1.0, 0.5], [2.0, -1.0], [-0.5, 0.25]])
    sig = np.array([[1.0, 2.0], [0.5, 1.0]])  # [N, C]
    k = oracle.kernel_synth(shape, np.ones(Hf), np.zeros((2, Hf)), None, Wout, sig,
                            bias=np.full((1, Hf), math.pi / 2), pad_mode="centered")
    f = Wout.sum(axis=0)  # 2.5, -0.25
    assert k.shape == (2, 5, 3)
    # channel 0: corner exp(-(1 + 4)/2), centre 1, (r0 = 1/2, r1 = 0): exp(-1/8)
    assert abs(k[0, 0, 0] - f[0] * 0.0820849986238988) < 1e-15
    assert abs(k[0, 2, 1] - f[0]) < 1e-15
    assert abs(k[0, 3, 1] - f[0] * 0.8824969025845955) < 1e-15
    # channel 1: sigma (2, 1): corner exp(-(1/4 + 1)/2) = exp(-5/8)
    assert abs(k[1, 4, 2] - f[1] * 0.5352614285189903) < 1e-15


def test_exponential_window_printed():
    """Linear 1D, L = 5, alpha = 2: w = exp(-2 i / 4) for i = 0..4."""
    k = _one_unit((1, 1, 5), "linear", w1=0.0, bias=math.pi / 2, alpha=2.0)
    expect = [1.0, 0.6065306597126334, 0.36787944117144233, 0.22313016014842982, 0.1353352832366127]
    assert np.allclose(k[0], expect, rtol=1e-15, atol=0)


def test_output_projection_orientation():
    """Hf = 2, C = 3, W1 = 0, biases (pi/2, pi/6): h = (1, 1/2), so
    f[c] = Wout[0, c] + Wout[1, c] / 2 at every point (window off)."""
    Wout = np.array([[1.0, -2.0, 0.5], [4.0, 3.0, -6.0]])
    k = oracle.kernel_synth((1, 3, 4), np.ones(2), np.zeros((1, 2)), None, Wout, np.zeros(3),
                            bias=[[math.pi / 2, math.pi / 6]], window_kind="exponential", pad_mode="linear")
    assert np.allclose(k, np.array([3.0, -0.5, -2.5])[:, None], rtol=1e-15, atol=1e-15)


def _rand_net(rng, nd, Hf, J, C, B):
    return dict(omega0=rng.uniform(1.0, 6.0, Hf), W1=rng.uniform(-1, 1, (nd, Hf)) / np.sqrt(nd),
                Wh=rng.uniform(-1, 1, (J - 1, Hf, Hf)) * np.sqrt(6.0 / Hf),
                Wout=rng.standard_normal((Hf, C)) / np.sqrt(Hf), window=rng.uniform(0.2, 1.0, (nd, C)),
                gamma=1.0 + 0.3 * rng.standard_normal((B, J, Hf)), beta=0.2 * rng.standard_normal((B, J, Hf)),
                bias=0.3 * rng.standard_normal((J, Hf)))


def test_cyclic_shift_layer_exposes_orientation():
    """With W2[i, o] = 1 when o = i + 1 (mod Hf), layer 2 gives
    h2[o] = sin(h1[o - 1]); with Wout = I the two-layer kernel of channel c is
    the sine of the one-layer kernel of channel c - 1 (window off).  A
    transposed W2 would give channel c + 1."""
    Hf = 4
    rng = np.random.default_rng(3)
    om, W1 = rng.uniform(1, 3, Hf), rng.uniform(-1, 1, (2, Hf))
    shift = np.zeros((1, Hf, Hf))
    for i in range(Hf):
        shift[0, i, (i + 1) % Hf] = 1.0
    args = dict(window_kind="exponential", pad_mode="centered")
    one = oracle.kernel_synth((1, Hf, 3, 4), om, W1, None, np.eye(Hf), np.zeros(Hf), **args)
    two = oracle.kernel_synth((1, Hf, 3, 4), om, W1, shift, np.eye(Hf), np.zeros(Hf), **args)
    assert np.allclose(two, np.sin(np.roll(one, 1, axis=0)), rtol=1e-14, atol=1e-15)
    assert not np.allclose(two, np.sin(np.roll(one, -1, axis=0)), atol=1e-3)


def test_film_identity_is_the_unmodulated_kernel():
    rng = np.random.default_rng(4)
    net = _rand_net(rng, 2, 8, 3, 5, 3)
    shape = (3, 5, 6, 7)
    base = oracle.kernel_synth(shape, net["omega0"], net["W1"], net["Wh"], net["Wout"], net["window"],
                               bias=net["bias"], pad_mode="centered")
    mod = oracle.kernel_synth(shape, net["omega0"], net["W1"], net["Wh"], net["Wout"], net["window"],
                              gamma=np.ones((3, 3, 8)), beta=np.zeros((3, 3, 8)), bias=net["bias"],
                              pad_mode="centered")
    assert mod.shape == (3,) + base.shape
    for b in range(3):
        assert np.array_equal(mod[b], base)


def test_film_acts_after_the_sine():
    """One layer: K = w * ((gamma * sin(.) + beta) Wout), affine in beta and
    linear in gamma; FiLM inside the sine would be neither."""
    rng = np.random.default_rng(5)
    net = _rand_net(rng, 1, 6, 1, 4, 1)
    shape = (1, 4, 9)
    g = 1.0 + 0.5 * rng.standard_normal((1, 1, 6))
    b1, b2 = rng.standard_normal((2, 1, 1, 6))
    z = np.zeros((1, 1, 6))

    def K(gam, bet):
        return oracle.kernel_synth(shape, net["omega0"], net["W1"], None, net["Wout"], net["window"],
                                   gamma=gam, beta=bet, bias=net["bias"][:1])

    assert np.allclose(K(g, b1 + b2) - K(g, z), (K(g, b1) - K(g, z)) + (K(g, b2) - K(g, z)), atol=1e-13)
    assert np.allclose(K(2.0 * g, z), 2.0 * K(g, z), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("grid", [(7,), (4, 6), (3, 4, 5)])
def test_odd_symmetry_without_offsets(grid):
    """No bias and no FiLM shift: f is odd in r and the window even, so the
    centered kernel changes sign under r -> -r."""
    rng = np.random.default_rng(6)
    nd = len(grid)
    net = _rand_net(rng, nd, 8, 3, 3, 2)
    k = oracle.kernel_synth((2, 3) + grid, net["omega0"], net["W1"], net["Wh"], net["Wout"], net["window"],
                            gamma=net["gamma"], beta=np.zeros_like(net["beta"]), pad_mode="centered")
    flipped = k[(slice(None), slice(None)) + (slice(None, None, -1),) * nd]
    assert np.allclose(flipped, -k, rtol=1e-13, atol=1e-14)


def test_hidden_unit_relabelling():
    rng = np.random.default_rng(7)
    Hf, J = 8, 3
    net = _rand_net(rng, 2, Hf, J, 4, 2)
    shape = (2, 4, 5, 6)
    perm = rng.permutation(Hf)
    a = oracle.kernel_synth(shape, net["omega0"], net["W1"], net["Wh"], net["Wout"], net["window"],
                            gamma=net["gamma"], beta=net["beta"], bias=net["bias"], pad_mode="linear")
    b = oracle.kernel_synth(shape, net["omega0"][perm], net["W1"][:, perm], net["Wh"][:, perm][:, :, perm],
                            net["Wout"][perm], net["window"], gamma=net["gamma"][..., perm],
                            beta=net["beta"][..., perm], bias=net["bias"][:, perm], pad_mode="linear")
    assert np.allclose(a, b, rtol=1e-12, atol=1e-14)


def test_linear_in_output_weights():
    rng = np.random.default_rng(8)
    net = _rand_net(rng, 3, 8, 2, 3, 1)
    shape = (1, 3, 3, 4, 5)
    W2 = rng.standard_normal(net["Wout"].shape)

    def K(Wo):
        return oracle.kernel_synth(shape, net["omega0"], net["W1"], net["Wh"], Wo, net["window"],
                                   bias=net["bias"], pad_mode="circular")

    assert np.allclose(K(2.0 * net["Wout"] - 3.0 * W2), 2.0 * K(net["Wout"]) - 3.0 * K(W2), rtol=1e-12,
                       atol=1e-13)


def test_argument_checks():
    with pytest.raises(ValueError):
        oracle.kernel_synth((1, 2, 4), np.ones(3), np.ones((1, 3)), None, np.ones((3, 2)), np.ones((2, 2)))
    with pytest.raises(ValueError):
        oracle.kernel_synth((1, 2, 4), np.ones(3), np.ones((1, 3)), None, np.ones((3, 2)), np.ones((1, 2)),
                            gamma=np.ones((1, 1, 3)))
