"""Kernel synthesis on the GPU (hyenand_kernel_synth: SIREN over the grid
coordinates on the matrix cores, per-sample FiLM, Gaussian or exponential
window) against the fp64 oracle's kernel synthesis on the same fp32
parameters; and the synthesised kernel fed to the convolution, against the
oracle's kernel fed to the oracle's convolution."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

from gpu_util import TOL, from_device, log, rel_l2, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _dev(p):
    import torch
    return {k: (None if v is None else torch.from_numpy(v).cuda()) for k, v in p.items()}


def _synth_pair(shape, hidden, layers, mode, dtype, seed, modulated=True, bias=True, window_kind="gaussian"):
    import torch
    from paper_2607_19378_amd import hyenand as H
    B, C = shape[:2]
    p = W.siren_params(seed, len(shape) - 2, hidden, layers, C, B, modulated=modulated, bias=bias,
                       window_kind=window_kind)
    d = _dev(p)
    k = H.kernel_synth(shape, d["omega0"], d["W1"], d["Wh"], d["Wout"], d["window"], gamma=d["gamma"],
                       beta=d["beta"], bias=d["bias"], window_kind=window_kind, pad_mode=mode,
                       dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)
    torch.cuda.synchronize()
    f = {kk: (None if v is None else v.astype(np.float64)) for kk, v in p.items()}
    ref = oracle.kernel_synth(shape, f["omega0"], f["W1"], f["Wh"], f["Wout"], f["window"], gamma=f["gamma"],
                              beta=f["beta"], bias=f["bias"], window_kind=window_kind, pad_mode=mode)
    return k, ref, p


def _check(tag, shape, hidden, layers, mode, dtype, seed, **kw):
    k, ref, _ = _synth_pair(shape, hidden, layers, mode, dtype, seed, **kw)
    got = from_device(k)
    assert got.shape == ref.shape
    err = rel_l2(got, ref)
    log(f"[synth] {tag} {shape} Hf={hidden} J={layers} {mode} {dtype} {kw}: rel_l2={err:.3e}")
    assert np.all(np.isfinite(got)) and err <= TOL[dtype]


@pytest.mark.parametrize("mode", ["linear", "circular", "centered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(2, 5, 1000), (3, 33, 14, 14), (2, 7, 5, 6, 7)])
def test_modes_and_grids(shape, mode, dtype):
    _check("grid", shape, 64, 3, mode, dtype, sum(shape))


@pytest.mark.parametrize("hidden", [32, 64, 128])
@pytest.mark.parametrize("layers", [1, 2, 4])
def test_widths_and_depths(hidden, layers):
    _check("width", (2, 40, 24, 20), hidden, layers, "centered", "f32", hidden + layers)


@pytest.mark.parametrize("C", [1, 31, 32, 300])
def test_channel_counts(C):
    _check("channels", (2, C, 9, 11), 32, 2, "linear", "f32", C)


@pytest.mark.parametrize("hidden,C", [(64, 1200), (32, 3000), (128, 300)])
def test_streamed_weights(hidden, C):
    """Weights too large to stay in LDS together: hidden matrices and chunks
    of output channels are staged one at a time (the last chunk ragged)."""
    _check("streamed", (2, C, 8, 8), hidden, 3, "centered", "f32", C + hidden)


def test_unmodulated_is_shared():
    _check("shared", (4, 16, 30, 17), 64, 3, "centered", "f32", 9, modulated=False)


def test_no_bias_exponential_window():
    _check("exp", (2, 12, 4096), 32, 3, "linear", "f32", 10, bias=False, window_kind="exponential")


def test_single_point_and_unit_axes():
    _check("unit", (3, 4, 1), 32, 2, "centered", "f32", 11)
    _check("unit", (2, 4, 1, 9), 32, 2, "linear", "f32", 12)


def test_image_workload_shape():
    """8 samples x 256 channels, 64 x 64 images, Hf = 64, J = 3: the kernel of
    the image workload, every point against the oracle."""
    _check("image", (8, 256, 64, 64), 64, 3, "linear", "f32", 13)


def test_image_workload_shape_centered_bf16():
    _check("image-centered", (8, 256, 64, 64), 64, 3, "centered", "bf16", 14)


@pytest.mark.parametrize("mode,shape", [("centered", (2, 8, 32, 32)), ("linear", (2, 6, 3000)),
                                        ("circular", (2, 8, 64, 32))])
def test_synthesised_kernel_through_the_convolution(mode, shape):
    """y = conv(K(x)) on the GPU (both stages on the GPU) against the oracle's
    kernel through the oracle's convolution."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    k, kref, _ = _synth_pair(shape, 64, 3, mode, "f32", 20)
    rng = np.random.default_rng(21)
    x1, x2, v = (rng.standard_normal(shape).astype(np.float32) for _ in range(3))
    D = rng.standard_normal(shape[1]).astype(np.float32)
    y = H.fftconv(*[to_device(a, "f32") for a in (x1, x2, v)], k, to_device(D, "f32"), pad_mode=mode)
    torch.cuda.synchronize()
    ref = oracle.conv_fft(x1.astype(np.float64), x2.astype(np.float64), v.astype(np.float64), kref,
                          D.astype(np.float64), mode)
    err = rel_l2(from_device(y), ref)
    log(f"[synth] through conv {shape} {mode}: rel_l2={err:.3e}")
    assert err <= TOL["f32"]


def test_repeated_calls_identical():
    import torch
    from paper_2607_19378_amd import hyenand as H
    shape = (2, 20, 16, 16)
    p = _dev(W.siren_params(30, 2, 64, 3, 20, 2))
    k = torch.empty(H.kernel_shape(shape, "linear"), device="cuda")
    call = H.PreparedSynth(k, shape, p["omega0"], p["W1"], p["Wh"], p["Wout"], p["window"], p["gamma"], p["beta"],
                           p["bias"])
    call()
    first = k.clone()
    for _ in range(3):
        call()
    torch.cuda.synchronize()
    assert torch.equal(first, k)
