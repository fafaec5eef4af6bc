"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Inputs are the seeded storage bytes of paper_2607_19378_amd.workloads; both
sides consume exactly the same values.  The bar is the relative L2 error over
the whole output: <= 1e-5 for fp32 storage, <= 2e-2 for bf16 storage (fp32
compute in both cases).
"""
import os

import numpy as np
import pytest

from paper_2607_19378_amd import workloads as W

from gpu_util import TOL, log, oracle_ref, per_line_worst, rel_l2, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_19378_amd import hyenand as H
    H.lib()  # fail loudly if the HIP library is missing


def check(inp, tag, lines=None, **kw):
    w = inp.workload
    log(f"[parity] {tag}: shape={w.shape} mode={w.pad_mode} dtype={w.dtype} seed={w.seed}")
    y = run_gpu(inp, **kw)
    ref = oracle_ref(inp, lines=lines)
    if lines is not None:
        nl = w.B * w.C
        y = y.reshape(nl, -1)[lines]
        ref = ref.reshape(nl, -1)[lines]
    err = rel_l2(y, ref)
    log(f"[parity] {tag}: rel_l2={err:.3e} (tol {TOL[w.dtype]:.0e})")
    assert np.all(np.isfinite(y))
    assert err <= TOL[w.dtype], f"{tag}: rel L2 {err:.3e}"
    return y, ref


FUSED1D = [1, 2, 4, 8, 16, 32, 64, 256, 1024, 4096]


@pytest.mark.parametrize("L", FUSED1D)
@pytest.mark.parametrize("mode", ["linear", "circular"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused1d_small(L, mode, dtype):
    inp = W.random_case(3, 5, (L,), mode, dtype, seed=100 + L)
    check(inp, f"fused1d L={L}")


@pytest.mark.parametrize("mode,L", [("linear", 8192), ("circular", 8192), ("circular", 16384)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused1d_largest(mode, L, dtype):
    inp = W.random_case(2, 3, (L,), mode, dtype, seed=7)
    check(inp, f"fused1d L={L}")


FUSED2D = [(4, 4), (8, 8), (16, 16), (32, 32), (64, 64), (128, 128), (64, 128), (128, 64), (32, 64),
           (64, 32)]


@pytest.mark.parametrize("P", FUSED2D)
@pytest.mark.parametrize("mode", ["linear", "circular"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused2d_sizes(P, mode, dtype):
    grid = tuple(p // 2 for p in P) if mode == "linear" else P
    inp = W.random_case(2, 3, grid, mode, dtype, seed=200 + P[0] + 3 * P[1])
    check(inp, f"fused2d grid={grid}")


def test_conv1d_4k_full():
    inp = W.generate(W.WORKLOADS["conv1d_4k"])
    y, ref = check(inp, "conv1d_4k")
    assert per_line_worst(y, ref, 64) <= 1e-5


def test_conv2d_64_full():
    inp = W.generate(W.WORKLOADS["conv2d_64"])
    y, ref = check(inp, "conv2d_64")
    assert per_line_worst(y, ref, 8 * 256) <= 1e-5


def test_deterministic_and_inputs_untouched():
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import to_device
    inp = W.random_case(2, 4, (32, 32), "linear", "f32", seed=3)
    dev = [to_device(a, "f32") for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
    before = [t.clone() for t in dev]
    y1 = H.fftconv(*dev, pad_mode="linear")
    y2 = H.fftconv(*dev, pad_mode="linear")
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    for a, b in zip(dev, before):
        assert torch.equal(a, b)


def test_non_default_stream():
    import torch
    inp = W.random_case(2, 3, (64,), "circular", "f32", seed=4)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y = run_gpu(inp, stream=s)
    ref = oracle_ref(inp)
    assert rel_l2(y, ref) <= 1e-5


def test_shape_with_unit_axes():
    # unit axes are squeezed: a [B, C, 1, 64] problem is the 1D problem of length 64
    inp = W.random_case(2, 3, (1, 64), "linear", "f32", seed=5)
    check(inp, "unit axis 2d")
    inp = W.random_case(1, 2, (1, 1, 1), "circular", "bf16", seed=6)
    check(inp, "single point 3d")
