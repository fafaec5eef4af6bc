"""Parity of the centered mode (the paper's kernel on the double grid of
2 L_d - 1 points per axis, section 3.2.1) with the fp64 oracle, on every plan:
single-pass 1D/2D, four-step 1D, multi-pass 2D/3D (natural and forced), one
kernel per channel, chunked workspaces, and the 64x64 image workload shape."""
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


def _case(B, C, grid, dtype, seed, shared=False):
    """N(0,1) signals; a centered kernel with a Gaussian window around the
    zero displacement (the window form of section 3.2.2)."""
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    x1, x2, v = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
    kgrid = tuple(2 * L - 1 for L in grid)
    win = np.ones(kgrid)
    for d, L in enumerate(grid):
        j = np.arange(2 * L - 1) - (L - 1)
        sh = [1] * len(grid)
        sh[d] = -1
        win = win * np.exp(-0.5 * (j / max(1.0, L / 3.0)) ** 2).reshape(sh)
    kshape = ((C,) if shared else (B, C)) + kgrid
    k = W.quantise(rng.standard_normal(kshape) * win / np.sqrt(np.prod(grid)), dtype)
    D = W.quantise(rng.standard_normal(C), dtype)
    return shape, x1, x2, v, k, D


def _run(shape, x1, x2, v, k, D, dtype, shared=False, workspace_bytes=None):
    import torch
    from paper_2607_19378_amd import hyenand as H
    dev = [to_device(a, dtype) for a in (x1, x2, v, k, D)]
    ws = None
    if workspace_bytes is not None:
        ws = torch.empty(workspace_bytes, dtype=torch.uint8, device="cuda")
    y = H.fftconv(*dev, pad_mode="centered", workspace=ws, shared_k=shared)
    torch.cuda.synchronize()
    return from_device(y)


def _ref(shape, x1, x2, v, k, D, dtype, shared=False):
    f = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, k, D)]
    if shared:
        f[3] = np.broadcast_to(f[3][None], (shape[0],) + f[3].shape)
    return oracle.conv_fft(*f, "centered")


def _check(tag, B, C, grid, dtype, seed, shared=False, expect_plan=None):
    from paper_2607_19378_amd import hyenand as H
    shape, x1, x2, v, k, D = _case(B, C, grid, dtype, seed, shared)
    plan = H.plan_name(shape, "centered", dtype)
    if expect_plan:
        assert plan == expect_plan, plan
    y = _run(shape, x1, x2, v, k, D, dtype, shared)
    err = rel_l2(y, _ref(shape, x1, x2, v, k, D, dtype, shared))
    log(f"[centered] {tag} {shape} {dtype} plan={plan}: rel_l2={err:.3e}")
    assert np.all(np.isfinite(y)) and err <= TOL[dtype]


@pytest.mark.parametrize("L", [2, 4, 8, 64, 1024, 4096, 8192])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused1d(L, dtype):
    _check("fused1d", 2, 3, (L,), dtype, 10 + L, expect_plan="fused1d")


@pytest.mark.parametrize("L", [16384, 65536])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fourstep(L, dtype):
    _check("fourstep", 1, 3, (L,), dtype, 20 + L % 97, expect_plan="fourstep1d")


@pytest.mark.parametrize("grid", [(2, 2), (4, 4), (8, 8), (16, 32), (32, 32), (64, 64), (32, 64), (64, 32)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused2d(grid, dtype):
    _check("fused2d", 2, 3, grid, dtype, 30 + sum(grid), expect_plan="fused2d")


@pytest.mark.parametrize("grid", [(128, 128), (256, 64), (16, 512), (256, 256)])
def test_multipass2d(grid):
    _check("mp2d", 1, 3, grid, "f32", 40 + sum(grid), expect_plan="multipass2d")


@pytest.mark.parametrize("grid", [(2, 2), (8, 4), (32, 32)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_multipass2d_forced(monkeypatch, grid, dtype):
    monkeypatch.setenv("HYENAND_PLAN", "multipass")
    _check("mp2d-forced", 2, 3, grid, dtype, 50 + sum(grid), expect_plan="multipass2d")


@pytest.mark.parametrize("grid", [(2, 2, 2), (4, 8, 2), (8, 16, 32), (32, 32, 32), (16, 4, 64)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_multipass3d(grid, dtype):
    _check("mp3d", 1, 3, grid, dtype, 60 + sum(grid), expect_plan="multipass3d")


@pytest.mark.parametrize("grid", [(64,), (32768,), (16, 16), (128, 64), (8, 8, 8)])
def test_shared_kernel(grid):
    _check("shared", 3, 2, grid, "f32", 70 + sum(grid), shared=True)


@pytest.mark.parametrize("grid", [(128, 64), (8, 8, 16), (32768,)])
def test_chunked_workspace_bitwise(grid):
    from paper_2607_19378_amd import hyenand as H
    shape, x1, x2, v, k, D = _case(1, 5, grid, "f32", 80)
    wmin = H.workspace_min(shape, "centered", "f32")
    assert wmin > 0
    ys = [_run(shape, x1, x2, v, k, D, "f32", workspace_bytes=n) for n in (wmin, 2 * wmin, None)]
    assert np.array_equal(ys[0], ys[1]) and np.array_equal(ys[0], ys[2])
    assert rel_l2(ys[2], _ref(shape, x1, x2, v, k, D, "f32")) <= TOL["f32"]


def test_image_workload_shape_sampled_lines():
    """8 x 256 images of 64 x 64 with 127 x 127 centered kernels (fp32): the
    image workload's shape in the paper's non-circular form; parity on
    sampled lines."""
    from paper_2607_19378_amd import hyenand as H
    shape, x1, x2, v, k, D = _case(8, 256, (64, 64), "f32", 90)
    assert H.plan_name(shape, "centered", "f32") == "fused2d"
    y = _run(shape, x1, x2, v, k, D, "f32")
    nl = 8 * 256
    lines = np.array([0, 1, 255, 256, 1000, nl - 1])
    f = [W.storage_to_f64(a.reshape((nl, 1) + a.shape[2:])[lines].reshape((1, len(lines)) + a.shape[2:]), "f32")
         for a in (x1, x2, v, k)]
    Dl = W.storage_to_f64(D, "f32")[lines % 256]
    ref = oracle.conv_fft(*f, Dl, "centered")[0]
    err = rel_l2(y.reshape((nl,) + shape[2:])[lines], ref)
    log(f"[centered] image workload lines {lines.tolist()}: rel_l2={err:.3e}")
    assert err <= TOL["f32"]
