"""The HyenaND operator (Eq. (HyenaND): l2(q) * SiLU(kin), RMSNorm across
channels, the gated long convolution with Sigmoid(vin), RMSNorm across
channels) through hyenand_operator, against the fp64 oracle's operator, on
every plan and pad mode, and on the 8 x 256 x 64^2 image workload shape."""
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


def _case(B, C, grid, mode, dtype, seed):
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    q, kin, vin = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
    kshape = oracle.kernel_shape(shape, mode)
    npts = int(np.prod(kshape[2:]))
    k = W.quantise(rng.standard_normal(kshape) / np.sqrt(npts), dtype)
    D = W.quantise(0.5 * rng.standard_normal(C), dtype)
    w_in = W.quantise(1.0 + 0.2 * rng.standard_normal(C), dtype)
    w_out = W.quantise(1.0 + 0.2 * rng.standard_normal(C), dtype)
    return shape, (q, kin, vin, k, D, w_in, w_out)


def _check(tag, B, C, grid, mode, dtype, seed, eps=(1e-6, 1e-6), expect_plan=None):
    import torch
    from paper_2607_19378_amd import hyenand as H
    shape, arrs = _case(B, C, grid, mode, dtype, seed)
    plan = H.plan_name(shape, mode, dtype)
    if expect_plan:
        assert plan == expect_plan, plan
    dev = [to_device(a, dtype) for a in arrs]
    y = H.operator(*dev, eps_l2=eps[0], eps_rms=eps[1], pad_mode=mode)
    torch.cuda.synchronize()
    got = from_device(y)
    f64 = [W.storage_to_f64(a, dtype) for a in arrs]
    ref = oracle.operator(*f64, eps_l2=eps[0], eps_rms=eps[1], pad_mode=mode)
    err = rel_l2(got, ref)
    log(f"[operator] {tag} {shape} {mode} {dtype} plan={plan}: rel_l2={err:.3e}")
    assert np.all(np.isfinite(got)) and err <= TOL[dtype]


@pytest.mark.parametrize("mode", ["linear", "circular", "centered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid,plan", [((1,), "fused1d"), ((256,), "fused1d"), ((4096,), "fused1d"),
                                       ((16, 16), "fused2d"), ((32, 64), "fused2d"), ((64, 64), "fused2d")])
def test_single_pass(grid, plan, mode, dtype):
    _check("single", 2, 8, grid, mode, dtype, 100 + sum(grid), expect_plan=plan)


@pytest.mark.parametrize("mode", ["linear", "circular", "centered"])
@pytest.mark.parametrize("grid,plan", [((32768,), "fourstep1d"), ((256, 128), "multipass2d"),
                                       ((256, 64), "multipass2d"), ((8, 16, 32), "multipass3d"),
                                       ((32, 32, 32), "slab3d")])
def test_multi_pass(grid, plan, mode):
    if plan == "slab3d" and mode != "linear":
        # the slab plan takes linear 32^3 (64-point transforms); circular 32^3
        # (32-point) and centred grids stay on the five-pass plan
        plan = "multipass3d"
    _check("multi", 2, 6, grid, mode, "f32", 200 + sum(grid), expect_plan=plan)


@pytest.mark.parametrize("grid", [(65536,), (64, 128), (16, 16, 32), (8, 64, 64)])
def test_multi_pass_bf16(grid):
    _check("multi-bf16", 1, 5, grid, "linear", "bf16", 300 + sum(grid))


@pytest.mark.parametrize("C", [1, 3, 300])
def test_channel_counts(C):
    """One channel (both norms reduce to signs), an odd count and more
    channels than the output norm's 64-point tile holds at full width."""
    _check(f"C={C}", 2, C, (16, 16), "linear", "f32", 400 + C)


def test_zero_epsilons():
    _check("eps=0", 2, 8, (64,), "linear", "f32", 500, eps=(0.0, 0.0))


def test_image_workload_shape():
    """8 x 256 images of 64 x 64, fp32, linear: the image workload's shape."""
    _check("image", 8, 256, (64, 64), "linear", "f32", 600, expect_plan="fused2d")
