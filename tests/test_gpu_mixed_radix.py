"""Mixed-radix single-pass kernels (transform extents with prime factors 2, 3,
5 and 7): circular axes of such extents are transformed on their own points,
other axes on the smallest such P >= 2L - 1.  Parity with the fp64 oracle on
1D, 2D and 3D grids, every pad mode, fp32 and bf16, odd line counts (a
workgroup's last pair half empty), several pairs per workgroup, one kernel per
channel and the HyenaND operator; whole-tensor relative L2 and the worst
line."""
import os

import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

from gpu_util import TOL, from_device, log, per_line_worst, rel_l2, summary, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


class _env:
    """Set environment variables for the duration of a call."""

    def __init__(self, **kv):
        self.kv = kv

    def __enter__(self):
        self.prev = {k: os.environ.get(k) for k in self.kv}
        for k, v in self.kv.items():
            os.environ[k] = str(v)

    def __exit__(self, *exc):
        for k, v in self.prev.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


def _case(B, C, grid, mode, dtype, seed, shared=False):
    rng = np.random.default_rng(seed)
    shape = (B, C) + tuple(grid)
    x1, x2, v = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
    kshape = oracle.kernel_shape(shape, mode)
    if shared:
        kshape = kshape[1:]
    k = W.quantise(rng.standard_normal(kshape) / np.sqrt(np.prod(kshape[-len(grid):])), dtype)
    D = W.quantise(rng.standard_normal(C), dtype)
    return shape, x1, x2, v, k, D


def _check(tag, B, C, grid, mode, dtype, seed, shared=False, **env):
    """Run one call (with env set), compare with the oracle, return the plan."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    shape, x1, x2, v, k, D = _case(B, C, grid, mode, dtype, seed, shared)
    dev = [to_device(a, dtype) for a in (x1, x2, v, k, D)]
    with _env(**env):
        plan = H.plan_name(shape, mode, dtype)
        log(f"[mixed] {tag} {shape} {mode} {dtype} plan={plan} {env}")
        y = H.fftconv(*dev, pad_mode=mode, shared_k=shared)
        torch.cuda.synchronize()
    got = from_device(y)
    f = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, k, D)]
    if shared:
        f[3] = np.broadcast_to(f[3][None], (B,) + f[3].shape)
    ref = (oracle.conv_direct if mode == "circular" else oracle.conv_fft)(*f, mode)
    err = rel_l2(got, ref)
    worst = per_line_worst(got, ref, B * C)
    log(f"[mixed] {tag}: rel_l2={err:.3e} worst line={worst:.3e}")
    assert np.all(np.isfinite(got)) and err <= TOL[dtype] and worst <= TOL[dtype]
    return plan


def _mixed(nd):
    return {1: "mixed1d", 2: "mixed2d", 3: "mixed3d"}[nd]


# circular extents with prime factors 2, 3, 5, 7, on their own points
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", [3, 5, 7, 12, 15, 100, 300, 1000, 3000])
def test_1d_circular(L, dtype):
    assert _check("1d-circ", 3, 5, (L,), "circular", dtype, 100 + L, HYENAND_PLAN="mixed") == "mixed1d"


def test_1d_default_choice():
    from paper_2607_19378_amd import hyenand as H
    assert H.plan_name((2, 3, 300), "circular", "f32") == "mixed1d"
    assert H.plan_name((2, 3, 5), "circular", "f32") == "mixed1d"
    assert H.plan_name((2, 3, 100), "circular", "f32") == "mixed1d"
    assert H.plan_name((2, 3, 1000), "circular", "f32") == "fused1d_any"
    assert H.plan_name((2, 3, 3000), "circular", "f32") == "mixed1d"
    assert H.plan_name((2, 3, 67), "circular", "f32") == "fused1d_any"
    assert H.plan_name((2, 3, 100), "linear", "f32") == "fused1d_any"
    _check("1d-default", 4, 16, (300,), "circular", "f32", 77)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid", [(14, 14), (3, 5), (7, 30), (16, 14), (2, 3), (12, 20), (48, 64), (63, 64)])
def test_2d_circular(grid, dtype):
    assert _check("2d-circ", 3, 5, grid, "circular", dtype, 200 + sum(grid)) == "mixed2d"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid", [(5, 6, 7), (6, 10, 14), (12, 12, 12), (3, 4, 5)])
def test_3d_circular(grid, dtype):
    assert _check("3d-circ", 3, 5, grid, "circular", dtype, 300 + sum(grid)) == "mixed3d"


# a circular axis of another extent (13, 11): k repeated periodically on P >= 2L - 1
@pytest.mark.parametrize("grid", [(13, 14), (14, 11), (13,), (11, 13)])
def test_periodic_axes(grid):
    assert _check("periodic", 2, 3, grid, "circular", "f32", 400 + sum(grid),
                  HYENAND_PLAN="mixed") == _mixed(len(grid))


# non-circular modes on the smallest 2-3-5-7 extent >= 2L - 1 (forced where
# the power-of-two kernels are the default)
@pytest.mark.parametrize("mode", ["linear", "centered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid", [(3,), (14,), (100,), (1000,), (14, 14), (7, 30), (24, 40), (2, 3), (5, 6, 7)])
def test_noncircular(grid, mode, dtype):
    assert _check("noncirc", 3, 5, grid, mode, dtype, 500 + sum(grid), HYENAND_PLAN="mixed") == _mixed(len(grid))


# pairs per workgroup: one, a few, and the default, on 7 lines (the last pair
# of the call half empty) and on 2 (a single pair)
@pytest.mark.parametrize("pairs", [1, 2, 3, 0])
@pytest.mark.parametrize("lines", [(7, 1), (1, 2), (1, 1)])
def test_pairs_per_workgroup(pairs, lines):
    env = {"HYENAND_MIXED_PAIRS": pairs} if pairs else {}
    _check("pairs", lines[0], lines[1], (14, 14), "circular", "f32", 600 + pairs, **env)
    _check("pairs", lines[0], lines[1], (15,), "centered", "f32", 610 + pairs, HYENAND_PLAN="mixed", **env)


# every radix family (the base radices 8, 7, 5, 4, 3, 2 and 14 + 12, 16 + 10,
# 15 + 9), forced on grids whose axes factor differently under each
@pytest.mark.parametrize("family", [0, 1, 2, 3])
@pytest.mark.parametrize("grid,mode", [((30, 28), "circular"), ((720,), "circular"), ((12, 10, 9), "circular"),
                                       ((14, 20), "centered"), ((2160,), "circular")])
def test_radix_families(family, grid, mode):
    assert _check("family", 2, 3, grid, mode, "f32", 800 + family, HYENAND_PLAN="mixed",
                  HYENAND_MIXED_FAMILY=family) == _mixed(len(grid))


# the largest grids these kernels take (3600 points, 144 KB of LDS, and 3840
# of at most 4096 points; one pair per workgroup) and unit axes squeezed away
@pytest.mark.parametrize("grid,mode", [((3600,), "circular"), ((16, 16, 15), "circular"), ((1, 14), "circular"),
                                       ((14, 1), "centered"), ((1, 1, 21), "linear")])
def test_extremes(grid, mode):
    plan = _check("extreme", 2, 3, grid, mode, "f32", 950 + sum(grid), HYENAND_PLAN="mixed")
    assert plan == _mixed(sum(1 for g in grid if g > 1))


@pytest.mark.parametrize("grid,mode", [((14, 14), "circular"), ((100,), "circular"), ((14, 14), "centered")])
def test_shared_kernel(grid, mode):
    _check("shared", 3, 4, grid, mode, "f32", 700, shared=True, HYENAND_PLAN="mixed")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("grid,mode", [((14, 14), "circular"), ((1000,), "circular"), ((15,), "centered"),
                                       ((6, 10, 14), "circular"), ((14, 14), "linear")])
def test_dynamic_range(grid, mode, dtype):
    """Two real signals share each complex transform (the u of two lines, the
    k of two lines, two lines' products), each scaled on its own.  Kernels
    1e4 times smaller than u, and the lines of each pair at scales apart by up
    to 1e7: every line within the tolerance of the oracle."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    B, C = 2, 4
    shape, x1, x2, v, k, D = _case(B, C, grid, mode, "f32", 900)
    line_scale = np.array([1e4, 1.0, 1e-3, 3.0, 1.0, 1e-2, 1e2, 1.0])
    x1 = x1 * line_scale.reshape((B, C) + (1,) * len(grid))
    k = k * 1e-4
    D = D * 1e-4
    x1, x2, v, k, D = (W.quantise(a, dtype) for a in (x1, x2, v, k, D))
    dev = [to_device(a, dtype) for a in (x1, x2, v, k, D)]
    with _env(HYENAND_PLAN="mixed"):
        assert H.plan_name(shape, mode, dtype) == _mixed(len(grid))
        y = H.fftconv(*dev, pad_mode=mode)
        torch.cuda.synchronize()
    got = from_device(y)
    f = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, k, D)]
    ref = (oracle.conv_direct if mode == "circular" else oracle.conv_fft)(*f, mode)
    worst = per_line_worst(got, ref, B * C)
    log(f"[mixed] dynamic range {shape} {mode} {dtype}: worst line={worst:.3e}")
    assert np.all(np.isfinite(got)) and worst <= TOL[dtype]


def test_image_patch_grid_batch():
    """A batch of 14 x 14 patch grids (the paper's ImageNet models' grid),
    circular: 16 x 384 images on 196-point transforms."""
    assert _check("patches", 16, 384, (14, 14), "circular", "f32", 11) == "mixed2d"
    summary("[mixed] 16 x 384 x 14 x 14 circular: whole tensor and every line within 1e-5 of the oracle")


@pytest.mark.parametrize("grid,mode", [((14, 14), "circular"), ((30,), "circular"), ((14, 14), "centered")])
def test_operator(grid, mode):
    import torch
    from paper_2607_19378_amd import hyenand as H
    rng = np.random.default_rng(5)
    shape = (3, 6) + grid
    q, kin, vin = (rng.standard_normal(shape).astype(np.float32) for _ in range(3))
    kshape = oracle.kernel_shape(shape, mode)
    k = (rng.standard_normal(kshape) / np.sqrt(np.prod(kshape[2:]))).astype(np.float32)
    D, wi, wo = (rng.standard_normal(6).astype(np.float32) for _ in range(3))
    dev = [to_device(a, "f32") for a in (q, kin, vin, k, D, wi, wo)]
    with _env(HYENAND_PLAN="mixed"):
        assert H.plan_name(shape, mode, "f32") == _mixed(len(grid))
        y = H.operator(*dev, pad_mode=mode)
        torch.cuda.synchronize()
    ref = oracle.operator(*[a.astype(np.float64) for a in (q, kin, vin, k, D, wi, wo)], pad_mode=mode)
    err = rel_l2(from_device(y), ref)
    log(f"[mixed] operator {shape} {mode}: rel_l2={err:.3e}")
    assert err <= TOL["f32"]


def test_same_result_as_power_of_two_kernels():
    """The mixed-radix and power-of-two single-pass kernels agree on the same
    inputs (both within the oracle's tolerance of each other)."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    shape, x1, x2, v, k, D = _case(4, 8, (14, 14), "circular", "f32", 9)
    dev = [to_device(a, "f32") for a in (x1, x2, v, k, D)]
    out = {}
    for route in ("mixed", "nomixed"):
        with _env(HYENAND_PLAN=route):
            out[route] = from_device(H.fftconv(*dev, pad_mode="circular"))
            torch.cuda.synchronize()
    assert rel_l2(out["mixed"], out["nomixed"]) <= 1e-5
