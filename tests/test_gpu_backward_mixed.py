"""Backward on the mixed-radix transform grids (hyenand_fftconv_backward's
single pass for extents that are not powers of two): every gradient against
the oracle's direct-sum backward, whole tensors and the worst line, every
pad mode, fp32 and bf16, 1D/2D/3D, odd line counts, several pairs per
workgroup, every radix family, and inputs of very different scales."""
import os

import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

from gpu_util import TOL, from_device, log, per_line_worst, rel_l2, summary, to_device

pytestmark = pytest.mark.gpu

NAMES = ("gx1", "gx2", "gv", "gk", "gD")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


class _env:
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


def _mixed_workspace(shape):
    """The mixed-radix backward's workspace: one float per line (gD sums)."""
    return (shape[0] * shape[1] * 4 + 255) // 256 * 256


def _check(shape, mode, dtype, seed, scales=None, kscale=1.0, **env):
    import torch
    from paper_2607_19378_amd import hyenand as H
    rng = np.random.default_rng(seed)
    kshape = oracle.kernel_shape(shape, mode)
    npts = int(np.prod(kshape[2:]))
    x1, x2, v, gy = (rng.standard_normal(shape) for _ in range(4))
    k = rng.standard_normal(kshape) / np.sqrt(npts) * kscale
    D = rng.standard_normal(shape[1]) * kscale
    if scales is not None:  # per-line scales of x1 and gy
        s = np.asarray(scales).reshape(shape[:2] + (1,) * (len(shape) - 2))
        x1, gy = x1 * s, gy * s[::-1]
    x1, x2, v, gy, k, D = (W.quantise(a, dtype) for a in (x1, x2, v, gy, k, D))
    dev = [to_device(a, dtype) for a in (x1, x2, v, k, D, gy)]
    with _env(**env):
        assert H.backward_workspace_min(shape, mode, dtype) == _mixed_workspace(shape), "not the mixed-radix plan"
        outs = H.backward(*dev, pad_mode=mode)
        torch.cuda.synchronize()
    f = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, k, D, gy)]
    refs = oracle.backward_direct(*f, pad_mode=mode)
    nl = shape[0] * shape[1]
    errs, worst = {}, {}
    for n, o, r in zip(NAMES, outs, refs):
        got = from_device(o)
        assert got.shape == r.shape and np.all(np.isfinite(got))
        errs[n] = rel_l2(got, r)
        if n != "gD":
            worst[n] = per_line_worst(got, r, nl)
    log(f"[bwd-mixed] {shape} {mode} {dtype} {env}: " + " ".join(f"{n}={e:.2e}" for n, e in errs.items())
        + " worst line " + " ".join(f"{n}={e:.2e}" for n, e in worst.items()))
    assert max(errs.values()) <= TOL[dtype] and max(worst.values()) <= TOL[dtype], (errs, worst)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(3, 5, 14, 14), (2, 3, 12), (1, 3, 1000), (3, 5, 3, 5), (1, 2, 12, 12, 12),
                                   (2, 3, 6, 10, 14), (3, 3, 48, 64)])
def test_circular(shape, dtype):
    _check(shape, "circular", dtype, 1 + sum(shape))


@pytest.mark.parametrize("shape", [(2, 3, 13, 14), (2, 3, 14, 11), (2, 3, 13), (1, 2, 11, 13)])
def test_periodic_axes(shape):
    """A circular axis of 13 or 11 points: k periodic on P >= 2L - 1; gk
    gathers both displacements of each kernel point."""
    _check(shape, "circular", "f32", 2 + sum(shape))


@pytest.mark.parametrize("mode", ["linear", "centered"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(3, 5, 14, 14), (2, 3, 15), (2, 3, 100), (1, 2, 5, 6, 7), (2, 3, 7, 30),
                                   (2, 3, 2, 3)])
def test_noncircular(shape, mode, dtype):
    _check(shape, mode, dtype, 3 + sum(shape))


@pytest.mark.parametrize("pairs", [1, 2, 3])
@pytest.mark.parametrize("lines", [(7, 1), (1, 1)])
def test_pairs_per_workgroup(pairs, lines):
    _check(lines + (14, 14), "circular", "f32", 4 + pairs, HYENAND_MIXED_PAIRS=pairs)
    _check(lines + (15,), "centered", "f32", 5 + pairs, HYENAND_MIXED_PAIRS=pairs)


@pytest.mark.parametrize("family", [0, 1, 2, 3])
@pytest.mark.parametrize("shape,mode", [((2, 3, 30, 28), "circular"), ((2, 3, 720), "circular"),
                                        ((2, 3, 14, 20), "centered")])
def test_radix_families(family, shape, mode):
    _check(shape, mode, "f32", 6 + family, HYENAND_MIXED_FAMILY=family)


@pytest.mark.parametrize("shape,mode", [((2, 4, 14, 14), "circular"), ((2, 4, 15), "centered"),
                                        ((2, 4, 6, 10, 14), "circular")])
def test_dynamic_range(shape, mode):
    """Kernels and D 1e4 times below the data; x1 and gy of the lines of a
    pair at scales apart by up to 1e7."""
    _check(shape, mode, "f32", 7, scales=[1e4, 1.0, 1e-3, 3.0, 1.0, 1e-2, 1e2, 1.0], kscale=1e-4)


def test_image_patch_grid_batch():
    """A batch of 14 x 14 patch grids with centered kernels (the patch-16
    ImageNet grid), 16 x 384 lines, every gradient."""
    _check((16, 384, 14, 14), "centered", "f32", 8)
    summary("[bwd-mixed] 16 x 384 x 14 x 14 centered: every gradient within 1e-5 of the oracle (whole tensor "
            "and every line)")
