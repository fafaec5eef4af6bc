"""GPU backward against the oracle's backward (gradients through y for a
seeded gy), through the C ABI: every tensor element by element, within the
forward's tolerances (relative L2: fp32 1e-5, bf16 2e-2)."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
NAMES = ("gx1", "gx2", "gv", "gk", "gD")


def _run(shape, mode, dtype, seed):
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    log(f"backward case {shape} {mode} {dtype} seed {seed}")
    rng = np.random.default_rng(seed)
    host = [W.quantise(rng.standard_normal(shape), dtype) for _ in range(5)]
    Dh = W.quantise(rng.standard_normal(shape[1]), dtype)
    x1, x2, v, k, gy = host
    dev = [to_device(a, dtype) for a in (x1, x2, v, k)]
    got = H.backward(*dev, to_device(Dh, dtype), to_device(gy, dtype), mode)
    torch.cuda.synchronize()
    f64 = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, k, Dh, gy)]
    ref = oracle.backward_fft(*f64[:5], f64[5], mode)
    out = []
    for name, g, r in zip(NAMES, got, ref):
        gh = from_device(g)
        err = np.linalg.norm(gh - r) / max(np.linalg.norm(r), 1e-300)
        out.append((name, float(err)))
    return out


CASES = [
    ((2, 3, 16), "linear"), ((2, 3, 16), "circular"), ((1, 4, 256), "linear"), ((3, 2, 64), "circular"),
    ((1, 64, 4096), "linear"), ((1, 8, 4096), "circular"), ((2, 2, 1), "linear"), ((1, 3, 2), "circular"),
    ((2, 3, 4, 4), "linear"), ((2, 3, 8, 8), "circular"), ((1, 5, 16, 32), "linear"), ((2, 2, 32, 64), "circular"),
    ((3, 4, 64, 64), "linear"), ((2, 2, 32, 64), "linear"), ((1, 3, 64, 128), "circular"),
    ((1, 3, 128, 64), "circular"), ((3, 5, 32, 32), "circular"),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape,mode", CASES)
def test_backward_matches_oracle(shape, mode, dtype):
    errs = _run(shape, mode, dtype, 1234 + len(shape))
    print(f"backward {shape} {mode} {dtype}: " + " ".join(f"{n}={e:.2e}" for n, e in errs))
    for name, e in errs:
        assert e <= TOL[dtype], (name, e)


def test_backward_full_size_image_workload():
    """The 2D workload shape (8 x 256 images of 64 x 64, linear, fp32)."""
    errs = _run((8, 256, 64, 64), "linear", "f32", 99)
    print("backward 8x256x64x64: " + " ".join(f"{n}={e:.2e}" for n, e in errs))
    for name, e in errs:
        assert e <= TOL["f32"], (name, e)
