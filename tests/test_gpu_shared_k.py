"""One kernel per channel (k of shape [C, L...], hyenand_fftconv_shared_k)
against the oracle run with that kernel repeated for every sample, on every
forward plan."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def _run(shape, mode, dtype, seed, plan=None, monkeypatch=None):
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    if plan:
        monkeypatch.setenv("HYENAND_PLAN", plan)
    log(f"shared-k case {shape} {mode} {dtype} plan {plan or 'default'}")
    rng = np.random.default_rng(seed)
    x1, x2, v = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
    kc = W.quantise(rng.standard_normal(shape[1:]), dtype)
    D = W.quantise(rng.standard_normal(shape[1]), dtype)
    dev = [to_device(a, dtype) for a in (x1, x2, v, kc, D)]
    y = H.fftconv(*dev, pad_mode=mode, shared_k=True)
    torch.cuda.synchronize()
    got = from_device(y)
    f = [W.storage_to_f64(a, dtype) for a in (x1, x2, v, kc, D)]
    kfull = np.ascontiguousarray(np.broadcast_to(f[3], shape))
    ref = oracle.conv_fft(f[0], f[1], f[2], kfull, f[4], mode)
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape,mode,plan", [
    ((3, 5, 256), "linear", None), ((2, 3, 1024), "circular", None),        # fused 1D
    ((3, 4, 32, 32), "linear", None), ((2, 3, 64, 64), "circular", None),   # fused 2D
    ((3, 2, 16, 64), "linear", "multipass"), ((2, 3, 8, 16, 32), "circular", None),  # multi-pass 2D / 3D
    ((3, 2, 1 << 15), "linear", None),                                      # four-step 1D
])
def test_shared_kernel_matches_oracle(shape, mode, plan, dtype, monkeypatch):
    err = _run(shape, mode, dtype, 4321 + len(shape), plan, monkeypatch)
    print(f"shared-k {shape} {mode} {dtype}: rel_l2={err:.2e}")
    assert err <= TOL[dtype]
