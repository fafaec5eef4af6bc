"""GPU backward on the multi-pass plans (2D/3D grids beyond LDS and long 1D
lines) against the oracle's backward, through the C ABI: every gradient
element by element on small and ragged cases and bitwise the same result
for every workspace size (the full workload shapes are compared element by
element in test_gpu_full_workloads.py)."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

from gpu_util import from_device, log, to_device

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
NAMES = ("gx1", "gx2", "gv", "gk", "gD")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _gy(shape, dtype, seed):
    return W.quantise(np.random.default_rng(seed).standard_normal(shape), dtype)


def _gpu_backward(inp, gy, workspace_bytes=None):
    import torch
    from paper_2607_19378_amd import hyenand as H
    w = inp.workload
    dev = [to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
    ws = None
    if workspace_bytes is not None:
        ws = torch.empty(workspace_bytes, dtype=torch.uint8, device="cuda")
    got = H.backward(*dev, to_device(gy, w.dtype), w.pad_mode, workspace=ws)
    torch.cuda.synchronize()
    return got


def _errs(got_host, ref):
    out = []
    for name, g, r in zip(NAMES, got_host, ref):
        err = np.linalg.norm(np.asarray(g, np.float64) - r) / max(np.linalg.norm(r), 1e-300)
        out.append((name, float(err)))
    return out


CASES = [
    ((1, 3, 256, 256), "linear", "f32"), ((2, 2, 64, 128), "linear", "bf16"), ((2, 3, 16, 32), "circular", "f32"),
    ((1, 2, 512, 512), "circular", "f32"), ((3, 2, 8, 4), "linear", "f32"), ((1, 2, 1024, 8), "circular", "bf16"),
    ((2, 2, 8, 16, 32), "linear", "f32"), ((1, 2, 32, 32, 32), "circular", "bf16"), ((1, 2, 16, 8, 64), "linear", "bf16"),
    ((2, 3, 4, 2, 8), "circular", "f32"), ((1, 2, 64, 64, 64), "linear", "f32"),
    ((1, 3, 8192), "linear", "f32"), ((2, 2, 16384), "circular", "bf16"),
    ((1, 3, 16384), "linear", "f32"), ((2, 2, 32768), "circular", "f32"), ((1, 2, 65536), "linear", "bf16"),
    ((1, 2, 1 << 20), "linear", "f32"),
    # the largest transforms the plans take: 2^22 points in 1D, 1024 on an axis
    ((1, 2, 1 << 21), "linear", "bf16"), ((1, 2, 1 << 22), "circular", "f32"), ((1, 2, 512, 512), "linear", "f32"),
    ((1, 2, 1024, 1024), "circular", "bf16"), ((1, 2, 512, 4, 8), "linear", "f32"),
    ((1, 2, 4, 1024, 16), "circular", "f32"), ((1, 2, 8, 4, 512), "linear", "bf16"),
]


@pytest.mark.parametrize("shape,mode,dtype", CASES)
def test_backward_multipass_matches_oracle(shape, mode, dtype):
    B, C, grid = shape[0], shape[1], shape[2:]
    inp = W.random_case(B, C, grid, mode, dtype, seed=700 + sum(shape))
    gy = _gy(shape, dtype, 800 + sum(shape))
    log(f"[bwd-mp] {shape} {mode} {dtype}")
    got = [from_device(g) for g in _gpu_backward(inp, gy)]
    f64 = [W.storage_to_f64(a, dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D, gy)]
    ref = oracle.backward_fft(*f64[:5], f64[5], mode)
    errs = _errs(got, ref)
    log(f"[bwd-mp] {shape} {mode} {dtype}: " + " ".join(f"{n}={e:.2e}" for n, e in errs))
    for name, e in errs:
        assert e <= TOL[dtype], (name, e)


@pytest.mark.parametrize("shape,mode,dtype", [((1, 5, 128, 256), "linear", "f32"), ((1, 3, 8, 8, 64), "circular", "f32"),
                                              ((1, 5, 32768), "linear", "bf16")])
def test_backward_workspace_sizes_bitwise(shape, mode, dtype):
    """One line of spectra per chunk, two lines, and the recommended size give
    the same bits (chunking and side streams only change the launch order)."""
    from paper_2607_19378_amd import hyenand as H
    B, C, grid = shape[0], shape[1], shape[2:]
    inp = W.random_case(B, C, grid, mode, dtype, seed=41)
    gy = _gy(shape, dtype, 42)
    wmin = H.backward_workspace_min(shape, mode, dtype)
    wrec = H.backward_workspace_size(shape, mode, dtype)
    log(f"[bwd-ws] {shape}: min={wmin} rec={wrec}")
    assert 0 < wmin <= wrec
    runs = [[from_device(g) for g in _gpu_backward(inp, gy, n)] for n in (wmin, 2 * wmin, wrec)]
    for other in runs[1:]:
        for a, b in zip(runs[0], other):
            assert np.array_equal(a, b)
