"""One kernel per channel on the single-pass 2D plan: with the workspace that
hyenand_fftconv_shared_k_workspace_size reports, each channel's kernel is
transformed once and every image of that channel reads the spectrum.  Checked
against the oracle (k repeated for every sample) on every instantiated
transform grid, against the same call without the workspace (each image
transforms k itself), and on the fallbacks (one sample, a short workspace).
Kernel spectra kept across calls (hyenand_kernel_spectrum and
hyenand_fftconv_spectrum) against the one-call path and the oracle."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def _inputs(shape, dtype, seed):
    rng = np.random.default_rng(seed)
    x1, x2, v = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
    kc = W.quantise(rng.standard_normal(shape[1:]), dtype)
    D = W.quantise(rng.standard_normal(shape[1]), dtype)
    return x1, x2, v, kc, D


def _oracle(arrs, shape, mode, dtype):
    f = [W.storage_to_f64(a, dtype) for a in arrs]
    kfull = np.ascontiguousarray(np.broadcast_to(f[3], shape))
    return oracle.conv_fft(f[0], f[1], f[2], kfull, f[4], mode)


def _run(dev, shape, mode, dtype, ws_bytes):
    """hyenand_fftconv_shared_k with a workspace of ws_bytes (None: NULL)."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    y = torch.empty_like(dev[0])
    ws = None if ws_bytes is None else torch.empty(max(1, ws_bytes), dtype=torch.uint8, device=dev[0].device)
    H.fftconv_into(y, *dev, pad_mode=mode, workspace=ws, shared_k=True)
    torch.cuda.synchronize()
    return y


GRIDS = [(4, 4), (8, 8), (16, 16), (32, 32), (64, 64), (128, 128), (64, 128), (128, 64), (32, 64), (64, 32)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("mode", ["linear", "circular"])
@pytest.mark.parametrize("grid", GRIDS)
def test_khat_path_matches_oracle_and_per_image_path(grid, mode, dtype):
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    P = grid
    L = tuple(p // 2 for p in P) if mode == "linear" else P
    shape = (3, 5) + L
    log(f"khat case {shape} {mode} {dtype}")
    assert H.plan_name(shape, mode, dtype) == "fused2d"
    need = H.workspace_size(shape, mode, dtype, shared_k=True)
    assert need == -(-5 * P[0] * (P[1] // 2) * 8 // 256) * 256
    assert H.workspace_size(shape, mode, dtype) == 0
    arrs = _inputs(shape, dtype, 97 + P[0] + 3 * P[1])
    dev = [to_device(a, dtype) for a in arrs]
    got = from_device(_run(dev, shape, mode, dtype, need))
    per_image = from_device(_run(dev, shape, mode, dtype, None))
    ref = _oracle(arrs, shape, mode, dtype)
    err = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    worst = max(float(np.linalg.norm(got[b, c] - ref[b, c]) / np.linalg.norm(ref[b, c]))
                for b in range(shape[0]) for c in range(shape[1]))
    diff = float(np.abs(got - per_image).max())
    print(f"khat {shape} {mode} {dtype}: rel_l2={err:.2e} worst line={worst:.2e} max|khat - per-image|={diff:.1e}")
    assert err <= TOL[dtype] and worst <= TOL[dtype]
    # the same arithmetic on k, once per channel instead of once per image
    scale = float(np.abs(ref).max())
    assert diff <= (1e-6 if dtype == "f32" else 1e-2) * scale


@pytest.mark.parametrize("shape", [(3, 8, 16, 16), (2, 24, 32, 32), (5, 16, 16, 32)])
def test_khat_channel_multiple_of_8(shape):
    """C a multiple of 8: the images run in the XCD-grouped order (the B
    images of a channel on one XCD); every (b, c) still gets its own output."""
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    log(f"khat xcd order {shape}")
    arrs = _inputs(shape, "f32", 11 + shape[1])
    dev = [to_device(a, "f32") for a in arrs]
    assert H.plan_name(shape, "linear", "f32") == "fused2d"
    need = H.workspace_size(shape, "linear", "f32", shared_k=True)
    assert need > 0
    got = from_device(_run(dev, shape, "linear", "f32", need))
    per_image = from_device(_run(dev, shape, "linear", "f32", None))
    ref = _oracle(arrs, shape, "linear", "f32")
    worst = max(float(np.linalg.norm(got[b, c] - ref[b, c]) / np.linalg.norm(ref[b, c]))
                for b in range(shape[0]) for c in range(shape[1]))
    diff = float(np.abs(got - per_image).max())
    print(f"khat xcd order {shape}: worst line={worst:.2e} max|khat - per-image|={diff:.1e}")
    assert worst <= TOL["f32"]
    assert diff <= 1e-6 * float(np.abs(ref).max())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_khat_fallbacks(dtype):
    """One sample (nothing to share), and a workspace below the spectra's
    size: the per-image path runs and gives the oracle's results."""
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    for shape, ws in (((1, 6, 64, 64), "query"), ((4, 3, 32, 32), "short")):
        log(f"khat fallback {shape} {ws} {dtype}")
        need = H.workspace_size(shape, "linear", dtype, shared_k=True)
        if ws == "query":
            assert need == 0
            nbytes = need
        else:
            assert need > 0
            nbytes = need - 256
        arrs = _inputs(shape, dtype, 5 + shape[0])
        dev = [to_device(a, dtype) for a in arrs]
        got = from_device(_run(dev, shape, "linear", dtype, nbytes))
        ref = _oracle(arrs, shape, "linear", dtype)
        err = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        print(f"khat fallback {shape} {ws} {dtype}: rel_l2={err:.2e}")
        assert err <= TOL[dtype]


def test_khat_workload_size():
    """8 x 256 images of 64 x 64 (128 x 128 transforms), fp32: the spectra
    path against the per-image path over the whole tensor, and against the
    oracle on sampled (b, c) lines."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    shape, mode, dtype = (8, 256, 64, 64), "linear", "f32"
    log(f"khat workload {shape}")
    arrs = _inputs(shape, dtype, 2026)
    dev = [to_device(a, dtype) for a in arrs]
    need = H.workspace_size(shape, mode, dtype, shared_k=True)
    assert need == 256 * 128 * 64 * 8
    got = from_device(_run(dev, shape, mode, dtype, need))
    per_image = from_device(_run(dev, shape, mode, dtype, None))
    diff = float(np.abs(got - per_image).max())
    f = [W.storage_to_f64(a, dtype) for a in arrs]
    rng = np.random.default_rng(7)
    worst = 0.0
    for b, c in zip(rng.integers(0, 8, 12), rng.integers(0, 256, 12)):
        ref = oracle.conv_fft(f[0][b:b + 1, c:c + 1], f[1][b:b + 1, c:c + 1], f[2][b:b + 1, c:c + 1],
                              f[3][c:c + 1][None], f[4][c:c + 1], mode)[0, 0]
        worst = max(worst, float(np.linalg.norm(got[b, c] - ref) / np.linalg.norm(ref)))
    print(f"khat workload: worst sampled line rel_l2={worst:.2e} max|khat - per-image|={diff:.1e}")
    assert worst <= TOL[dtype]
    assert diff <= 1e-6 * float(np.abs(per_image).max())
    del dev
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("mode,grid", [("linear", (64, 64)), ("circular", (32, 64)), ("linear", (16, 16))])
def test_kept_spectra_serve_several_calls(mode, grid, dtype):
    """One kernel_spectrum, then convolutions of two input sets and of a
    different batch size from the same spectra: bitwise the one-call shared-k
    results, and the oracle's within the tolerance."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import from_device, log, to_device
    C = 8
    log(f"kept spectra {mode} {grid} {dtype}")
    arrs = _inputs((3, C) + grid, dtype, 31 + grid[0])
    kc_dev = to_device(arrs[3], dtype)
    D_dev = to_device(arrs[4], dtype)
    khat = H.kernel_spectrum(kc_dev, (3, C) + grid, mode)
    assert khat.numel() == H.kernel_spectrum_size((1, C) + grid, mode, dtype)
    rng = np.random.default_rng(5)
    for B in (3, 3, 1):
        shape = (B, C) + grid
        x1, x2, v = (W.quantise(rng.standard_normal(shape), dtype) for _ in range(3))
        dev = [to_device(a, dtype) for a in (x1, x2, v)]
        y = H.fftconv_spectrum(dev[0], dev[1], dev[2], khat, D_dev, mode)
        torch.cuda.synchronize()
        got = from_device(y)
        one_call = from_device(H.fftconv(dev[0], dev[1], dev[2], kc_dev, D_dev, pad_mode=mode, shared_k=True))
        ref = _oracle((x1, x2, v, arrs[3], arrs[4]), shape, mode, dtype)
        err = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        print(f"kept spectra {mode} {grid} {dtype} B={B}: rel_l2={err:.2e}")
        assert err <= TOL[dtype]
        if B >= 2:  # the one-call path uses the spectra too (B = 1 transforms k per image)
            assert np.array_equal(got, one_call)
