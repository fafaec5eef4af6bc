"""Seeded input generators: determinism, shapes, one-step RNE rounding."""
import hashlib

import numpy as np
import pytest

from paper_2607_19378_amd import workloads as W


def test_registry_shapes():
    assert [W.WORKLOADS[n].shape for n in W.ORDER] == [
        (1, 64, 4096), (8, 256, 64, 64), (4, 128, 512, 512), (1, 64, 128, 128, 128), (1, 256, 1 << 20)]
    assert [W.WORKLOADS[n].pad_mode for n in W.ORDER] == ["linear", "linear", "circular", "linear", "linear"]
    assert [W.WORKLOADS[n].dtype for n in W.ORDER] == ["f32", "f32", "f32", "bf16", "bf16"]


def _digest(inp):
    h = hashlib.sha256()
    for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def test_generation_is_deterministic():
    w = W.WORKLOADS["conv2d_64"].scaled(B=2, C=3, name="small")
    assert _digest(W.generate(w)) == _digest(W.generate(w))
    w2 = w.scaled(seed=w.seed + 1)
    assert _digest(W.generate(w)) != _digest(W.generate(w2))


def test_bf16_rounding_is_single_rne():
    # exact bf16 values survive; ties go to even; no double rounding through fp32
    vals = np.array([1.0, -2.5, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -30, 3.0e-5])
    bits = W.round_to_bf16_bits(vals)
    back = W.bf16_bits_to_f64(bits)
    assert back[0] == 1.0 and back[1] == -2.5
    assert back[2] == 1.0                      # tie -> even (down)
    assert back[3] == 1.0 + 4 * 2 ** -8        # tie -> even (up)
    assert back[4] == 1.0 + 2 * 2 ** -8        # just above the tie -> up (fp32 first would tie)
    assert abs(back[5] - 3.0e-5) <= 2 ** -8 * 3.0e-5
    rng = np.random.default_rng(0)
    x = rng.standard_normal(10000)
    r = W.bf16_bits_to_f64(W.round_to_bf16_bits(x))
    assert np.max(np.abs(r - x) / np.abs(x)) <= 2 ** -8 * (1 + 1e-12)  # unit roundoff of p = 8


def test_kernel_windows():
    w = W.WORKLOADS["conv1d_4k"]
    win = W.decay_window(w.grid, w.tau, periodic=False)
    assert win[0] == 1.0 and abs(win[1024] - np.exp(-1.0)) < 1e-15
    win2 = W.decay_window((8, 8), 2.0, periodic=True)
    assert win2[1, 7] == win2[1, 1] == win2[7, 7]


def test_smooth_fields_unit_variance_and_periodic():
    rng = np.random.default_rng(1)
    noise = rng.standard_normal((2, 64, 64))
    f = W.smooth_fields(noise, 4.0)
    assert np.allclose(f.mean(axis=(1, 2)), 0, atol=1e-12)
    assert np.allclose(f.std(axis=(1, 2)), 1, atol=1e-12)
    # periodic filter commutes with a roll of the input
    g = W.smooth_fields(np.roll(noise, (5, 9), axis=(1, 2)), 4.0)
    assert np.allclose(g, np.roll(f, (5, 9), axis=(1, 2)), atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_random_case_dtypes(dtype):
    inp = W.random_case(2, 3, (8, 4), "linear", dtype, seed=5)
    want = np.float32 if dtype == "f32" else np.uint16
    for a in (inp.x1, inp.x2, inp.v, inp.k):
        assert a.dtype == want and a.shape == (2, 3, 8, 4)
    assert inp.D.shape == (3,)


def test_bench_algorithmic_flops():
    """Per-call flop count used for the ALU roofline: three pruned real FFTs
    (5 n log2 n complex, 2.5 n log2 n real), 6 flops per half-spectrum
    product, 4 per output.  The 64x64 image (128x128 padded) written out:
    forward rows 64 x 2.5*128*7, forward columns 65 x 5*128*7 (u and k),
    inverse columns 65 x 5*128*7, inverse rows 64 x 2.5*128*7."""
    import bench
    w = W.WORKLOADS["conv2d_64"]
    fwd = 64 * 2.5 * 128 * 7 + 65 * 5 * 128 * 7
    inv = 65 * 5 * 128 * 7 + 64 * 2.5 * 128 * 7
    per_img = 2 * fwd + inv + 6 * 128 * 65 + 4 * 64 * 64
    assert bench.alg_flops(w) == per_img * 8 * 256
    # 1D 2^20 linear: real transforms of 2^21 points
    w = W.WORKLOADS["conv1d_1m"]
    n = 2 ** 21
    per_line = 3 * 2.5 * n * 21 + 6 * (n // 2 + 1) + 4 * 2 ** 20
    assert abs(bench.alg_flops(w) - per_line * 256) < 1e-6 * per_line


def test_bench_settle_count():
    """The untimed settling calls: a fixed count per workload worth about the
    requested time at the rough per-call rate, at least one, at most 2000,
    none when switched off."""
    import bench
    w = W.WORKLOADS["conv2d_64"]
    f, b = bench.alg_flops(w), bench.alg_bytes(w)
    n = bench.settle_count(f, b, 30.0)
    per_call = max(b / 5e12, f / (0.5 * bench.FP32_VALU_TFLOPS * 1e12))
    assert n == int(np.ceil(0.030 / per_call)) and 100 < n < 2000
    assert bench.settle_count(f, b, 60.0) >= 2 * n - 1
    assert bench.settle_count(f, b, 0.0) == 0
    tiny = W.WORKLOADS["conv1d_4k"]
    assert bench.settle_count(bench.alg_flops(tiny), bench.alg_bytes(tiny), 30.0) == 2000
    big = W.WORKLOADS["conv3d_128"]
    assert 1 <= bench.settle_count(bench.alg_flops(big), bench.alg_bytes(big), 30.0) < 50


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus above 1 exits with a message and
    status 2 before touching a device."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
