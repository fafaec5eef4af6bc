"""Helpers shared by the GPU parity tests: move seeded storage arrays to the
GPU, run the HIP path through the C ABI, and compare with the fp64 oracle."""
import sys

import numpy as np

from paper_2607_19378_amd import workloads as W

TOL = {"f32": 1e-5, "bf16": 2e-2}  # relative L2, fp32 compute in both cases


def log(msg):
    sys.stdout.write(msg + "\n")
    sys.stdout.flush()


# result lines printed in the terminal summary of the run (pytest keeps a
# passing test's own output to itself)
SUMMARY = []


def summary(msg):
    log(msg)
    SUMMARY.append(msg)


def to_device(arr, dtype):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).cuda()
    return t.view(torch.bfloat16)


def from_device(t):
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return W.bf16_bits_to_f64(bits)
    return t.cpu().numpy().astype(np.float64)


def run_gpu(inp, workspace_bytes=None, stream=None):
    import torch
    from paper_2607_19378_amd import hyenand as H
    w = inp.workload
    dev = [to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
    ws = None
    if workspace_bytes is not None:
        ws = torch.empty(max(1, workspace_bytes), dtype=torch.uint8, device="cuda")
    y = H.fftconv(*dev, pad_mode=w.pad_mode, workspace=ws, stream=stream)
    torch.cuda.synchronize()
    return from_device(y)


def oracle_ref(inp, lines=None, method="fft"):
    import oracle
    x1, x2, v, k, D = inp.as_f64()
    fn = oracle.conv_fft if method == "fft" else oracle.conv_direct
    return fn(x1, x2, v, k, D, inp.workload.pad_mode, lines=lines)


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def per_line_worst(a, b, nlines):
    a = np.asarray(a, dtype=np.float64).reshape(nlines, -1)
    b = np.asarray(b, dtype=np.float64).reshape(nlines, -1)
    num = np.linalg.norm(a - b, axis=1)
    den = np.maximum(np.linalg.norm(b, axis=1), 1e-300)
    return float(np.max(num / den))


def oracle_lines(inp, lines):
    """Oracle output of selected flat (b*C + c) lines, shape [len(lines), grid...].

    Each selected line becomes one channel of a B=1 sub-problem carrying its
    own D[c], so only the selected lines are upcast and computed."""
    import oracle
    w = inp.workload
    nl = w.B * w.C
    lines = np.asarray(lines, dtype=np.int64)
    sub = []
    for a in (inp.x1, inp.x2, inp.v, inp.k):
        flat = a.reshape((nl,) + tuple(a.shape[2:]))[lines]  # k: the double grid when centered
        sub.append(W.storage_to_f64(flat, w.dtype)[None])
    Dsub = W.storage_to_f64(inp.D, w.dtype)[lines % w.C]
    return oracle.conv_fft(sub[0], sub[1], sub[2], sub[3], Dsub, w.pad_mode)[0]
