"""Benchmark of the gated N-D FFT long convolution on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one call of hyenand_fftconv over the whole workload (every step of
the path: gate, pad, forward FFTs, spectral product with the folded shortcut,
inverse FFT, crop, outer gate) with inputs already resident in HBM.  Several
independent input sets are rotated so the working set exceeds the 256 MiB
Infinity Cache and every step streams its inputs from HBM.  Before the W
warmup steps the same calls run untimed for --settle-ms (30 ms), so that the
GPU has left the low clocks of the idle time spent generating inputs; then
exactly K steps are timed.

With no --workload, the headline workload (8 x 256 images of 64 x 64, fp32)
and then each of the five workload configurations are timed in turn; one
JSON line reports the headline (GElem/s, its HBM-roofline fraction from HIP
events on the launch stream, the CPU oracle on a bounded sample) and a
per_config list with the same figures for every configuration, then an
extra_workloads list with the 14 x 14 patch-grid workload (extents that are
not powers of two, on the mixed-radix kernels).  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_19378_amd import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
# fp32 vector peak: 256 CUs x 4 SIMDs x 16 lanes x 2 flop (FMA) x 2.4 GHz.  The
# packed fp32 forms (two values per lane, 157.3 TFLOP/s) are not issued by
# these kernels, so 78.6 is the attainable peak.
FP32_VALU_TFLOPS = 78.6
FP32_PACKED_TFLOPS = 157.3
MALL_BYTES = 256 << 20
DEFAULT_WORKLOAD = "conv2d_64"
# the five configurations of the metric, in the order they are reported
CONFIG_ORDER = ["conv1d_4k", "conv2d_64", "conv2d_512c", "conv3d_128", "conv1d_1m"]
# timed after the five in the default run and listed apart: the 14 x 14 patch
# grid, whose extents are not powers of two (the mixed-radix kernels)
EXTRA_ORDER = ["conv2d_14_patches"]


def alg_bytes(w: W.Workload) -> int:
    """Read x1, v, x2 and k and write y once (D is C values); k has the grid's
    points, or 2 L_d - 1 per axis in the centered mode."""
    kelems = int(np.prod(w.kernel_shape))
    return (4 * w.elems + kelems) * w.storage_bytes


def alg_flops(w: W.Workload) -> float:
    """Algorithmic flops of one call: three line-pruned real N-D FFTs on the
    padded grid (5 n log2 n per complex line, 2.5 n log2 n per real line; only
    lines that can be nonzero or that the crop keeps), 6 flops per complex
    product of the half spectrum, 4 flops per output element."""
    import math
    n = w.ndim
    L = list(w.grid)
    P = [x if w.pad_mode == "circular" else 2 * x for x in L]
    H = P[-1] // 2 + 1

    def cplx(m):
        return 5.0 * m * math.log2(m) if m > 1 else 0.0

    def real(m):
        return 2.5 * m * math.log2(m) if m > 1 else 0.0

    # forward: last axis real on the nonzero lines, then axes n-2 .. 0
    ext = L[:-1] + [H]
    fwd = real(P[-1]) * math.prod(L[:-1])
    for d in range(n - 2, -1, -1):
        fwd += cplx(P[d]) * math.prod(ext[:d] + ext[d + 1:])
        ext[d] = P[d]
    # inverse: axes 0 .. n-2 (each then cropped), then the last axis real
    ext = P[:-1] + [H]
    inv = 0.0
    for d in range(n - 1):
        inv += cplx(P[d]) * math.prod(ext[:d] + ext[d + 1:])
        ext[d] = L[d]
    inv += real(P[-1]) * math.prod(L[:-1])
    # k: the same pruned transform, or (centered) every line of the full grid
    if w.pad_mode == "centered":
        ext = P[:-1] + [H]
        fwd_k = real(P[-1]) * math.prod(P[:-1])
        for d in range(n - 1):
            fwd_k += cplx(P[d]) * math.prod(ext[:d] + ext[d + 1:])
    else:
        fwd_k = fwd
    per_line = fwd + fwd_k + inv + 6.0 * math.prod(P[:-1]) * H + 4.0 * math.prod(L)
    return per_line * w.B * w.C


def alg_flops_backward(w: W.Workload) -> float:
    """Backward: three forward and three inverse pruned real transforms (u, k,
    h in; z, gu, gk out), three half-spectrum products, 8 flops per element
    (u, h, gx2, gx1, gv and the h u sum)."""
    import math
    n = w.ndim
    L = list(w.grid)
    P = [x if w.pad_mode == "circular" else 2 * x for x in L]
    H = P[-1] // 2 + 1

    def cplx(m):
        return 5.0 * m * math.log2(m) if m > 1 else 0.0

    def real(m):
        return 2.5 * m * math.log2(m) if m > 1 else 0.0

    ext = L[:-1] + [H]
    fwd = real(P[-1]) * math.prod(L[:-1])
    for d in range(n - 2, -1, -1):
        fwd += cplx(P[d]) * math.prod(ext[:d] + ext[d + 1:])
        ext[d] = P[d]
    ext = P[:-1] + [H]
    inv = 0.0
    for d in range(n - 1):
        inv += cplx(P[d]) * math.prod(ext[:d] + ext[d + 1:])
        ext[d] = L[d]
    inv += real(P[-1]) * math.prod(L[:-1])
    per_line = 3 * fwd + 3 * inv + 3 * 6.0 * math.prod(P[:-1]) * H + 8.0 * math.prod(L)
    return per_line * w.B * w.C


def bench_backward(args, w, inp):
    """Time hyenand_fftconv_backward on the workload (dLoss/dy a seeded
    normal tensor); prints one JSON line of the same form as the forward's."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    rng = np.random.default_rng(w.seed + 7)
    gy_host = W.quantise(rng.standard_normal(w.shape), w.dtype)
    # read x1, x2, v, gy and k; write gx1, gx2, gv and gk (k and gk have the
    # kernel's shape: 2 L - 1 points per axis in the centred mode)
    kelems = int(np.prod(w.kernel_shape))
    set_bytes = (7 * w.elems + 2 * kelems) * w.storage_bytes
    rot = args.rotate or max(1, min(8, int(np.ceil(2 * MALL_BYTES / set_bytes))))
    dev = torch.device("cuda:0")
    base = [to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D, gy_host)]
    sets = [base] + [[t.clone() for t in base] for _ in range(1, rot)]
    outs = [[torch.empty_like(base[0]) for _ in range(3)] + [torch.empty_like(base[3]), torch.empty_like(base[4])]
            for _ in range(rot)]
    ws = torch.empty(H.backward_workspace_size(w.shape, w.pad_mode, w.dtype), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    calls = [H.PreparedBackward(*o, *st, w.pad_mode, ws, stream) for o, st in zip(outs, sets)]
    settle_clocks(lambda i: calls[i % rot](), settle_count(alg_flops_backward(w), set_bytes, args.settle_ms))
    for i in range(args.warmup):
        calls[i % rot]()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        calls[i % rot]()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    avg_s = ev0.elapsed_time(ev1) * 1e-3 / args.steps
    ms_per_step = wall * 1e3 / args.steps
    flops = alg_flops_backward(w)
    hbm_gbs = set_bytes / avg_s / 1e9
    alu_tflops = flops / avg_s / 1e12
    alu_bound = flops / (FP32_VALU_TFLOPS * 1e12) > set_bytes / (HBM_PEAK_GBS * 1e9)
    if alu_bound:
        roofline = {"bound": "alu", "achieved": round(alu_tflops, 3), "peak": FP32_VALU_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(alu_tflops / FP32_VALU_TFLOPS, 4)}
    else:
        roofline = {"bound": "hbm", "achieved": round(hbm_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(hbm_gbs / HBM_PEAK_GBS, 4)}
    roofline.update({"traffic": None, "hbm_frac": round(hbm_gbs / HBM_PEAK_GBS, 4),
                     "alu_frac": round(alu_tflops / FP32_VALU_TFLOPS, 4), "alg_bytes_per_call": set_bytes,
                     "alg_flops_per_call": round(flops), "avg_call_us": round(avg_s * 1e6, 3)})
    parity = None
    cpu = None
    if not args.no_parity or not args.no_cpu_baseline:
        # the lines of a few channels over every sample (so gD[c] is complete),
        # all of them for small workloads
        import oracle
        nl = w.B * w.C
        centred = w.pad_mode == W.CENTERED  # the oracle's centred backward is the direct sums
        chans = list(range(w.C)) if w.elems <= (1 << 24) and not centred else sorted({0, w.C - 1})
        lines = np.array([b * w.C + c for b in range(w.B) for c in chans], dtype=np.int64)
        sub = []
        for a in (inp.x1, inp.x2, inp.v, inp.k, gy_host):
            g = tuple(a.shape[2:])
            flat = a.reshape((nl,) + g)[lines]
            sub.append(W.storage_to_f64(flat, w.dtype).reshape((w.B, len(chans)) + g))
        Dsub = W.storage_to_f64(inp.D, w.dtype)[chans]
        t0 = time.perf_counter()
        ref = (oracle.backward_direct if centred else oracle.backward_fft)(sub[0], sub[1], sub[2], sub[3], Dsub,
                                                                          sub[4], w.pad_mode)
        dt = time.perf_counter() - t0
        if not args.no_parity:
            got = outs[(args.steps - 1) % rot]
            idx = torch.as_tensor(lines, device=dev)
            errs = []
            for j, (g, r) in enumerate(zip(got, ref)):
                g = g.reshape(nl, -1).index_select(0, idx) if j < 4 else g[chans]
                if g.dtype == torch.bfloat16:
                    gh = W.bf16_bits_to_f64(g.view(torch.int16).cpu().numpy().view(np.uint16))
                else:
                    gh = g.cpu().numpy().astype(np.float64)
                r = r.reshape(gh.shape)
                errs.append(float(np.linalg.norm(gh - r) / max(np.linalg.norm(r), 1e-300)))
            parity = max(errs)
        if not args.no_cpu_baseline:
            cpu = {"value": round(len(lines) * (w.elems // nl) / dt / 1e9, 6), "unit": "GElem/s",
                   "cores": oracle.default_threads(), "kind": "oracle",
                   "sample": f"{len(lines)} of the {nl} (b,c) lines of {w.name} (fp64 "
                             f"{'direct-sum' if centred else 'FFT'} oracle backward, {dt:.2f} s wall)"}
    out = {
        "metric": "gated N-D FFT-conv backward GElem/s and % of roofline on 1 MI355X",
        "value": round(w.elems / (ms_per_step * 1e-3) / 1e9, 3), "unit": "GElem/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded, shapes and distributions of the paper's workloads; gy seeded normal)",
        "config": {"workload": w.name, "pass": "backward", "B": w.B, "C": w.C, "grid": list(w.grid),
                   "pad_mode": w.pad_mode, "storage": w.dtype, "rotated_input_sets": rot},
        "roofline": roofline, "cpu_baseline": cpu, "parity_rel_l2_worst_tensor": parity,
        "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


def bench_operator(args, w, inp):
    """Time hyenand_operator (the whole HyenaND operator: normalised prologue,
    the gated long convolution, output RMSNorm) on the workload's shape, with
    x1, v, x2 as q, kin, vin; prints one JSON line."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    rng = np.random.default_rng(w.seed + 11)
    w_in = W.quantise(1.0 + 0.2 * rng.standard_normal(w.C), w.dtype)
    w_out = W.quantise(1.0 + 0.2 * rng.standard_normal(w.C), w.dtype)
    set_bytes = alg_bytes(w)  # q, kin, vin, k in and y out once: the fused minimum
    rot = args.rotate or max(1, min(8, int(np.ceil(2 * MALL_BYTES / set_bytes))))
    dev = torch.device("cuda:0")
    base = [to_device(a, w.dtype) for a in (inp.x1, inp.v, inp.x2, inp.k, inp.D, w_in, w_out)]
    sets = [base] + [[t.clone() for t in base] for _ in range(1, rot)]
    ys = [torch.empty_like(base[0]) for _ in range(rot)]
    ws = torch.empty(H.operator_workspace_size(w.shape, w.pad_mode, w.dtype), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    calls = [H.PreparedOperator(y, *st, 1e-6, 1e-6, w.pad_mode, ws, stream) for y, st in zip(ys, sets)]
    settle_clocks(lambda i: calls[i % rot](), settle_count(alg_flops(w), alg_bytes(w), args.settle_ms))
    for i in range(args.warmup):
        calls[i % rot]()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        calls[i % rot]()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    avg_s = ev0.elapsed_time(ev1) * 1e-3 / args.steps
    ms_per_step = wall * 1e3 / args.steps
    hbm_gbs = set_bytes / avg_s / 1e9
    parity = None
    if not args.no_parity:
        import oracle
        f64 = [W.storage_to_f64(a, w.dtype) for a in (inp.x1, inp.v, inp.x2, inp.k, inp.D, w_in, w_out)]
        ref = oracle.operator(*f64, eps_l2=1e-6, eps_rms=1e-6, pad_mode=w.pad_mode)
        yv = ys[(args.steps - 1) % rot]
        if yv.dtype == torch.bfloat16:
            got = W.bf16_bits_to_f64(yv.view(torch.int16).cpu().numpy().view(np.uint16))
        else:
            got = yv.cpu().numpy().astype(np.float64)
        parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    out = {
        "metric": "HyenaND operator (Eq. HyenaND) GElem/s on 1 MI355X",
        "value": round(w.elems / (ms_per_step * 1e-3) / 1e9, 3), "unit": "GElem/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded, shapes and distributions of the paper's workloads)",
        "config": {"workload": w.name, "pass": "operator", "B": w.B, "C": w.C, "grid": list(w.grid),
                   "pad_mode": w.pad_mode, "storage": w.dtype, "rotated_input_sets": rot},
        "roofline": {"bound": "hbm", "achieved": round(hbm_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(hbm_gbs / HBM_PEAK_GBS, 4), "traffic": None, "alg_bytes_per_call": set_bytes,
                     "avg_call_us": round(avg_s * 1e6, 3)},
        "cpu_baseline": None, "parity_rel_l2": parity, "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


SYNTH_HIDDEN, SYNTH_LAYERS = 64, 3
MFMA_F32_PEAK_TFLOPS = 157.3
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense


def synth_flops(w: W.Workload, hidden: int, layers: int) -> float:
    """Multiply-adds of kernel synthesis, 2 flops each: per grid point and
    sample the first layer (N x Hf), the hidden layers ((J - 1) x Hf x Hf) and
    the output projection (Hf x C); sines, FiLM and the window are not counted."""
    npos = int(np.prod(w.kernel_shape[2:]))
    per = len(w.grid) * hidden + (layers - 1) * hidden * hidden + hidden * w.C
    return 2.0 * w.B * npos * per


def bench_synth(args, w, inp):
    """Time hyenand_kernel_synth (the FiLM-modulated SIREN kernel and its
    window, Hf = 64, J = 3) on the workload's kernel grid, alone and followed
    by the gated convolution that consumes it; prints one JSON line."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    p = W.siren_params(w.seed + 21, len(w.grid), SYNTH_HIDDEN, SYNTH_LAYERS, w.C, w.B)
    d = {k: (None if v is None else torch.from_numpy(v).to(dev)) for k, v in p.items()}
    k = torch.empty(H.kernel_shape(w.shape, w.pad_mode), dtype=tdt, device=dev)
    stream = torch.cuda.current_stream(dev)
    synth = H.PreparedSynth(k, w.shape, d["omega0"], d["W1"], d["Wh"], d["Wout"], d["window"], d["gamma"],
                            d["beta"], d["bias"], "gaussian", w.pad_mode, stream)
    x1, x2, v, D = (to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.D))
    y = torch.empty_like(x1)
    ws_bytes = H.workspace_size(w.shape, w.pad_mode, w.dtype)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes else None
    conv = H.Prepared(y, x1, x2, v, k, D, w.pad_mode, ws, stream)

    def timed(fns, steps):
        settle_clocks(lambda i: [f() for f in fns], settle_count(alg_flops(w), alg_bytes(w), args.settle_ms))
        for _ in range(args.warmup):
            for f in fns:
                f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(steps):
            for f in fns:
                f()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / steps, (time.perf_counter() - t0) / steps

    synth_s, _ = timed([synth], args.steps)
    conv_s, _ = timed([conv], args.steps)
    both_s, both_wall = timed([synth, conv], args.steps)
    copy_calibration(args, dev)
    flops = synth_flops(w, SYNTH_HIDDEN, SYNTH_LAYERS)
    tflops = flops / synth_s / 1e12
    # fp32 kernels multiply on the fp32 matrix cores, bf16 kernels on the bf16
    # ones; the bound is whichever of products and the k write takes longer at
    # peak
    mpeak = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
    k_bytes = int(k.numel() * k.element_size())
    hbm_gbs = k_bytes / synth_s / 1e9
    if flops / (mpeak * 1e12) >= k_bytes / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(tflops, 3), "peak": mpeak, "unit": "TFLOP/s",
                "frac": round(tflops / mpeak, 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(hbm_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(hbm_gbs / HBM_PEAK_GBS, 4)}
    roof.update({"traffic": None, "kernel": "siren_synth", "alg_flops_per_call": flops,
                 "mfma_tflops": round(tflops, 3), "mfma_peak": mpeak, "k_bytes_written": k_bytes,
                 "avg_call_us": round(synth_s * 1e6, 3)})
    parity = None
    if not args.no_parity:
        import oracle
        f = {kk: (None if vv is None else vv.astype(np.float64)) for kk, vv in p.items()}
        kb = min(w.B, 2)  # the first samples' kernels, every channel and point
        ref = oracle.kernel_synth((kb,) + w.shape[1:], f["omega0"], f["W1"], f["Wh"], f["Wout"], f["window"],
                                  gamma=f["gamma"][:kb], beta=f["beta"][:kb], bias=f["bias"], pad_mode=w.pad_mode)
        got = k[:kb]
        got = (W.bf16_bits_to_f64(got.view(torch.int16).cpu().numpy().view(np.uint16)) if got.dtype == torch.bfloat16
               else got.cpu().numpy().astype(np.float64))
        parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    out = {
        "metric": "input-dependent kernel synthesis + gated N-D FFT conv GElem/s on 1 MI355X",
        "value": round(w.elems / both_wall / 1e9, 3), "unit": "GElem/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(both_wall * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded parameters drawn by the paper's initialisation recipe)",
        "synth_products": "bf16 matrix cores, fp32 accumulate" if w.dtype == "bf16" else "fp32 matrix cores",
        "config": {"workload": w.name, "pass": "synth+conv", "B": w.B, "C": w.C, "grid": list(w.grid),
                   "kernel_grid": list(w.kernel_shape[2:]), "pad_mode": w.pad_mode, "storage": w.dtype,
                   "hidden": SYNTH_HIDDEN, "layers": SYNTH_LAYERS, "film": True, "window": "gaussian"},
        "roofline": roof,
        "synth_us": round(synth_s * 1e6, 3), "conv_us": round(conv_s * 1e6, 3),
        "synth_then_conv_us": round(both_s * 1e6, 3),
        "cpu_baseline": None, "parity_rel_l2": parity, "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


MODAL_ORDER = 16


def bench_modal(args, w, inp):
    """Time hyenand_modal_filter (order-16 modal filters, one per channel, over
    the workload's 1D length) alone and followed by the one-kernel-per-channel
    convolution that consumes it; prints one JSON line."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    if len(w.grid) != 1 or w.pad_mode != W.LINEAR:
        raise SystemExit("--modal takes a 1D linear workload")
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    L = w.grid[0]
    p = W.modal_params(w.seed + 31, w.C, MODAL_ORDER, L)
    d = [torch.from_numpy(p[n]).to(dev) for n in ("log_mag", "angle", "res_re", "res_im")]
    k = torch.empty((w.C, L), dtype=tdt, device=dev)
    stream = torch.cuda.current_stream(dev)
    gen = H.PreparedModal(k, *d, stream=stream)
    x1, x2, v, D = (to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.D))
    y = torch.empty_like(x1)
    ws_bytes = H.workspace_size(w.shape, w.pad_mode, w.dtype)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes else None
    conv = H.Prepared(y, x1, x2, v, k, D, w.pad_mode, ws, stream, shared_k=True)

    def timed(fns):
        settle_clocks(lambda i: [f() for f in fns], settle_count(alg_flops(w), alg_bytes(w), args.settle_ms))
        for _ in range(args.warmup):
            for f in fns:
                f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            for f in fns:
                f()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / args.steps, (time.perf_counter() - t0) / args.steps

    y2 = torch.empty_like(x1)
    fused = H.PreparedModalConv(y2, x1, x2, v, *d, D, w.pad_mode, ws, stream)
    gen_s, _ = timed([gen])
    conv_s, _ = timed([conv])
    both_s, both_wall = timed([gen, conv])
    fused_s, fused_wall = timed([fused])
    copy_calibration(args, dev)
    # Per point and mode the sum takes Re(z w) = Re z Re w - Im z Im w and
    # accumulates it: two multiply-adds, 4 flops, run as a matrix-core
    # product for orders up to 32 (bf16 products for a bf16 kernel tensor,
    # fp32 otherwise).  The bound is the longer of that product at its
    # matrix peak and the k write at the HBM peak.
    flops = 4.0 * MODAL_ORDER * w.C * L
    tflops = flops / gen_s / 1e12
    k_bytes = k.numel() * k.element_size()
    mpeak = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
    t_mfma = flops / (mpeak * 1e12)
    t_write = k_bytes / (HBM_PEAK_GBS * 1e9)
    if t_mfma >= t_write:
        roof = {"bound": "mfma", "achieved": round(tflops, 3), "peak": mpeak, "unit": "TFLOP/s",
                "frac": round(tflops / mpeak, 4)}
    else:
        gbs = k_bytes / gen_s / 1e9
        roof = {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4)}
    parity = None
    if not args.no_parity:
        import oracle
        rows = [0, w.C // 2, w.C - 1]
        ref = oracle.modal_filter(*[p[n][rows].astype(np.float64) for n in ("log_mag", "angle", "res_re", "res_im")], L)
        got = k[rows]
        got = (W.bf16_bits_to_f64(got.view(torch.int16).cpu().numpy().view(np.uint16)) if got.dtype == torch.bfloat16
               else got.cpu().numpy().astype(np.float64))
        parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    fused_parity = None
    if not args.no_parity:
        # the fused call's output on three channels' lines against the
        # oracle's filter through the oracle's convolution
        import oracle
        rows = [0, w.C // 2, w.C - 1]
        kf = oracle.modal_filter(*[p[n][rows].astype(np.float64) for n in ("log_mag", "angle", "res_re", "res_im")], L)
        sub = [W.storage_to_f64(a[0, rows], w.dtype)[None] for a in (inp.x1, inp.x2, inp.v)]
        ref = oracle.conv_fft(sub[0], sub[1], sub[2], kf[None], W.storage_to_f64(inp.D, w.dtype)[rows],
                              w.pad_mode)[0]
        got = y2[0, rows]
        got = (W.bf16_bits_to_f64(got.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
               if got.dtype == torch.bfloat16 else got.cpu().numpy().astype(np.float64))
        fused_parity = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    out = {
        "metric": "modal filter generation + gated 1D FFT conv GElem/s on 1 MI355X",
        "value": round(w.elems / both_wall / 1e9, 3), "unit": "GElem/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(both_wall * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded poles and residues)",
        "config": {"workload": w.name, "pass": "modal+conv", "B": w.B, "C": w.C, "L": L, "order": MODAL_ORDER,
                   "storage": w.dtype},
        "roofline": dict(roof, traffic=None, kernel="modal_mfma_kernel", alg_flops_per_call=flops,
                         avg_call_us=round(gen_s * 1e6, 3), mfma_tflops=round(tflops, 3),
                         mfma_frac=round(tflops / mpeak, 4), k_bytes_written=k_bytes,
                         hbm_frac_of_k_write=round(k_bytes / gen_s / 1e9 / HBM_PEAK_GBS, 4)),
        "modal_us": round(gen_s * 1e6, 3), "conv_us": round(conv_s * 1e6, 3),
        "modal_then_conv_us": round(both_s * 1e6, 3),
        "fused_modal_conv_us": round(fused_s * 1e6, 3),
        "fused_modal_conv_gelems": round(w.elems / fused_wall / 1e9, 3),
        "fused_alg_bytes_per_call": 4 * w.elems * w.storage_bytes,
        "fused_hbm_frac": round(4 * w.elems * w.storage_bytes / fused_s / 1e9 / HBM_PEAK_GBS, 4),
        "cpu_baseline": None, "parity_rel_l2_sampled_channels": parity, "fused_parity_rel_l2_sampled_lines": fused_parity,
        "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


def bench_shared_k(args, w, inp):
    """One kernel per channel (hyenand_fftconv_shared_k, k[c] = the workload's
    kernel of sample 0) on a single-pass 2D workload: each channel's spectrum
    computed once and read by every image, against every image transforming
    k itself (the same call without a workspace); prints one JSON line."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    if len(w.grid) != 2 or H.plan_name(w.shape, w.pad_mode, w.dtype) != "fused2d":
        raise SystemExit("--shared-k takes a workload on the single-pass 2D plan")
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    x1, x2, v, D = (to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.D))
    kc = to_device(np.ascontiguousarray(inp.k[0]), w.dtype)
    y_hat, y_img = torch.empty_like(x1), torch.empty_like(x1)
    need = H.workspace_size(w.shape, w.pad_mode, w.dtype, shared_k=True)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    with_hat = H.Prepared(y_hat, x1, x2, v, kc, D, w.pad_mode, ws, stream, shared_k=True)
    per_image = H.Prepared(y_img, x1, x2, v, kc, D, w.pad_mode, None, stream, shared_k=True)

    def timed(fn):
        settle_clocks(lambda i: fn(), settle_count(alg_flops(w), alg_bytes(w), args.settle_ms))
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / args.steps, (time.perf_counter() - t0) / args.steps

    img_s, _ = timed(per_image)
    hat_s, hat_wall = timed(with_hat)
    # spectra kept across calls (a static kernel): the images' pass alone
    khat = H.kernel_spectrum(kc, w.shape, w.pad_mode, stream)
    y_kept = torch.empty_like(x1)
    nd, dims = H._dims(w.shape)
    kept_args = (H._ptr(x1), H._ptr(x2), H._ptr(v), H._ptr(khat), khat.numel(), H._ptr(D), H._ptr(y_kept), nd, dims,
                 H._mode(w.pad_mode), H._dtype_code(x1.dtype), ctypes.c_void_p(stream.cuda_stream))
    kept_fn = H.lib().hyenand_fftconv_spectrum
    kept_s, _ = timed(lambda: kept_fn(*kept_args))
    kept_diff = float((y_kept.float() - y_hat.float()).abs().max().item())
    diff = float((y_hat.float() - y_img.float()).abs().max().item())
    # the same images repeated along the batch: B x 4 (inputs for timing only)
    big = [t.repeat((4,) + (1,) * (t.dim() - 1)) for t in (x1, x2, v)]
    shape4 = tuple(big[0].shape)
    yb1, yb2 = torch.empty_like(big[0]), torch.empty_like(big[0])
    ws4 = torch.empty(H.workspace_size(shape4, w.pad_mode, w.dtype, shared_k=True), dtype=torch.uint8, device=dev)
    img4_s, _ = timed(H.Prepared(yb1, *big, kc, D, w.pad_mode, None, stream, shared_k=True))
    hat4_s, _ = timed(H.Prepared(yb2, *big, kc, D, w.pad_mode, ws4, stream, shared_k=True))
    del big, yb1, yb2, ws4
    parity = None
    if not args.no_parity:
        import oracle
        f = [W.storage_to_f64(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
        rng = np.random.default_rng(w.seed + 5)
        worst = 0.0
        got_all = y_hat
        for b, c in zip(rng.integers(0, w.B, 6), rng.integers(0, w.C, 6)):
            ref = oracle.conv_fft(f[0][b:b + 1, c:c + 1], f[1][b:b + 1, c:c + 1], f[2][b:b + 1, c:c + 1],
                                  f[3][0:1, c:c + 1], f[4][c:c + 1], w.pad_mode)[0, 0]
            got = got_all[b, c]
            got = (W.bf16_bits_to_f64(got.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
                   if got.dtype == torch.bfloat16 else got.cpu().numpy().astype(np.float64))
            worst = max(worst, float(np.linalg.norm(got - ref) / np.linalg.norm(ref)))
        parity = worst
    # x1, v, x2 read and y written per image, k read once per channel
    kpts = int(np.prod(w.grid))
    alg = (4 * w.elems + w.C * kpts) * w.storage_bytes
    gbs = alg / hat_s / 1e9
    out = {
        "metric": "gated 2D FFT conv, one kernel per channel, GElem/s on 1 MI355X",
        "value": round(w.elems / hat_wall / 1e9, 3), "unit": "GElem/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(hat_wall * 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded; k[c] = the workload's kernel of sample 0)",
        "config": {"workload": w.name, "pass": "forward, shared k", "B": w.B, "C": w.C, "grid": list(w.grid),
                   "pad_mode": w.pad_mode, "storage": w.dtype},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "alg_bytes_per_call": alg},
        "spectra_once_per_channel_us": round(hat_s * 1e6, 3),
        "per_image_transform_us": round(img_s * 1e6, 3),
        "speedup": round(img_s / hat_s, 3),
        "spectra_kept_across_calls_us": round(kept_s * 1e6, 3),
        "spectra_kept_speedup": round(img_s / kept_s, 3),
        "max_abs_diff_kept_vs_one_call": kept_diff,
        "batch_x4": {"B": 4 * w.B, "spectra_once_per_channel_us": round(hat4_s * 1e6, 3),
                     "per_image_transform_us": round(img4_s * 1e6, 3), "speedup": round(img4_s / hat4_s, 3)},
        "workspace_bytes": need,
        "max_abs_diff_between_paths": diff,
        "cpu_baseline": None, "parity_rel_l2_worst_sampled_line": parity,
        "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


def copy_calibration(args, dev):
    """One plain device copy of --copy-calibration-mb MiB, whose FETCH_SIZE and
    WRITE_SIZE counters scale the library's own to HBM bytes."""
    import torch
    if args.copy_calibration_mb > 0:
        src = torch.ones(args.copy_calibration_mb << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst


def to_device(arr, dtype):
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint16).view(np.int16)).cuda()
    return t.view(torch.bfloat16)


def kernel_source_hash() -> str:
    from paper_2607_19378_amd.build import source_hash
    return source_hash()


def stored_traffic(workload: str):
    """HBM bytes per call from FETCH_SIZE/WRITE_SIZE counters stored under
    profiles/, scaled by the same counters on a plain copy of known size;
    None when absent or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_call")


def settle_count(flops: float, set_bytes: float, ms: float) -> int:
    """Calls that keep the GPU busy for about `ms` milliseconds, from a rough
    per-call time (HBM at 5 TB/s or the fp32 VALU at half its peak, whichever
    is longer); a fixed count, so profiling runs know how many calls ran."""
    import math
    t = max(set_bytes / 5e12, flops / (0.5 * FP32_VALU_TFLOPS * 1e12), 1e-6)
    return int(min(2000, max(1, math.ceil(ms * 1e-3 / t)))) if ms > 0 else 0


def settle_clocks(step, n: int) -> None:
    """n untimed calls of the benchmarked step, then a synchronize."""
    import torch
    for i in range(n):
        step(i)
        if i % 16 == 15:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def bench_line_sweep(args):
    """Latency floor of a single-pass workload: the same call on 1 .. 4096
    (b, c) lines of the workload's shape (one workgroup per line), mean call
    time over args.steps calls under HIP events; prints one JSON line.  With
    fewer lines than CUs the call takes one line's latency."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    w0 = W.WORKLOADS[args.workload or "conv1d_4k"]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    rows = []
    for n in (1, 8, 64, 256, 512, 1024, 4096):
        inp = W.random_case(1, n, w0.grid, w0.pad_mode, w0.dtype, seed=w0.seed)
        t = [to_device(a, w0.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
        y = torch.empty_like(t[0])
        call = H.Prepared(y, *t, w0.pad_mode, None, stream)
        for _ in range(200):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        rows.append({"lines": n, "call_us": round(us, 2), "gelems": round(n * int(np.prod(w0.grid)) / us / 1e3, 2)})
        progress(f"line sweep {w0.name}: {n} lines {us:.2f} us")
    print(json.dumps({"metric": "call time against (b, c) lines", "workload": w0.name, "grid": list(w0.grid),
                      "plan": H.plan_name((1, 1) + tuple(w0.grid), w0.pad_mode, w0.dtype), "steps": args.steps,
                      "rows": rows, "kernel_source_hash": kernel_source_hash()}))


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(inp, budget_s: float):
    """The oracle (convolution theorem, fp64, own FFT) on a bounded sample of
    lines: chunks of lines cycling over all of them until budget_s has
    elapsed (at least one chunk), after one warm-up chunk."""
    import oracle
    w = inp.workload
    nthreads = oracle.default_threads()
    nl = w.B * w.C
    per_line = w.elems // nl
    chunk = min(nl, max(nthreads, nl // 8)) if per_line <= (1 << 16) else min(nl, nthreads)
    warm = list(range(min(nl, nthreads if per_line <= (1 << 16) else 1)))
    _oracle_on_lines(inp, warm, nthreads)
    done, nxt = 0, 0
    t0 = time.perf_counter()
    while done == 0 or time.perf_counter() - t0 < budget_s:
        lines = [(nxt + j) % nl for j in range(chunk)]
        _oracle_on_lines(inp, lines, nthreads)
        done += chunk
        nxt = (nxt + chunk) % nl
    dt = time.perf_counter() - t0
    sample = (f"{done} line evaluations cycling over the {nl} (b,c) lines of {w.name} ({done / nl:.2f} passes; "
              f"fp64 FFT oracle, {dt:.2f} s wall)")
    return {"value": round(done * per_line / dt / 1e9, 6), "unit": "GElem/s", "cores": nthreads,
            "cpu_model": cpu_model(), "kind": "oracle", "sample": sample, "seconds": round(dt, 3)}


def _oracle_on_lines(inp, lines, nthreads=None):
    """The oracle's y on the given flat (b * C + c) lines, each run as one
    channel of a one-sample problem (only those lines are upcast)."""
    import oracle
    w = inp.workload
    nl = w.B * w.C
    lines = np.asarray(lines, dtype=np.int64)
    sub = [W.storage_to_f64(a.reshape((nl,) + tuple(a.shape[2:]))[lines], w.dtype)[None]
           for a in (inp.x1, inp.x2, inp.v, inp.k)]
    Dsub = W.storage_to_f64(inp.D, w.dtype)[lines % w.C]
    return oracle.conv_fft(*sub, Dsub, w.pad_mode, nthreads=nthreads)[0]


def measure_stream_peak(dev, stream):
    """A 1 GiB device-to-device copy (read + write), best of 6: GB/s."""
    import torch
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    best = None
    for _ in range(6):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del src, dst
    return 2.0 * (1 << 28) * 4 / (best * 1e-3) / 1e9


def bench_forward(args, w, inp, cpu_budget, stream_gbs=None):
    """Time hyenand_fftconv on one workload: exactly args.steps calls after
    the settling calls and args.warmup warmup steps.  Returns the workload's
    entry: throughput from the wall clock over the timed steps, per-call
    times from HIP events on the launch stream (mean over the bracket; median
    and min of the per-step intervals), the HBM- and ALU-roofline fractions
    of the algorithmic work, the counter traffic when it was taken on these
    kernel sources, parity on sampled lines and the CPU oracle baseline."""
    import torch
    from paper_2607_19378_amd import hyenand as H
    set_bytes = alg_bytes(w)
    rot = args.rotate or max(1, min(8, int(np.ceil(2 * MALL_BYTES / set_bytes))))
    dev = torch.device("cuda:0")
    base = [to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
    sets = [base]
    for r in range(1, rot):
        # distinct buffers with the same values: the cache cannot serve one set from another
        sets.append([t.clone() for t in base])
    ys = [torch.empty_like(base[0]) for _ in range(rot)]
    ws_bytes = H.workspace_size(w.shape, w.pad_mode, w.dtype)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev) if ws_bytes else None
    plan = H.plan_name(w.shape, w.pad_mode, w.dtype)
    stream = torch.cuda.current_stream(dev)
    # one prepared call per input set: the timed loop only enqueues
    calls = [H.Prepared(ys[r], s[0], s[1], s[2], s[3], s[4], w.pad_mode, ws, stream) for r, s in enumerate(sets)]

    def step(i):
        calls[i % rot]()

    # The GPU sits idle while the host generates the inputs and comes back
    # at low clocks; a few milliseconds of the same calls, untimed, bring it
    # to its working clock before the warmup steps.
    n_settle = settle_count(alg_flops(w), alg_bytes(w), args.settle_ms)
    settle_clocks(step, n_settle)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # HIP events on the launch stream: one before every timed step and one
    # after the last.  Recording an event between launches leaves them
    # queued back to back.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        evs[i].record(stream)
        step(i)
    evs[-1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    avg_call_s = evs[0].elapsed_time(evs[-1]) * 1e-3 / args.steps
    flops = alg_flops(w)
    hbm_gbs = set_bytes / avg_call_s / 1e9
    alu_tflops = flops / avg_call_s / 1e12
    traffic = stored_traffic(w.name)
    entry = {
        "workload": w.name, "desc": w.description, "B": w.B, "C": w.C, "grid": list(w.grid),
        "pad_mode": w.pad_mode, "storage_dtype": w.dtype, "compute_dtype": "f32", "plan": plan,
        "value": round(w.elems / (ms_per_step * 1e-3) / 1e9, 3), "unit": "GElem/s",
        "ms_per_step": round(ms_per_step, 5),
        "call_us_mean": round(avg_call_s * 1e6, 3), "call_us_median": round(float(np.median(per_step)) * 1e3, 3),
        "call_us_min": round(float(per_step.min()) * 1e3, 3),
        "alg_bytes_per_call": set_bytes, "alg_flops_per_call": round(flops),
        "hbm_achieved_gbs": round(hbm_gbs, 2), "hbm_frac": round(hbm_gbs / HBM_PEAK_GBS, 4),
        "hbm_frac_wall": round(set_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "alu_achieved_tflops": round(alu_tflops, 3), "alu_frac": round(alu_tflops / FP32_VALU_TFLOPS, 4),
        "alu_frac_of_packed_peak": round(alu_tflops / FP32_PACKED_TFLOPS, 4),
        "first_bound": ("alu" if flops / (FP32_VALU_TFLOPS * 1e12) > set_bytes / (HBM_PEAK_GBS * 1e9) else "hbm"),
        "counter_bytes_per_call": traffic,
        "counter_to_alg_bytes": None if traffic is None else round(traffic / set_bytes, 3),
        "rotated_input_sets": rot, "untimed_calls": {"settle": n_settle, "warmup": args.warmup},
    }
    if stream_gbs:
        entry["hbm_frac_of_stream_peak"] = round(hbm_gbs / stream_gbs, 4)
    prof = os.path.join("profiles", f"{plan}_{w.name}.md")
    if os.path.exists(os.path.join(ROOT, prof)):
        entry["profile"] = prof  # rocprofv3 kernel trace and counter summary of this workload

    copy_calibration(args, dev)

    if not args.no_parity:
        # the last output against the oracle on sampled (b, c) lines; every
        # element of every workload is compared in the GPU tests
        nl = w.B * w.C
        chk = np.array(sorted(set([0, nl // 2, nl - 1])), dtype=np.int64)
        ref = _oracle_on_lines(inp, chk).reshape(len(chk), -1)
        yv = ys[(args.steps - 1) % rot].reshape(nl, -1)[torch.as_tensor(chk, device=dev)]
        if yv.dtype == torch.bfloat16:
            got = W.bf16_bits_to_f64(yv.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
        else:
            got = yv.cpu().numpy().astype(np.float64)
        entry["parity_rel_l2_sampled_lines"] = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        entry["parity_lines"] = chk.tolist()
    del calls, sets, base, ys, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    entry["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(inp, cpu_budget)
    return entry


def headline_roofline(e):
    """The roofline object of the JSON line: the HBM roofline of the metric,
    algorithmic bytes of one call over the mean call time under HIP events;
    the ALU fraction beside it."""
    r = {"bound": "hbm", "achieved": e["hbm_achieved_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": e["hbm_frac"], "traffic": e["counter_bytes_per_call"],
         "kernel_plan": e["plan"], "alg_bytes_per_call": e["alg_bytes_per_call"],
         "avg_call_us": e["call_us_mean"], "median_call_us": e["call_us_median"], "min_call_us": e["call_us_min"],
         "alu_achieved_tflops": e["alu_achieved_tflops"], "alu_peak_tflops": FP32_VALU_TFLOPS,
         "alu_frac": e["alu_frac"], "alu_frac_of_packed_peak": e["alu_frac_of_packed_peak"],
         "alg_flops_per_call": e["alg_flops_per_call"], "first_bound": e["first_bound"],
         "counter_to_alg_bytes": e["counter_to_alg_bytes"]}
    for k in ("profile", "hbm_frac_of_stream_peak"):
        if k in e:
            r[k] = e[k]
    return r


def progress(msg: str) -> None:
    sys.stderr.write(f"[bench] {msg}\n")
    sys.stderr.flush()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-ms", type=float, default=30.0,
                    help="untimed calls worth about this long before the warmup steps, to leave the GPU's idle "
                         "clocks (0: none)")
    ap.add_argument("--workload", default=None, choices=list(W.WORKLOADS),
                    help="time this workload only (default: the headline conv2d_64 plus every configuration)")
    ap.add_argument("--rotate", type=int, default=0, help="input sets to rotate (0: enough to exceed 2x the MALL)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the headline's cpu_baseline")
    ap.add_argument("--cpu-budget-other", type=float, default=5.0,
                    help="seconds of oracle work for each other configuration's cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true", help="skip the sampled oracle check (profiling runs)")
    ap.add_argument("--no-stream-peak", action="store_true", help="skip the 1 GiB copy that measures the stream peak")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward (gradients for x1, x2, v, k, D) instead of the forward")
    ap.add_argument("--operator", action="store_true",
                    help="time the whole HyenaND operator (norms and activations around the convolution)")
    ap.add_argument("--synth", action="store_true",
                    help="time kernel synthesis (FiLM-modulated SIREN + window) alone and followed by the conv")
    ap.add_argument("--modal", action="store_true",
                    help="time modal filter generation (order 16, one filter per channel) alone and with the conv")
    ap.add_argument("--shared-k", action="store_true",
                    help="one kernel per channel on a single-pass 2D workload: spectra once per channel "
                         "against per-image transforms")
    ap.add_argument("--line-sweep", action="store_true",
                    help="time the workload's single-pass call on 1 .. 4096 lines (latency floor)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the timed steps, run one plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the operator shards by "
              f"independent (b, c) lines; this benchmark runs on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.line_sweep:
        bench_line_sweep(args)
        return
    if args.backward or args.operator or args.synth or args.modal or args.shared_k:
        w = W.WORKLOADS[args.workload or DEFAULT_WORKLOAD]
        inp = W.generate(w)
        if args.shared_k:
            bench_shared_k(args, w, inp)
        elif args.backward:
            bench_backward(args, w, inp)
        elif args.operator:
            bench_operator(args, w, inp)
        elif args.synth:
            bench_synth(args, w, inp)
        else:
            bench_modal(args, w, inp)
        return

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    stream_gbs = None if args.no_stream_peak else measure_stream_peak(dev, stream)
    head_name = args.workload or DEFAULT_WORKLOAD
    names = [head_name] if args.workload else [head_name] + [n for n in CONFIG_ORDER if n != head_name]
    extra = [] if args.workload else [n for n in EXTRA_ORDER if n not in names]
    entries = {}
    for n in names + extra:
        w = W.WORKLOADS[n]
        progress(f"{n}: generating inputs {w.shape} {w.pad_mode} {w.dtype}")
        inp = W.generate(w)
        progress(f"{n}: timing {args.steps} steps")
        entries[n] = bench_forward(args, w, inp, args.cpu_budget if n == head_name else args.cpu_budget_other,
                                   stream_gbs)
        e = entries[n]
        progress(f"{n}: {e['value']} GElem/s, {e['call_us_mean']} us per call, hbm_frac {e['hbm_frac']}")
        del inp
    h = entries[head_name]
    w = W.WORKLOADS[head_name]
    out = {
        "metric": "gated N-D FFT-conv GElem/s and % of HBM roofline on 1 MI355X",
        "value": h["value"], "unit": "GElem/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": h["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "storage_dtype": w.dtype,
        "data": "synthetic (seeded, shapes and distributions of the paper's workloads)",
        "config": {"workload": w.name, "desc": w.description, "B": w.B, "C": w.C, "grid": list(w.grid),
                   "pad_mode": w.pad_mode, "storage": w.dtype, "plan": h["plan"],
                   "rotated_input_sets": h["rotated_input_sets"]},
        "roofline": headline_roofline(h),
        "cpu_baseline": h["cpu_baseline"],
        "parity_rel_l2_sampled": h.get("parity_rel_l2_sampled_lines"),
        "untimed_calls": h["untimed_calls"],
        "stream_peak_gbs": None if stream_gbs is None else round(stream_gbs, 1),
        "per_config": [entries[n] for n in names],
        "extra_workloads": [entries[n] for n in extra],
        "kernel_source_hash": kernel_source_hash(),
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
