"""Turn rocprofv3 runs of bench.py into the text summaries kept under profiles/.

    python -m paper_2607_19378_amd.profile_summary --workload W --calls N \\
        --trace DIR --fetch DIR --write DIR --copy-mib M \\
        --cmd-trace "..." --cmd-fetch "..." --cmd-write "..."

The three directories hold the CSV output of three rocprofv3 runs of one
bench.py command: ``--kernel-trace --stats``, ``--pmc FETCH_SIZE`` and
``--pmc WRITE_SIZE``.  With ``--synth`` the runs are of ``bench.py --synth``
and the summary, ``profiles/siren_synth_<workload>.md``, covers the kernel
synthesis kernel; with ``--modal`` they are of ``bench.py --modal`` and
``profiles/modal_filter_<workload>.md`` covers the modal filter kernel.  N is the number of hyenand_fftconv calls the command
made (bench.py: warmup + steps).  Writes

* ``profiles/<plan>_<workload>.md``: per-kernel average durations, HBM bytes
  per call against the algorithmic minimum, and the commands;
* ``profiles/traffic_<workload>.json``: HBM bytes per call, which bench.py
  reports as ``roofline.traffic`` while the kernel sources are unchanged.

FETCH_SIZE and WRITE_SIZE count KiB per dispatch.  Each is scaled by
known bytes / counter value of the plain device-to-device copy
(``__amd_rocclr_copyBuffer`` of M MiB) that ``bench.py --copy-calibration-mb M``
runs after its timed steps, so the figures are HBM bytes.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json

import numpy as np
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def _rows(d: str, suffix: str):
    files = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    out = []
    for f in files:
        with open(f) as fh:
            out += list(csv.DictReader(fh))
    return out


def short_name(full: str) -> str:
    """'void hyenand::(anonymous namespace)::mp_core<512, true>(...)' -> 'mp_core<512, true>'."""
    n = full.strip('"')
    if n.startswith("void "):
        n = n[5:]
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and not n[i:].startswith("(anonymous"):
            cut = i
            break
    n = n[:cut]
    return n.split("::")[-1]


def counter_per_call(rows, counter: str, calls: int):
    """Sum of the counter over hyenand dispatches / calls, and the copy's value."""
    op = 0.0
    copy = 0.0
    per_kernel = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        v = float(r["Counter_Value"])
        name = r["Kernel_Name"]
        if "hyenand" in name:
            op += v
            k = short_name(name)
            per_kernel[k] = per_kernel.get(k, 0.0) + v
        elif COPY_KERNEL in name:
            copy = max(copy, v)
    return op / calls, copy, {k: v / calls for k, v in per_kernel.items()}


SQ_COUNTERS = ("SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_ACTIVE_INST_VALU", "SQ_BUSY_CYCLES",
               "SQ_WAVES", "SQ_LDS_IDX_ACTIVE", "SQ_WAIT_INST_LDS", "GRBM_GUI_ACTIVE")
DRAM_COUNTERS = ("TCC_EA0_RDREQ_DRAM_32B_sum", "TCC_EA0_WRREQ_WRITE_DRAM_32B_sum", "TCC_EA0_RDREQ_sum",
                 "TCC_EA0_WRREQ_sum")


def timed_counters(rows, counters, calls: int, steps: int):
    """Per-call sums of each counter over the library's dispatches of the
    last `steps` calls (the timed steps), and per kernel.  The library's
    dispatches are taken in Dispatch_Id order; a call is the same number of
    them throughout the command."""
    lib = sorted({int(r["Dispatch_Id"]) for r in rows if "hyenand" in r["Kernel_Name"]})
    per_call = len(lib) // calls
    keep = set(lib[-per_call * steps:])
    tot = {c: 0.0 for c in counters}
    per_kernel = {}
    for r in rows:
        c = r["Counter_Name"]
        if c not in tot or int(r["Dispatch_Id"]) not in keep:
            continue
        v = float(r["Counter_Value"])
        tot[c] += v
        k = short_name(r["Kernel_Name"])
        per_kernel.setdefault(k, {}).setdefault(c, 0.0)
        per_kernel[k][c] += v
    return ({c: v / steps for c, v in tot.items()},
            {k: {c: v / steps for c, v in d.items()} for k, d in per_kernel.items()}, per_call)


def synth_summary(a, W, source_hash):
    """profiles/siren_synth_<workload>.md from rocprofv3 runs of
    ``bench.py --synth``: the synthesis kernel's duration, HBM bytes and
    matrix-core rate, beside the convolution kernels of the same run."""
    sys.path.insert(0, ROOT)
    import bench
    w = W.WORKLOADS[a.workload]
    stats = [r for r in _rows(a.trace, "_kernel_stats.csv") if "hyenand" in r["Name"]]
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    syn = [r for r in stats if "siren_synth" in r["Name"]]
    if not syn:
        raise SystemExit("no siren_synth dispatches in the trace")
    avg_ns = float(syn[0]["AverageNs"])
    flops = bench.synth_flops(w, bench.SYNTH_HIDDEN, bench.SYNTH_LAYERS)
    tf = flops / (avg_ns * 1e-9) / 1e12
    npos = int(np.prod(w.kernel_shape[2:]))
    k_bytes = w.B * w.C * npos * w.storage_bytes

    def per_dispatch(rows, counter):
        tot, n, copy = 0.0, set(), 0.0
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            if "siren_synth" in r["Kernel_Name"]:
                tot += float(r["Counter_Value"])
                n.add(r["Dispatch_Id"])
            elif COPY_KERNEL in r["Kernel_Name"]:
                copy = max(copy, float(r["Counter_Value"]))
        return tot / max(1, len(n)), copy

    f_d, f_copy = per_dispatch(_rows(a.fetch, "_counter_collection.csv"), "FETCH_SIZE")
    w_d, w_copy = per_dispatch(_rows(a.write, "_counter_collection.csv"), "WRITE_SIZE")
    if f_copy <= 0 or w_copy <= 0:
        raise SystemExit("copy calibration dispatch not found in the counter runs")
    copy_kib = a.copy_mib * 1024.0
    fb = f_d * 1024.0 * copy_kib / f_copy
    wb = w_d * 1024.0 * copy_kib / w_copy
    lines = [f"# siren_synth on {w.name}", "",
             f"Kernel synthesis (FiLM-modulated SIREN, Hf = {bench.SYNTH_HIDDEN}, J = {bench.SYNTH_LAYERS}, "
             f"Gaussian window) on the kernel grid of {w.description}: {w.B} x {w.C} x {npos} points.  "
             f"Kernel source hash `{source_hash()}`.", "",
             "Commands (run from /tmp with TMPDIR=/tmp on the MI355X box):", "",
             "```", a.cmd_trace, a.cmd_fetch, a.cmd_write, "```", "",
             "## Kernel durations (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | dispatches | avg us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for r in stats:
        lines.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    mpeak, mkind = ((bench.MFMA_BF16_PEAK_TFLOPS, "bf16") if w.dtype == "bf16"
                    else (bench.MFMA_F32_PEAK_TFLOPS, "fp32"))
    lines += ["", f"siren_synth: {flops / 1e9:.3f} GFLOP of matrix-core multiply-adds per call in "
                  f"{avg_ns / 1e3:.2f} us = {tf:.1f} TFLOP/s, {100 * tf / mpeak:.1f}% of the "
                  f"{mpeak} TFLOP/s {mkind} matrix peak; the k write alone takes {k_bytes / 8e12 * 1e6:.1f} us "
                  f"at 8 TB/s ({100 * k_bytes / (avg_ns * 1e-9) / 8e12:.1f}% of it achieved).", "",
              "## HBM traffic per siren_synth dispatch (rocprofv3 --pmc)", "",
              f"Copy calibration: {a.copy_mib} MiB device copy read {f_copy:.1f} KiB (FETCH_SIZE) and wrote "
              f"{w_copy:.1f} KiB (WRITE_SIZE).", "",
              f"Read {fb / 1e6:.2f} MB (the weights, by every workgroup, mostly from the caches), write "
              f"{wb / 1e6:.2f} MB; the kernel tensor is {k_bytes / 1e6:.2f} MB (written once).", ""]
    md = os.path.join(a.out, f"siren_synth_{w.name}.md")
    with open(md, "w") as fh:
        fh.write("\n".join(lines))
    print(md)


def modal_summary(a, W, source_hash):
    """profiles/modal_filter_<workload>.md from rocprofv3 runs of
    ``bench.py --modal``: the modal filter kernel's duration, HBM bytes and
    matrix-core rate, beside the convolution kernels of the same run."""
    sys.path.insert(0, ROOT)
    import bench
    w = W.WORKLOADS[a.workload]
    stats = [r for r in _rows(a.trace, "_kernel_stats.csv") if "hyenand" in r["Name"]]
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    gen = [r for r in stats if "modal_" in r["Name"]]
    if not gen:
        raise SystemExit("no modal filter dispatches in the trace")
    avg_ns = float(gen[0]["AverageNs"])
    L = w.grid[0]
    flops = 4.0 * bench.MODAL_ORDER * w.C * L
    tf = flops / (avg_ns * 1e-9) / 1e12
    k_bytes = w.C * L * w.storage_bytes

    def per_dispatch(rows, counter):
        tot, n, copy = 0.0, set(), 0.0
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            if "modal_" in r["Kernel_Name"]:
                tot += float(r["Counter_Value"])
                n.add(r["Dispatch_Id"])
            elif COPY_KERNEL in r["Kernel_Name"]:
                copy = max(copy, float(r["Counter_Value"]))
        return tot / max(1, len(n)), copy

    f_d, f_copy = per_dispatch(_rows(a.fetch, "_counter_collection.csv"), "FETCH_SIZE")
    w_d, w_copy = per_dispatch(_rows(a.write, "_counter_collection.csv"), "WRITE_SIZE")
    if f_copy <= 0 or w_copy <= 0:
        raise SystemExit("copy calibration dispatch not found in the counter runs")
    copy_kib = a.copy_mib * 1024.0
    fb = f_d * 1024.0 * copy_kib / f_copy
    wb = w_d * 1024.0 * copy_kib / w_copy
    lines = [f"# modal filter on {w.name}", "",
             f"Modal filter generation, order {bench.MODAL_ORDER}, one filter per channel over the length of "
             f"{w.description}: {w.C} x {L} points.  Kernel source hash `{source_hash()}`.", "",
             "Commands (run from /tmp with TMPDIR=/tmp on the MI355X box):", "",
             "```", a.cmd_trace, a.cmd_fetch, a.cmd_write, "```", "",
             "## Kernel durations (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | dispatches | avg us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for r in stats:
        lines.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    mpeak, mkind = ((bench.MFMA_BF16_PEAK_TFLOPS, "bf16") if w.dtype == "bf16"
                    else (bench.MFMA_F32_PEAK_TFLOPS, "fp32"))
    lines += ["", f"{short_name(gen[0]['Name'])}: {flops / 1e9:.3f} GFLOP (4 per mode and point) per call in "
                  f"{avg_ns / 1e3:.2f} us = {tf:.1f} TFLOP/s, {100 * tf / mpeak:.1f}% of the "
                  f"{mpeak} TFLOP/s {mkind} matrix peak; the k write alone takes "
                  f"{k_bytes / 8e12 * 1e6:.1f} us at 8 TB/s ({100 * k_bytes / (avg_ns * 1e-9) / 8e12:.1f}% of it "
                  "achieved).", "",
              "## HBM traffic per modal filter dispatch (rocprofv3 --pmc)", "",
              f"Copy calibration: {a.copy_mib} MiB device copy read {f_copy:.1f} KiB (FETCH_SIZE) and wrote "
              f"{w_copy:.1f} KiB (WRITE_SIZE).", "",
              f"Read {fb / 1e6:.2f} MB (poles and residues), write {wb / 1e6:.2f} MB; the kernel tensor is "
              f"{k_bytes / 1e6:.2f} MB (written once).", ""]
    md = os.path.join(a.out, f"modal_filter_{w.name}.md")
    with open(md, "w") as fh:
        fh.write("\n".join(lines))
    print(md)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--calls", type=int, required=True)
    ap.add_argument("--steps", type=int, default=10, help="timed steps of the bench.py command (the last calls)")
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--cmd-trace", required=True)
    ap.add_argument("--cmd-fetch", required=True)
    ap.add_argument("--cmd-write", required=True)
    ap.add_argument("--sq", default=None, help="counter run of SQ_* (and GRBM_GUI_ACTIVE) on the same command")
    ap.add_argument("--dram", default=None, help="counter run of TCC_EA0_*DRAM* requests on the same command")
    ap.add_argument("--cmd-sq", default="")
    ap.add_argument("--cmd-dram", default="")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    ap.add_argument("--synth", action="store_true", help="runs of bench.py --synth: summarise the synthesis kernel")
    ap.add_argument("--modal", action="store_true", help="runs of bench.py --modal: summarise the modal filter kernel")
    a = ap.parse_args(argv)

    sys.path.insert(0, ROOT)
    from paper_2607_19378_amd import workloads as W
    from paper_2607_19378_amd.build import source_hash
    from paper_2607_19378_amd import hyenand as H
    if a.synth:
        synth_summary(a, W, source_hash)
        return
    if a.modal:
        modal_summary(a, W, source_hash)
        return

    w = W.WORKLOADS[a.workload]
    plan = H.plan_name(w.shape, w.pad_mode, w.dtype)
    alg = (4 * w.elems + int(np.prod(w.kernel_shape))) * w.storage_bytes  # x1, v, x2, k in; y out

    stats = [r for r in _rows(a.trace, "_kernel_stats.csv") if "hyenand" in r["Name"]]
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    total_ns = sum(float(r["TotalDurationNs"]) for r in stats)
    # GPU busy time: the union of the library's kernel intervals (the
    # multi-pass plans run chunks on concurrent streams, so durations overlap)
    iv = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
                for r in _rows(a.trace, "_kernel_trace.csv") if "hyenand" in r["Kernel_Name"])
    busy_ns, cur_s, cur_e = 0, None, None
    for s0, e0 in iv:
        if cur_e is None or s0 > cur_e:
            if cur_e is not None:
                busy_ns += cur_e - cur_s
            cur_s, cur_e = s0, e0
        else:
            cur_e = max(cur_e, e0)
    if cur_e is not None:
        busy_ns += cur_e - cur_s

    f_call, f_copy, f_k = counter_per_call(_rows(a.fetch, "_counter_collection.csv"), "FETCH_SIZE", a.calls)
    w_call, w_copy, w_k = counter_per_call(_rows(a.write, "_counter_collection.csv"), "WRITE_SIZE", a.calls)
    copy_kib = a.copy_mib * 1024.0
    if f_copy <= 0 or w_copy <= 0:
        raise SystemExit("copy calibration dispatch not found in the counter runs")
    f_scale = copy_kib / f_copy
    w_scale = copy_kib / w_copy
    fetch_b = f_call * 1024.0 * f_scale
    write_b = w_call * 1024.0 * w_scale
    h = source_hash()

    lines = [f"# {plan} on {w.name}", "",
             f"{w.description}.  Plan `{plan}`; kernel source hash `{h}`.", "",
             "Commands (run from /tmp with TMPDIR=/tmp on the MI355X box; bench.py made "
             f"{a.calls} hyenand_fftconv calls in each, the last {a.steps} timed):", "",
             "```", a.cmd_trace, a.cmd_fetch, a.cmd_write, "```", "",
             "## Kernel durations (rocprofv3 --kernel-trace --stats)", "",
             "| kernel | dispatches | avg us | min us | max us | share of op time |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in stats:
        lines.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{100.0 * float(r['TotalDurationNs']) / total_ns:.1f}% |")
    busy = busy_ns / a.calls
    # the timed steps alone: the dispatches of the last a.steps calls, whose
    # union per call is what bench.py's HIP events see (the earlier calls
    # include the untimed settling calls, some at idle clocks)
    tail = iv[-max(1, round(len(iv) * a.steps / a.calls)):]
    tail_ns, cs, ce = 0, None, None
    for s0, e0 in tail:
        if ce is None or s0 > ce:
            if ce is not None:
                tail_ns += ce - cs
            cs, ce = s0, e0
        else:
            ce = max(ce, e0)
    if ce is not None:
        tail_ns += ce - cs
    tail_busy = tail_ns / a.steps
    lines += ["", f"GPU busy time per call over the last {a.steps} calls (the timed steps): "
                  f"{tail_busy / 1e3:.2f} us ({alg / tail_busy:.1f} GB/s of algorithmic bytes, "
                  f"{100.0 * alg / tail_busy / 8000.0:.2f}% of 8 TB/s).", ""]
    # per-kernel averages over the timed steps alone
    tr = sorted(((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), short_name(r["Kernel_Name"]))
                 for r in _rows(a.trace, "_kernel_trace.csv") if "hyenand" in r["Kernel_Name"]))
    tr = tr[-max(1, round(len(tr) * a.steps / a.calls)):]
    agg = {}
    for s0, e0, k in tr:
        d = agg.setdefault(k, [])
        d.append(e0 - s0)
    lines += [f"Per-kernel durations over the timed steps only ({a.steps} calls):", "",
              "| kernel | dispatches | avg us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for k, d in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"| `{k}` | {len(d)} | {np.mean(d) / 1e3:.2f} | {np.min(d) / 1e3:.2f} | {np.max(d) / 1e3:.2f} |")
    lines.append("")
    lines += [f"GPU busy time per call over all calls (union of the kernels' intervals): {busy / 1e3:.2f} us "
                  f"({alg / busy:.1f} GB/s of algorithmic bytes, {100.0 * alg / busy / 8000.0:.2f}% of 8 TB/s).  "
                  f"Sum of kernel durations per call: {total_ns / a.calls / 1e3:.2f} us"
                  + (" (kernels of chunks on different side streams overlap, and each one's duration includes "
                     "the time it shares the GPU)." if total_ns > 1.02 * busy_ns else "."), "",
              "## HBM traffic per call (rocprofv3 --pmc)", "",
              f"Copy calibration: {a.copy_mib} MiB device copy read {f_copy:.1f} KiB (FETCH_SIZE) and wrote "
              f"{w_copy:.1f} KiB (WRITE_SIZE); scale factors {f_scale:.4f} and {w_scale:.4f}.", "",
              "| kernel | FETCH MB/call | WRITE MB/call |", "|---|---:|---:|"]
    for k in sorted(set(f_k) | set(w_k)):
        lines.append(f"| `{k}` | {f_k.get(k, 0.0) * 1024.0 * f_scale / 1e6:.2f} | {w_k.get(k, 0.0) * 1024.0 * w_scale / 1e6:.2f} |")
    lines += ["",
              f"Total: read {fetch_b / 1e6:.2f} MB + write {write_b / 1e6:.2f} MB = {(fetch_b + write_b) / 1e6:.2f} MB "
              f"per call; algorithmic minimum {alg / 1e6:.2f} MB (x1, x2, v, k read and y written once); "
              f"ratio {(fetch_b + write_b) / alg:.3f}.", ""]
    cmds = [a.cmd_trace, a.cmd_fetch, a.cmd_write]
    sq_rec = None
    if a.sq:
        cmds.append(a.cmd_sq)
        tot, per_k, per_call = timed_counters(_rows(a.sq, "_counter_collection.csv"), SQ_COUNTERS, a.calls,
                                              a.steps)
        sq_rec = tot
        lines += ["## Instruction and LDS counters per call, timed steps only (rocprofv3 --pmc)", "",
                  "`" + a.cmd_sq + "`", "",
                  f"{per_call} library dispatches per call.  SQ_INSTS_* count wave instructions; "
                  "SQ_ACTIVE_INST_VALU and SQ_WAIT_INST_LDS are in quad-cycles summed over waves; "
                  "SQ_LDS_BANK_CONFLICT and SQ_LDS_IDX_ACTIVE are cycles summed over CUs; SQ_BUSY_CYCLES "
                  "sums the shader engines' busy cycles; GRBM_GUI_ACTIVE is the GPU's busy clock count "
                  "(counter runs serialise the dispatches).", "",
                  "| kernel | " + " | ".join(SQ_COUNTERS) + " |", "|---|" + "---:|" * len(SQ_COUNTERS)]
        for k, d in sorted(per_k.items()):
            lines.append(f"| `{k}` | " + " | ".join(f"{d.get(c, 0.0):.4g}" for c in SQ_COUNTERS) + " |")
        lines.append("| **per call** | " + " | ".join(f"{tot[c]:.4g}" for c in SQ_COUNTERS) + " |")
        valu_floor_us = tot["SQ_INSTS_VALU"] * 4 / (256 * 4) / 2.4e3
        lines += ["", f"VALU issue floor: {tot['SQ_INSTS_VALU'] / 1e6:.2f} M wave instructions x 4 cycles over "
                      f"1024 SIMDs = {valu_floor_us:.1f} us at 2.4 GHz.  LDS bank-conflict cycles are "
                      f"{100.0 * tot['SQ_LDS_BANK_CONFLICT'] / max(1.0, tot['SQ_LDS_IDX_ACTIVE']):.2f}% of the "
                      "LDS-active cycles.", ""]
    dram_rec = None
    if a.dram:
        cmds.append(a.cmd_dram)
        tot, per_k, _ = timed_counters(_rows(a.dram, "_counter_collection.csv"), DRAM_COUNTERS, a.calls, a.steps)
        rd = 32.0 * tot["TCC_EA0_RDREQ_DRAM_32B_sum"]
        wr = 32.0 * tot["TCC_EA0_WRREQ_WRITE_DRAM_32B_sum"]
        dram_rec = {"read_bytes_per_call": round(rd), "write_bytes_per_call": round(wr)}
        lines += ["## Requests from the L2 to the memory controller per call, timed steps only", "",
                  "`" + a.cmd_dram + "`", "",
                  f"Read {rd / 1e6:.2f} MB and write {wr / 1e6:.2f} MB in 32-byte units "
                  f"(TCC_EA0_RDREQ_DRAM_32B, TCC_EA0_WRREQ_WRITE_DRAM_32B); {tot['TCC_EA0_RDREQ_sum']:.4g} read "
                  f"and {tot['TCC_EA0_WRREQ_sum']:.4g} write requests in all.  These requests go to the "
                  "memory controller's side of the data fabric, where the 256 MiB Infinity Cache sits, so they "
                  "too count Infinity-Cache hits as well as HBM accesses; no counter exposed to rocprofv3 on "
                  "gfx950 separates the two.", ""]
    os.makedirs(a.out, exist_ok=True)
    md = os.path.join(a.out, f"{plan}_{w.name}.md")
    with open(md, "w") as fh:
        fh.write("\n".join(lines))
    rec = {"workload": w.name, "plan": plan, "source_hash": h, "bytes_per_call": round(fetch_b + write_b),
           "fetch_bytes_per_call": round(fetch_b), "write_bytes_per_call": round(write_b),
           "alg_bytes_per_call": alg, "fetch_scale": round(f_scale, 5), "write_scale": round(w_scale, 5),
           "calls": a.calls, "steps": a.steps, "commands": cmds, "sq_per_call": sq_rec, "dram_per_call": dram_rec}
    with open(os.path.join(a.out, f"traffic_{w.name}.json"), "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(md)


if __name__ == "__main__":
    main()
