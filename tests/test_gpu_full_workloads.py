"""Every output element of the five benchmark workloads against the fp64
oracle, on the GPU in the launch configuration the benchmark times (the
recommended workspace, the caller's stream): the relative L2 over the whole
tensor and the worst relative L2 of a (b, c) line, forward on all five and
every gradient of the backward on the three multi-pass workloads (all lines
and all channels).  The oracle runs over chunks of lines, so host memory
stays bounded."""
import numpy as np
import pytest

import oracle
from paper_2607_19378_amd import workloads as W

from gpu_util import TOL, from_device, log, oracle_lines, run_gpu, summary, to_device

pytestmark = pytest.mark.gpu

FORWARD = ["conv1d_4k", "conv2d_64", "conv2d_512c", "conv3d_128", "conv1d_1m", "conv2d_14_patches"]
BACKWARD = ["conv2d_512c", "conv3d_128", "conv1d_1m"]
NAMES = ("gx1", "gx2", "gv", "gk", "gD")


def _chunk_budget():
    """fp64 bytes one oracle chunk may hold: a quarter of the host's memory,
    at most 24 GiB."""
    import os
    try:
        phys = os.sysconf("SC_PHYS_PAGES") * os.sysconf("SC_PAGE_SIZE")
    except (ValueError, OSError, AttributeError):
        phys = 16 << 30
    return int(min(24 << 30, phys // 4))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_19378_amd import hyenand as H
    H.lib()


def _oracle_line_bytes(w):
    """fp64 bytes the oracle holds per line: the padded complex grids of u
    and k (16 bytes a point) and the five tensors of the line."""
    P = [x if w.pad_mode == "circular" else 2 * x for x in w.grid]
    return 32 * int(np.prod(P)) + 48 * int(np.prod(w.grid))


def _chunk_lines(w, unit_lines=1):
    nt = oracle.default_threads()
    n = max(1, _chunk_budget() // (_oracle_line_bytes(w) * unit_lines))
    if n >= nt:
        n -= n % nt
    return int(n)


class Acc:
    """Sums of squared differences and squared references, per tensor and
    per line, accumulated in fp64 over chunks."""

    def __init__(self):
        self.num = 0.0
        self.den = 0.0
        self.worst = 0.0

    def add(self, got, ref, per_line=True):
        got = np.asarray(got, np.float64).reshape(ref.shape[0], -1)
        ref = np.asarray(ref, np.float64).reshape(ref.shape[0], -1)
        d2 = np.sum((got - ref) ** 2, axis=1)
        r2 = np.sum(ref ** 2, axis=1)
        self.num += float(d2.sum())
        self.den += float(r2.sum())
        if per_line:
            self.worst = max(self.worst, float(np.max(np.sqrt(d2) / np.maximum(np.sqrt(r2), 1e-300))))

    @property
    def rel(self):
        return float(np.sqrt(self.num / max(self.den, 1e-300)))


@pytest.mark.parametrize("name", FORWARD)
def test_forward_every_element(name):
    w = W.WORKLOADS[name]
    log(f"[whole fwd] {name}: generating {w.shape} {w.pad_mode} {w.dtype}")
    inp = W.generate(w)
    y = run_gpu(inp)
    nl = w.B * w.C
    y = y.reshape(nl, -1)
    assert np.all(np.isfinite(y))
    chunk = _chunk_lines(w)
    acc = Acc()
    for l0 in range(0, nl, chunk):
        lines = np.arange(l0, min(nl, l0 + chunk), dtype=np.int64)
        ref = oracle_lines(inp, lines).reshape(len(lines), -1)
        acc.add(y[lines], ref)
        log(f"[whole fwd] {name}: lines {l0}..{lines[-1]} of {nl}, rel_l2 so far {acc.rel:.3e}")
    summary(f"[whole fwd] {name}: whole-tensor rel_l2={acc.rel:.3e} worst line={acc.worst:.3e} "
        f"(tol {TOL[w.dtype]:.0e}, {nl} lines)")
    assert acc.rel <= TOL[w.dtype] and acc.worst <= TOL[w.dtype]


@pytest.mark.parametrize("name", BACKWARD)
def test_backward_every_element(name):
    import torch
    from paper_2607_19378_amd import hyenand as H
    w = W.WORKLOADS[name]
    log(f"[whole bwd] {name}: generating {w.shape} {w.pad_mode} {w.dtype}")
    inp = W.generate(w)
    gy = W.quantise(np.random.default_rng(4321).standard_normal(w.shape), w.dtype)
    dev = [to_device(a, w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, inp.D)]
    got = H.backward(*dev, to_device(gy, w.dtype), w.pad_mode)
    torch.cuda.synchronize()
    del dev
    nl = w.B * w.C
    got_host = []
    for g in got[:4]:
        assert bool(torch.isfinite(g.float()).all())
        got_host.append(from_device(g).reshape(w.B, w.C, -1))
    gD = from_device(got[4])
    del got
    torch.cuda.empty_cache()
    cc = max(1, min(w.C, _chunk_lines(w, unit_lines=2 * w.B)))  # the backward holds three spectra
    accs = [Acc() for _ in range(4)]
    accD = Acc()
    grid = tuple(w.grid)
    for c0 in range(0, w.C, cc):
        chans = np.arange(c0, min(w.C, c0 + cc))
        sub = [W.storage_to_f64(a[:, chans], w.dtype) for a in (inp.x1, inp.x2, inp.v, inp.k, gy)]
        Dsub = W.storage_to_f64(inp.D, w.dtype)[chans]
        ref = oracle.backward_fft(sub[0], sub[1], sub[2], sub[3], Dsub, sub[4], w.pad_mode)
        for j in range(4):
            accs[j].add(got_host[j][:, chans].reshape(-1, int(np.prod(grid))),
                        ref[j].reshape(-1, int(np.prod(grid))))
        accD.add(gD[chans][None], ref[4][None], per_line=False)
        log(f"[whole bwd] {name}: channels {c0}..{chans[-1]} of {w.C}: "
            + " ".join(f"{n}={a.rel:.2e}" for n, a in zip(NAMES, accs + [accD])))
    summary(f"[whole bwd] {name}: whole-tensor " + " ".join(f"{n}={a.rel:.3e}" for n, a in zip(NAMES, accs + [accD]))
        + " worst line " + " ".join(f"{n}={a.worst:.3e}" for n, a in zip(NAMES, accs))
        + f" (tol {TOL[w.dtype]:.0e}, {nl} lines)")
    for a in accs:
        assert a.rel <= TOL[w.dtype] and a.worst <= TOL[w.dtype]
    assert accD.rel <= TOL[w.dtype]
