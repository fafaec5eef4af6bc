"""fp64 CPU oracle for the gated N-D FFT long convolution.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library and never imports it.

The arithmetic lives in ``oracle.c`` (plain C, IEEE double):

* :func:`conv_direct` / :func:`conv_direct_points` evaluate the operator's
  definition (Def. A.2 and Def. A.3 of the appendix "Gated Hyena Computes
  Separable Attention", with the long convolution of Eq. (HyenaND), section
  3.2) as an explicit sum;
* :func:`conv_fft` evaluates it through the convolution theorem with the C
  file's own radix-2 FFT;
* :func:`fft1d` exposes that FFT so it can be pinned against a naive DFT;
* :func:`operator` evaluates the whole HyenaND operator of Eq. (HyenaND):
  l2-normalised q times SiLU(kin), RMSNorm across channels, the gated long
  convolution with Sigmoid(vin), RMSNorm across channels;
* :func:`kernel_synth` evaluates the implicit, input-dependent kernel K(x) of
  sections 3.2.1-3.2.2 (a SIREN over the grid coordinates, FiLM-modulated per
  sample, times a per-channel window) on a convolution's kernel grid;
* :func:`modal_filter` evaluates the implicit modal filter of order M (the
  appendix "Filter Generation"): k[c, t] = Re sum_m R[c, m] lambda[c, m]^t;
* :func:`backward_direct` / :func:`backward_fft` give the gradients of a
  scalar loss through y (gx1, gx2, gv, gk, gD for a given gy = dLoss/dy), as
  explicit sums and through the FFT.

Inputs are float64 arrays of shape [B, C, L1, ..., LN] (x1, x2, v, k) and [C]
(D).  ``pad_mode`` is "linear" (zero-padded, cropped to the first L_d outputs
on every axis), "circular", or "centered" (forward only): the paper's kernel
on the double grid, k of shape [B, C, 2 L1 - 1, ..., 2 LN - 1] with index
L_d - 1 the zero displacement, input zero-padded and output cropped as in
"linear".
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")
# HYENAND_ORACLE_LIBRARY: a sanitizer build of the same oracle.c to load instead
_SO_OVERRIDE = os.environ.get("HYENAND_ORACLE_LIBRARY")
_lock = threading.Lock()
_lib = None

_i64p = ctypes.POINTER(ctypes.c_int64)
_f64p = ctypes.POINTER(ctypes.c_double)


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with the host C compiler."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC,
               "-lm", "-lpthread"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if _SO_OVERRIDE:
                L = ctypes.CDLL(_SO_OVERRIDE)
            else:
                if not os.path.exists(_SO):
                    build()
                L = ctypes.CDLL(_SO)
            sig = [_f64p] * 5
            L.oracle_direct.argtypes = sig + [_f64p, ctypes.c_int, _i64p, ctypes.c_int, _i64p,
                                              ctypes.c_int64, ctypes.c_int]
            L.oracle_fft.argtypes = L.oracle_direct.argtypes
            L.oracle_direct_points.argtypes = sig + [ctypes.c_int, _i64p, ctypes.c_int, _i64p,
                                                     ctypes.c_int64, _f64p, ctypes.c_int]
            L.oracle_fft1d.argtypes = [_f64p, ctypes.c_int64, ctypes.c_int]
            bsig = [_f64p] * 11 + [ctypes.c_int, _i64p, ctypes.c_int, ctypes.c_int]
            L.oracle_backward_direct.argtypes = bsig
            L.oracle_backward_fft.argtypes = bsig
            L.oracle_operator.argtypes = [_f64p] * 7 + [ctypes.c_double, ctypes.c_double, _f64p, ctypes.c_int,
                                                        _i64p, ctypes.c_int, ctypes.c_int]
            L.oracle_kernel_synth.argtypes = [_f64p] * 8 + [ctypes.c_int, _f64p, ctypes.c_int, _i64p,
                                                            ctypes.c_int, ctypes.c_int, ctypes.c_int]
            L.oracle_modal_filter.argtypes = [_f64p] * 5 + [ctypes.c_int64] * 3
            for f in (L.oracle_direct, L.oracle_fft, L.oracle_direct_points, L.oracle_fft1d,
                      L.oracle_backward_direct, L.oracle_backward_fft, L.oracle_operator,
                      L.oracle_kernel_synth, L.oracle_modal_filter):
                f.restype = ctypes.c_int
            _lib = L
        return _lib


def default_threads() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def kernel_shape(shape, pad_mode):
    """Shape of k for a call on tensors of `shape` ([B, C, L1..LN])."""
    shape = tuple(int(s) for s in shape)
    if pad_mode == "centered":
        return shape[:2] + tuple(2 * s - 1 for s in shape[2:])
    return shape


def _prep(x1, x2, v, k, D, pad_mode="linear"):
    arrs = [np.ascontiguousarray(a, dtype=np.float64) for a in (x1, x2, v, k, D)]
    shp = arrs[0].shape
    if len(shp) < 3 or len(shp) > 5:
        raise ValueError("tensors must be [B, C, L1..LN] with N in 1..3")
    for a in arrs[1:3]:
        if a.shape != shp:
            raise ValueError("x1, x2, v must share one shape")
    if arrs[3].shape != kernel_shape(shp, pad_mode):
        raise ValueError(f"k must have shape {kernel_shape(shp, pad_mode)} for pad_mode {pad_mode!r}")
    if arrs[4].shape != (shp[1],):
        raise ValueError("D must have shape [C]")
    dims = np.asarray(shp, dtype=np.int64)
    return arrs, dims, len(shp) - 2


def _ptr(a):
    return a.ctypes.data_as(_f64p)


_MODES = {"linear": 0, "circular": 1, "centered": 2}


def _mode(pad_mode: str) -> int:
    if pad_mode not in _MODES:
        raise ValueError(f"pad_mode must be 'linear', 'circular' or 'centered', got {pad_mode!r}")
    return _MODES[pad_mode]


def _lines_arg(lines):
    if lines is None:
        return None, None, 0
    la = np.ascontiguousarray(lines, dtype=np.int64)
    return la, la.ctypes.data_as(_i64p), la.size


def _run_lines(fn, x1, x2, v, k, D, pad_mode, lines, nthreads):
    arrs, dims, nd = _prep(x1, x2, v, k, D, pad_mode)
    y = np.zeros(arrs[0].shape, dtype=np.float64)
    la, lp, nl = _lines_arg(lines)
    rc = fn(*[_ptr(a) for a in arrs], _ptr(y), nd, dims.ctypes.data_as(_i64p), _mode(pad_mode),
            lp, nl, int(nthreads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    return y


def conv_direct(x1, x2, v, k, D, pad_mode="linear", lines=None, nthreads=None):
    """y by the explicit sum. ``lines`` selects flat (b*C + c) indices; other
    lines of the returned array are left at zero."""
    return _run_lines(lib().oracle_direct, x1, x2, v, k, D, pad_mode, lines, nthreads)


def conv_fft(x1, x2, v, k, D, pad_mode="linear", lines=None, nthreads=None):
    """y through the convolution theorem with the oracle's own FFT."""
    return _run_lines(lib().oracle_fft, x1, x2, v, k, D, pad_mode, lines, nthreads)


def conv_direct_points(x1, x2, v, k, D, flat_idx, pad_mode="linear", nthreads=None):
    """y at the given flat indices of the [B, C, L...] output, by the explicit sum."""
    arrs, dims, nd = _prep(x1, x2, v, k, D, pad_mode)
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.zeros(idx.size, dtype=np.float64)
    rc = lib().oracle_direct_points(*[_ptr(a) for a in arrs], nd, dims.ctypes.data_as(_i64p),
                                    _mode(pad_mode), idx.ctypes.data_as(_i64p), idx.size,
                                    _ptr(out), int(nthreads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    return out


def fft1d(x, sign=-1):
    """Unnormalised DFT of a complex vector (length a power of two) by the
    oracle's radix-2 FFT: X[f] = sum_n x[n] exp(sign 2 pi i f n / N)."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.complex128).copy())
    rc = lib().oracle_fft1d(a.ctypes.data_as(_f64p), a.size, int(sign))
    if rc != 0:
        raise RuntimeError(f"oracle_fft1d returned {rc}")
    return a


def _backward(fn, x1, x2, v, k, D, gy, pad_mode, nthreads):
    arrs, dims, nd = _prep(x1, x2, v, k, D, pad_mode)
    g = np.ascontiguousarray(gy, dtype=np.float64)
    if g.shape != arrs[0].shape:
        raise ValueError("gy must have the shape of y")
    outs = [np.zeros(arrs[0].shape, dtype=np.float64) for _ in range(3)]
    outs.append(np.zeros(arrs[3].shape, dtype=np.float64))  # gk, shaped like k
    gD = np.zeros(arrs[4].shape, dtype=np.float64)
    rc = fn(*[_ptr(a) for a in arrs], _ptr(g), *[_ptr(o) for o in outs], _ptr(gD), nd,
            dims.ctypes.data_as(_i64p), _mode(pad_mode), int(nthreads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    gx1, gx2, gv, gk = outs
    return gx1, gx2, gv, gk, gD


def backward_direct(x1, x2, v, k, D, gy, pad_mode="linear", nthreads=None):
    """(gx1, gx2, gv, gk, gD) for dLoss/dy = gy, by explicit sums (any extents,
    every pad mode; centred gk has the shape of the centred k)."""
    return _backward(lib().oracle_backward_direct, x1, x2, v, k, D, gy, pad_mode, nthreads)


def backward_fft(x1, x2, v, k, D, gy, pad_mode="linear", nthreads=None):
    """(gx1, gx2, gv, gk, gD) through the convolution theorem (linear and
    circular modes; circular needs power-of-two extents)."""
    if pad_mode == "centered":
        raise ValueError("the FFT backward takes pad_mode 'linear' or 'circular'")
    return _backward(lib().oracle_backward_fft, x1, x2, v, k, D, gy, pad_mode, nthreads)


def operator(q, kin, vin, k, D, w_in, w_out, eps_l2=1e-6, eps_rms=1e-6, pad_mode="linear", nthreads=None):
    """The HyenaND operator, Eq. (HyenaND): y = RMSNorm(Sigmoid(vin) * (k conv
    RMSNorm(l2(q) * SiLU(kin)) + D * that)), both norms across the C channels
    of every (b, grid point), with per-channel weights w_in and w_out."""
    arrs, dims, nd = _prep(q, vin, kin, k, D, pad_mode)
    qa, va, ka, kk, Da = arrs
    wi = np.ascontiguousarray(w_in, dtype=np.float64)
    wo = np.ascontiguousarray(w_out, dtype=np.float64)
    if wi.shape != Da.shape or wo.shape != Da.shape:
        raise ValueError("w_in and w_out must have shape [C]")
    y = np.zeros(qa.shape, dtype=np.float64)
    rc = lib().oracle_operator(_ptr(qa), _ptr(ka), _ptr(va), _ptr(kk), _ptr(Da), _ptr(wi), _ptr(wo),
                               float(eps_l2), float(eps_rms), _ptr(y), nd, dims.ctypes.data_as(_i64p),
                               _mode(pad_mode), int(nthreads or default_threads()))
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    return y


WINDOWS = {"gaussian": 0, "exponential": 1}


def synth_grid(shape, pad_mode):
    """Kernel-grid extents that kernel synthesis evaluates for a convolution
    on tensors of `shape` ([B, C, L1..LN])."""
    return kernel_shape(shape, pad_mode)[2:]


def kernel_synth(shape, omega0, W1, Wh, Wout, window, gamma=None, beta=None, bias=None,
                 window_kind="gaussian", pad_mode="linear"):
    """The HyenaND kernel K(x) on the kernel grid of a convolution of `shape`
    ([B, C, L1..LN]): a J-layer SIREN of width Hf over the normalised grid
    coordinates (Eq. (kernel)), each sine's output FiLM-modulated by the
    sample's (gamma_j, beta_j) (Eq. (film)), projected to the C channels and
    multiplied by the channel's window (Eq. (mask): Gaussian, win = sigma
    [N, C]; or exponential, win = alpha [C]).

    omega0 [Hf], W1 [N, Hf], Wh [J-1, Hf, Hf] (rows = input units), Wout
    [Hf, C], bias [J, Hf] or None, gamma / beta [B, J, Hf] or both None.
    Returns [B, C, grid...] (modulated) or [C, grid...] (both None)."""
    shape = tuple(int(s) for s in shape)
    nd = len(shape) - 2
    if nd < 1 or nd > 3:
        raise ValueError("shape must be [B, C, L1..LN] with N in 1..3")
    B, C = shape[:2]
    om = np.ascontiguousarray(omega0, dtype=np.float64)
    Hf = om.size
    w1 = np.ascontiguousarray(W1, dtype=np.float64)
    wo = np.ascontiguousarray(Wout, dtype=np.float64)
    wh = np.ascontiguousarray(Wh if Wh is not None else np.zeros((0, Hf, Hf)), dtype=np.float64)
    J = wh.shape[0] + 1
    if om.shape != (Hf,) or w1.shape != (nd, Hf) or wo.shape != (Hf, C) or wh.shape != (J - 1, Hf, Hf):
        raise ValueError("weight shapes do not match (omega0 [Hf], W1 [N, Hf], Wh [J-1, Hf, Hf], Wout [Hf, C])")
    if window_kind not in WINDOWS:
        raise ValueError(f"window_kind must be one of {sorted(WINDOWS)}")
    win = np.ascontiguousarray(window, dtype=np.float64)
    if win.shape != ((nd, C) if window_kind == "gaussian" else (C,)):
        raise ValueError("window must be sigma [N, C] (gaussian) or alpha [C] (exponential)")
    if (gamma is None) != (beta is None):
        raise ValueError("gamma and beta go together")
    mods = [None, None]
    if gamma is not None:
        mods = [np.ascontiguousarray(a, dtype=np.float64) for a in (gamma, beta)]
        if any(m.shape != (B, J, Hf) for m in mods):
            raise ValueError("gamma and beta must be [B, J, Hf]")
    bi = None
    if bias is not None:
        bi = np.ascontiguousarray(bias, dtype=np.float64)
        if bi.shape != (J, Hf):
            raise ValueError("bias must be [J, Hf]")
    grid = synth_grid(shape, pad_mode)
    out = np.zeros(((B,) if gamma is not None else ()) + (C,) + tuple(grid), dtype=np.float64)
    dims = np.asarray(shape, dtype=np.int64)
    null = ctypes.cast(None, _f64p)
    p = lambda a: null if a is None else _ptr(a)
    rc = lib().oracle_kernel_synth(_ptr(om), _ptr(w1), _ptr(wh), p(bi), p(mods[0]), p(mods[1]), _ptr(wo),
                                   _ptr(win), WINDOWS[window_kind], _ptr(out), nd,
                                   dims.ctypes.data_as(_i64p), _mode(pad_mode), Hf, J)
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    return out


def modal_filter(log_mag, angle, res_re, res_im, L):
    """k [C, L] with k[c, t] = Re sum_m (res_re + i res_im)[c, m] *
    exp((log_mag + i angle)[c, m] * t): a sum of M damped complex exponentials
    per channel.  Parameters are [C, M]."""
    arrs = [np.ascontiguousarray(x, dtype=np.float64) for x in (log_mag, angle, res_re, res_im)]
    if arrs[0].ndim != 2 or any(x.shape != arrs[0].shape for x in arrs):
        raise ValueError("log_mag, angle, res_re and res_im must share one [C, M] shape")
    C, M = arrs[0].shape
    k = np.zeros((C, int(L)), dtype=np.float64)
    rc = lib().oracle_modal_filter(*[_ptr(x) for x in arrs], _ptr(k), C, M, int(L))
    if rc != 0:
        raise RuntimeError(f"oracle returned {rc}")
    return k
