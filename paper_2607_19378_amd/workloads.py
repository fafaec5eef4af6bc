"""Seeded synthetic workloads for the gated N-D FFT long convolution.

This module only draws and quantises inputs.  It holds none of the operator's
arithmetic, so both the HIP path and the CPU oracle can consume the very same
bytes without sharing any code that computes the method.

Five named workloads stand in for the paper's data (none of the paper's
datasets is used):

* ``conv1d_4k``   -- 1D linear, fp32, B=1, C=64, L=4096 (the 1D spatial-recall
  canvas length of the controlled spatial-recall experiments).
* ``conv2d_64``   -- 2D linear, fp32, B=8, C=256, 64x64 (image-like; the 2D
  spatial-recall canvas size).
* ``conv2d_512c`` -- 2D circular, fp32, B=4, C=128, 512x512 smooth periodic
  fields (the periodic 512x512 PDE fields of the PDE-surrogate experiments).
* ``conv3d_128``  -- 3D linear, bf16 storage, B=1, C=64, 128^3 (volumes).
* ``conv1d_1m``   -- 1D linear, bf16 storage, B=1, C=256, L=2^20 (genomics-scale
  long context, the 1M point of the context-length study).

Two more, outside the five: ``conv2d_64_centered`` -- the image workload with
the paper's own non-circular kernel, evaluated on the double grid (127 x 127
points per 64 x 64 image, pad mode "centered"); ``conv2d_14_patches`` -- the
14 x 14 patch grid of a 224 x 224 image at patch 16 (the ImageNet models'
grid; ViT-Small width, C = 384), natural images and so the centered double
grid (27 x 27 kernel points), B = 16: a grid whose extents are not powers of
two.

Draw recipe (identical for every workload): ``numpy.random.SeedSequence(seed)``
spawns one child per tensor in the order x1, x2, v, kernel noise, D; each
tensor is drawn in C order in blocks of 2^22 elements, block j from a PCG64
stream seeded by the j-th child of that tensor's sequence (so blocks can be
filled in parallel and the bytes do not depend on the thread count).  Values
are ``standard_normal`` float64, rounded once, round-to-nearest-even, to the
storage dtype.  The per-sample kernel is
noise times a decay window evaluated in index units from index 0 (the
zero-displacement tap):

* 1D: ``exp(-l / tau) / sqrt(L)`` with ``l`` the index;
* 2D/3D linear: ``exp(-r / tau)`` with ``r`` the Euclidean index distance from
  the origin;
* 2D circular: ``exp(-r / tau)`` with ``r`` the periodic (wrap-around) distance;
* centered: ``exp(-r / tau)`` on the 2 L_d - 1 points per axis, ``r`` the
  Euclidean distance of the displacement (index minus L_d - 1) from zero.

The circular workload's x1, x2, v are smooth fields: white noise filtered with
a periodic separable Gaussian (sigma = 4 px, taps truncated at +-16, weights
normalised to sum 1), then standardised per (b, c) field to zero mean and unit
(population) variance.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np

LINEAR = "linear"
CIRCULAR = "circular"
CENTERED = "centered"


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    C: int
    grid: Tuple[int, ...]
    pad_mode: str
    dtype: str  # "f32" or "bf16" (storage); compute is fp32 in the kernels
    seed: int
    tau: float  # decay length of the kernel window, in index units
    kernel_norm: bool = False  # 1D windows carry an extra 1/sqrt(L)
    smooth_sigma: Optional[float] = None  # Gaussian low-pass of x1, x2, v
    description: str = ""

    @property
    def ndim(self) -> int:
        return len(self.grid)

    @property
    def shape(self) -> Tuple[int, ...]:
        return (self.B, self.C) + tuple(self.grid)

    @property
    def elems(self) -> int:
        n = self.B * self.C
        for g in self.grid:
            n *= g
        return n

    @property
    def kernel_shape(self) -> Tuple[int, ...]:
        """[B, C, K...]: the grid, or 2 L_d - 1 points per axis centered."""
        if self.pad_mode == CENTERED:
            return (self.B, self.C) + tuple(2 * g - 1 for g in self.grid)
        return self.shape

    @property
    def storage_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def scaled(self, B: Optional[int] = None, C: Optional[int] = None,
               grid: Optional[Tuple[int, ...]] = None, name: Optional[str] = None,
               seed: Optional[int] = None) -> "Workload":
        """Same recipe at another size (used for small parity cases)."""
        return Workload(
            name=name or (self.name + "_scaled"),
            B=self.B if B is None else B,
            C=self.C if C is None else C,
            grid=self.grid if grid is None else tuple(grid),
            pad_mode=self.pad_mode, dtype=self.dtype,
            seed=self.seed if seed is None else seed,
            tau=self.tau, kernel_norm=self.kernel_norm,
            smooth_sigma=self.smooth_sigma, description=self.description)


WORKLOADS: Dict[str, Workload] = {
    "conv1d_4k": Workload(
        "conv1d_4k", 1, 64, (4096,), LINEAR, "f32", 20261, 1024.0, kernel_norm=True,
        description="1D linear gated FFT conv, fp32, B=1 C=64 L=4096, pad 8192, crop first L"),
    "conv2d_64": Workload(
        "conv2d_64", 8, 256, (64, 64), LINEAR, "f32", 20262, 16.0,
        description="2D linear gated FFT conv, fp32, B=8 C=256 64x64, pad 128x128, crop 64x64"),
    "conv2d_512c": Workload(
        "conv2d_512c", 4, 128, (512, 512), CIRCULAR, "f32", 20263, 64.0, smooth_sigma=4.0,
        description="2D circular gated FFT conv, fp32, B=4 C=128 512x512 smooth periodic fields"),
    "conv3d_128": Workload(
        "conv3d_128", 1, 64, (128, 128, 128), LINEAR, "bf16", 20264, 24.0,
        description="3D linear gated FFT conv, bf16 storage, B=1 C=64 128^3, pad 256^3, crop 128^3"),
    "conv1d_1m": Workload(
        "conv1d_1m", 1, 256, (1 << 20,), LINEAR, "bf16", 20265, 65536.0, kernel_norm=True,
        description="1D linear gated FFT conv, bf16 storage, B=1 C=256 L=2^20, pad 2^21, crop first L"),
    "conv2d_64_centered": Workload(
        "conv2d_64_centered", 8, 256, (64, 64), CENTERED, "f32", 20266, 16.0,
        description="2D gated FFT conv with 127x127 centered kernels, fp32, B=8 C=256 64x64, pad 128x128"),
    "conv2d_14_patches": Workload(
        "conv2d_14_patches", 16, 384, (14, 14), CENTERED, "f32", 20267, 4.0,
        description="2D gated FFT conv on 14x14 patch grids with 27x27 centered kernels, fp32, B=16 C=384"),
}

# Order in which the workloads are listed (small 1D case first).
ORDER = ["conv1d_4k", "conv2d_64", "conv2d_512c", "conv3d_128", "conv1d_1m"]


# ----------------------------------------------------------------------------
# Rounding to the storage dtype (one RNE rounding from float64)
# ----------------------------------------------------------------------------

def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values once, to nearest-even, to bfloat16; return uint16 bits.

    The rounding is done on the float64 bit pattern: the 52-bit significand is
    cut to bfloat16's 7 stored bits with a round-half-to-even bias (a carry
    into the exponent is the correct result), so there is no intermediate
    float32 rounding.  The result is exactly representable in float32, whose
    upper 16 bits are the bfloat16 bits.  Finite, normal-range inputs.
    """
    b = np.ascontiguousarray(x, dtype=np.float64).view(np.uint64)
    drop = np.uint64(45)                     # 52 - 7 significand bits removed
    half = np.uint64((1 << 44) - 1)
    lsb = (b >> drop) & np.uint64(1)
    r = ((b + half + lsb) >> drop) << drop
    f32 = r.view(np.float64).astype(np.float32)   # exact
    return (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def quantise(x64: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage array (float32 values, or uint16 bf16 bits)."""
    if dtype == "f32":
        return np.ascontiguousarray(x64, dtype=np.float32)
    if dtype == "bf16":
        return np.ascontiguousarray(round_to_bf16_bits(x64))
    raise ValueError(f"unknown dtype {dtype!r}")


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact upcast of stored values to float64."""
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------
# Windows and smoothing used to shape the synthetic data
# ----------------------------------------------------------------------------

def decay_window(grid: Tuple[int, ...], tau: float, periodic: bool, centered: bool = False) -> np.ndarray:
    """exp(-r/tau) on the grid, r the (periodic) Euclidean index distance to 0;
    centered: on 2 n - 1 points per axis, r the distance of the displacement."""
    if centered:
        grid = tuple(2 * n - 1 for n in grid)
    r2 = np.zeros(grid, dtype=np.float64)
    for ax, n in enumerate(grid):
        i = np.arange(n, dtype=np.float64)
        if periodic:
            i = np.minimum(i, n - i)
        if centered:
            i = i - (n - 1) / 2
        shp = [1] * len(grid)
        shp[ax] = n
        r2 = r2 + (i * i).reshape(shp)
    return np.exp(-np.sqrt(r2) / tau)


def _gaussian_taps(sigma: float, radius: int) -> np.ndarray:
    t = np.arange(-radius, radius + 1, dtype=np.float64)
    w = np.exp(-0.5 * (t / sigma) ** 2)
    return w / w.sum()


def smooth_fields(noise: np.ndarray, sigma: float) -> np.ndarray:
    """Periodic separable Gaussian low-pass over the last two axes (taps
    truncated at +-round(4 sigma), weights normalised to sum 1, wrap-around
    boundaries), then per-field standardisation to zero mean and unit
    population variance.  Fields are processed independently, in threads."""
    from scipy import ndimage
    radius = int(4.0 * sigma + 0.5)
    taps = _gaussian_taps(sigma, radius)
    *lead, H, W = noise.shape
    src = np.ascontiguousarray(noise, dtype=np.float64).reshape(-1, H, W)
    out = np.empty_like(src)

    def one(i):
        f = ndimage.correlate1d(src[i], taps, axis=1, mode="wrap")
        f = ndimage.correlate1d(f, taps, axis=0, mode="wrap")
        f -= f.mean()
        f /= f.std()
        out[i] = f
    _parallel(one, src.shape[0])
    return out.reshape(noise.shape)


# ----------------------------------------------------------------------------
# Generation
# ----------------------------------------------------------------------------

@dataclass
class Inputs:
    """Quantised inputs of one workload instance (storage arrays)."""
    workload: Workload
    x1: np.ndarray
    x2: np.ndarray
    v: np.ndarray
    k: np.ndarray
    D: np.ndarray
    extra: dict = field(default_factory=dict)

    def as_f64(self):
        d = self.workload.dtype
        return tuple(storage_to_f64(a, d) for a in (self.x1, self.x2, self.v, self.k, self.D))


_BLOCK = 1 << 22


def _threads() -> int:
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _parallel(fn, nblocks: int) -> None:
    from concurrent.futures import ThreadPoolExecutor
    if nblocks <= 1:
        for j in range(nblocks):
            fn(j)
        return
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(fn, range(nblocks)))


def _normals(seq: np.random.SeedSequence, shape) -> np.ndarray:
    out = np.empty(shape, dtype=np.float64)
    flat = out.reshape(-1)
    nb = (flat.size + _BLOCK - 1) // _BLOCK
    kids = seq.spawn(nb)

    def fill(j):
        g = np.random.Generator(np.random.PCG64(kids[j]))
        g.standard_normal(out=flat[j * _BLOCK:(j + 1) * _BLOCK])
    _parallel(fill, nb)
    return out


def _quantise_parallel(x64: np.ndarray, dtype: str) -> np.ndarray:
    flat = x64.reshape(-1)
    out = np.empty(flat.size, dtype=np.float32 if dtype == "f32" else np.uint16)
    nb = (flat.size + _BLOCK - 1) // _BLOCK

    def q(j):
        sl = slice(j * _BLOCK, (j + 1) * _BLOCK)
        out[sl] = quantise(flat[sl], dtype)
    _parallel(q, nb)
    return out.reshape(x64.shape)


def generate(w: Workload) -> Inputs:
    seqs = np.random.SeedSequence(w.seed).spawn(5)  # x1, x2, v, kernel noise, D
    shp = w.shape
    out = []
    for i in range(3):
        a = _normals(seqs[i], shp)
        if w.smooth_sigma is not None:
            a = smooth_fields(a, w.smooth_sigma)
        out.append(_quantise_parallel(a, w.dtype))
        del a
    win = decay_window(w.grid, w.tau, periodic=(w.pad_mode == CIRCULAR), centered=(w.pad_mode == CENTERED))
    if w.kernel_norm:
        L = 1
        for g in w.grid:
            L *= g
        win = win / np.sqrt(L)
    kn = _normals(seqs[3], w.kernel_shape)
    kv = kn.reshape((-1,) + win.shape)

    def scale(j):
        kv[j] *= win
    _parallel(scale, kv.shape[0])
    k = _quantise_parallel(kn, w.dtype)
    del kn, kv
    D = quantise(_normals(seqs[4], (w.C,)), w.dtype)
    return Inputs(w, out[0], out[1], out[2], k, D)


def random_case(B: int, C: int, grid, pad_mode: str, dtype: str, seed: int,
                tau: Optional[float] = None) -> Inputs:
    """Small seeded case with the same recipe (N(0,1) data, decaying kernel)."""
    grid = tuple(int(g) for g in grid)
    if tau is None:
        tau = max(1.0, max(grid) / 4.0)
    w = Workload(f"case_{len(grid)}d_{pad_mode}_{dtype}_{seed}", B, C, grid, pad_mode,
                 dtype, seed, tau, kernel_norm=(len(grid) == 1))
    return generate(w)


def siren_params(seed: int, ndim: int, hidden: int, layers: int, C: int, B: int, modulated: bool = True,
                 bias: bool = True, window_kind: str = "gaussian", blocks: int = 4,
                 omega_range: Tuple[float, float] = (1.0, 30.0), scale_range: Tuple[float, float] = (0.5, 1.5),
                 rho: float = 0.1, sigma_range: Tuple[float, float] = (1.0, 0.05),
                 film_spread: float = 0.1) -> Dict[str, Optional[np.ndarray]]:
    """Seeded fp32 parameters of the kernel-synthesis network, drawn the way
    the paper initialises it (section 3.2.1 and the masking/initialisation
    appendix), with FiLM moved away from its identity start as training would:

    * omega0: ``blocks`` equal blocks of hidden units with base frequencies on
      a linear schedule over ``omega_range``, each unit's base scaled by
      s ~ U(``scale_range``);
    * W1 ~ U(-1/sqrt(N), 1/sqrt(N)) (the N-D first-layer correction);
    * hidden W_j and Wout ~ U(-sqrt(6/Hf), sqrt(6/Hf)) (SIREN's hidden-layer
      range), near-block-diagonal: entries linking different blocks (channels
      are assigned to blocks in order) scaled by ``rho``;
    * biases ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in));
    * Gaussian window: sigma[d, c] on a log-spaced ramp over the channels from
      ``sigma_range[0]`` (channel 0, paired with the lowest-frequency block)
      to ``sigma_range[1]``, times a per-axis factor U(0.8, 1.25);
      exponential window: alpha[c] log-spaced over [0.5, 8];
    * gamma = 1 + film_spread N(0, 1), beta = film_spread N(0, 1), per (b, j, unit).

    The draw order is fixed (one child SeedSequence per array, in the order of
    the keys below); arrays that are switched off are None."""
    seqs = np.random.SeedSequence(seed).spawn(9)
    rng = [np.random.Generator(np.random.PCG64(s)) for s in seqs]
    H, J = hidden, layers
    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    ublock = (np.arange(H) * blocks) // H
    cblock = (np.arange(C) * blocks) // C
    lo, hi = omega_range
    base = lo + (hi - lo) * ublock / max(1, blocks - 1)
    omega0 = base * rng[0].uniform(*scale_range, H)
    W1 = rng[1].uniform(-1.0, 1.0, (ndim, H)) / np.sqrt(ndim)
    lim = np.sqrt(6.0 / H)
    Wh = rng[2].uniform(-lim, lim, (J - 1, H, H))
    Wh *= np.where(ublock[:, None] == ublock[None, :], 1.0, rho)[None]
    Wout = rng[3].uniform(-lim, lim, (H, C)) * np.where(ublock[:, None] == cblock[None, :], 1.0, rho)
    b = None
    if bias:
        b = np.empty((J, H))
        b[0] = rng[4].uniform(-1.0, 1.0, H) / np.sqrt(ndim)
        b[1:] = rng[4].uniform(-1.0, 1.0, (J - 1, H)) / np.sqrt(H)
    if window_kind == "gaussian":
        ramp = np.geomspace(sigma_range[0], sigma_range[1], C)
        window = ramp[None, :] * rng[5].uniform(0.8, 1.25, (ndim, 1))
    else:
        window = np.geomspace(0.5, 8.0, C)
    gamma = beta = None
    if modulated:
        gamma = 1.0 + film_spread * rng[6].standard_normal((B, J, H))
        beta = film_spread * rng[7].standard_normal((B, J, H))
    return dict(omega0=f32(omega0), W1=f32(W1), Wh=f32(Wh) if J > 1 else None, Wout=f32(Wout),
                window=f32(window), bias=None if b is None else f32(b), gamma=None if gamma is None else f32(gamma),
                beta=None if beta is None else f32(beta))


def modal_params(seed: int, C: int, M: int, L: int) -> Dict[str, np.ndarray]:
    """Seeded fp32 poles and residues of a modal long filter of order M per
    channel, spread the way a trained long-convolution filter bank spans its
    context: decay rates log-uniform between one e-fold over the whole
    length (-1/L) and over two points (-0.5), angles uniform in [0, pi),
    residues N(0, 1 / M).  Draw order: log_mag, angle, res_re, res_im."""
    seqs = np.random.SeedSequence(seed).spawn(4)
    rng = [np.random.Generator(np.random.PCG64(s)) for s in seqs]
    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    log_mag = -np.exp(rng[0].uniform(np.log(1.0 / max(L, 2)), np.log(0.5), (C, M)))
    angle = rng[1].uniform(0.0, np.pi, (C, M))
    re = rng[2].standard_normal((C, M)) / np.sqrt(M)
    im = rng[3].standard_normal((C, M)) / np.sqrt(M)
    return dict(log_mag=f32(log_mag), angle=f32(angle), res_re=f32(re), res_im=f32(im))
