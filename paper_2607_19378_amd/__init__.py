"""MI355X-native gated N-D FFT long convolution (the HyenaND hot path).

``fftconv(x1, x2, v, k, D, pad_mode)`` computes, for every sample and channel,
``y = x2 * (k conv (x1*v) + D*(x1*v))`` on a 1D/2D/3D grid with zero-padded
(linear) or circular convolution, through the C ABI of libhyenand (HIP
kernels for gfx950).  Imports of the binding are lazy so that the workload
generators can be used without torch or the library.
"""

__all__ = ["fftconv", "fftconv_into", "workspace_size", "workspace_min", "plan_name"]


def __getattr__(name):
    if name in __all__:
        from . import hyenand as _h
        return getattr(_h, name)
    raise AttributeError(name)
