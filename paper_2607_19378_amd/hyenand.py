"""Python binding of libhyenand (ctypes): argument marshalling only.

Every step of the operation runs in the HIP kernels behind the C ABI declared
in include/hyenand.h; PyTorch only provides device memory and the stream.
There is no fallback: if the library is missing or cannot be loaded, every
call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
# HYENAND_LIBRARY selects another build of the same library (the sanitizer
# build of paper_2607_19378_amd.build --sanitize)
LIB_PATH = os.environ.get("HYENAND_LIBRARY") or os.path.join(_PKG, "libhyenand.so")

OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_WORKSPACE_TOO_SMALL, ERR_HIP = range(5)
PAD_LINEAR, PAD_CIRCULAR, PAD_CENTERED = 0, 1, 2
DTYPE_F32, DTYPE_BF16 = 0, 1

EXPORTED = ("hyenand_fftconv", "hyenand_fftconv_shared_k", "hyenand_fftconv_noalloc", "hyenand_fftconv_modal", "hyenand_fftconv_workspace_size",
            "hyenand_fftconv_shared_k_workspace_size", "hyenand_fftconv_workspace_min",
            "hyenand_kernel_spectrum_size", "hyenand_kernel_spectrum", "hyenand_fftconv_spectrum",
            "hyenand_fftconv_plan_name", "hyenand_fftconv_backward", "hyenand_fftconv_backward_workspace_size",
            "hyenand_fftconv_backward_workspace_min", "hyenand_operator", "hyenand_operator_workspace_size",
            "hyenand_kernel_synth", "hyenand_modal_filter", "hyenand_status_string", "hyenand_last_error", "hyenand_version")

_lock = threading.Lock()
_lib = None


class HyenandError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libhyenand.so (built in-tree by paper_2607_19378_amd.build)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2607_19378_amd.build`")
            # torch first: its HIP runtime then satisfies the library's
            # dependency on libamdhip64.so.7, so the process holds one HIP
            # runtime.  Loaded before torch, the library would bring in the
            # system one beside torch's, and whichever of the two initialises
            # second finds no device.
            import torch  # noqa: F401
            L = ctypes.CDLL(LIB_PATH)
            i64p = ctypes.POINTER(ctypes.c_int64)
            vp = ctypes.c_void_p
            L.hyenand_fftconv.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_int, i64p, ctypes.c_int,
                                          ctypes.c_int, vp, ctypes.c_size_t, vp]
            L.hyenand_fftconv.restype = ctypes.c_int
            L.hyenand_fftconv_shared_k.argtypes = L.hyenand_fftconv.argtypes
            L.hyenand_fftconv_shared_k.restype = ctypes.c_int
            L.hyenand_fftconv_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_int, i64p, ctypes.c_int,
                                                  ctypes.c_int, vp]
            L.hyenand_fftconv_noalloc.restype = ctypes.c_int
            L.hyenand_fftconv_modal.argtypes = [vp] * 7 + [ctypes.c_int, vp, vp, ctypes.c_int, i64p, ctypes.c_int,
                                                           ctypes.c_int, vp, ctypes.c_size_t, vp]
            L.hyenand_fftconv_modal.restype = ctypes.c_int
            L.hyenand_kernel_spectrum.argtypes = [vp, vp, ctypes.c_size_t, ctypes.c_int, i64p, ctypes.c_int,
                                                  ctypes.c_int, vp]
            L.hyenand_kernel_spectrum.restype = ctypes.c_int
            L.hyenand_fftconv_spectrum.argtypes = [vp, vp, vp, vp, ctypes.c_size_t, vp, vp, ctypes.c_int, i64p,
                                                   ctypes.c_int, ctypes.c_int, vp]
            L.hyenand_fftconv_spectrum.restype = ctypes.c_int
            for name in ("hyenand_fftconv_workspace_size", "hyenand_fftconv_shared_k_workspace_size",
                         "hyenand_fftconv_workspace_min", "hyenand_kernel_spectrum_size"):
                f = getattr(L, name)
                f.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int,
                              ctypes.POINTER(ctypes.c_size_t)]
                f.restype = ctypes.c_int
            L.hyenand_fftconv_backward.argtypes = [vp] * 11 + [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int, vp,
                                                           ctypes.c_size_t, vp]
            L.hyenand_fftconv_backward.restype = ctypes.c_int
            L.hyenand_fftconv_backward_workspace_size.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int,
                                                                  ctypes.POINTER(ctypes.c_size_t)]
            L.hyenand_fftconv_backward_workspace_size.restype = ctypes.c_int
            L.hyenand_fftconv_backward_workspace_min.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int,
                                                                 ctypes.POINTER(ctypes.c_size_t)]
            L.hyenand_fftconv_backward_workspace_min.restype = ctypes.c_int
            L.hyenand_operator.argtypes = [vp] * 7 + [ctypes.c_float, ctypes.c_float, vp, ctypes.c_int, i64p,
                                                      ctypes.c_int, ctypes.c_int, vp, ctypes.c_size_t, vp]
            L.hyenand_operator.restype = ctypes.c_int
            L.hyenand_operator_workspace_size.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int,
                                                          ctypes.POINTER(ctypes.c_size_t)]
            L.hyenand_operator_workspace_size.restype = ctypes.c_int
            L.hyenand_kernel_synth.argtypes = [vp] * 8 + [ctypes.c_int] * 3 + [vp, ctypes.c_int, i64p, ctypes.c_int,
                                                                       ctypes.c_int, vp]
            L.hyenand_kernel_synth.restype = ctypes.c_int
            L.hyenand_modal_filter.argtypes = [vp] * 4 + [ctypes.c_int, vp, ctypes.c_int64, ctypes.c_int64,
                                                       ctypes.c_int, vp]
            L.hyenand_modal_filter.restype = ctypes.c_int
            L.hyenand_fftconv_plan_name.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int,
                                                    ctypes.c_char_p, ctypes.c_size_t]
            L.hyenand_fftconv_plan_name.restype = ctypes.c_int
            L.hyenand_status_string.argtypes = [ctypes.c_int]
            L.hyenand_status_string.restype = ctypes.c_char_p
            L.hyenand_last_error.argtypes = []
            L.hyenand_last_error.restype = ctypes.c_char_p
            L.hyenand_version.argtypes = []
            L.hyenand_version.restype = ctypes.c_int
            _lib = L
        return _lib


def _check(status: int) -> None:
    if status != OK:
        L = lib()
        detail = L.hyenand_last_error().decode()
        raise HyenandError(status, f"{L.hyenand_status_string(status).decode()}: {detail}")


def _dims(shape: Sequence[int]):
    arr = (ctypes.c_int64 * len(shape))(*[int(s) for s in shape])
    return len(shape) - 2, arr


_MODES = {"linear": 0, "circular": 1, "centered": 2}


def _mode(pad_mode: str) -> int:
    if pad_mode not in _MODES:
        raise ValueError(f"pad_mode must be 'linear', 'circular' or 'centered', got {pad_mode!r}")
    return _MODES[pad_mode]


def kernel_shape(shape, pad_mode: str, shared_k: bool = False):
    """Shape of k for tensors of `shape` ([B, C, L1..LN]): the same, or
    [B, C, 2 L1 - 1, ...] centered; without B with shared_k."""
    shape = tuple(int(x) for x in shape)
    grid = tuple(2 * x - 1 for x in shape[2:]) if pad_mode == "centered" else shape[2:]
    return (shape[1],) + grid if shared_k else shape[:2] + grid


def _dtype_code(dtype) -> int:
    import torch
    if dtype in (torch.float32, "f32", "float32"):
        return DTYPE_F32
    if dtype in (torch.bfloat16, "bf16", "bfloat16"):
        return DTYPE_BF16
    raise ValueError(f"unsupported dtype {dtype}")


def workspace_size(shape, pad_mode: str, dtype, shared_k: bool = False) -> int:
    """Recommended workspace bytes of hyenand_fftconv (shared_k: of
    hyenand_fftconv_shared_k, which may use more to transform each channel's
    kernel once)."""
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    fn = lib().hyenand_fftconv_shared_k_workspace_size if shared_k else lib().hyenand_fftconv_workspace_size
    _check(fn(nd, dims, _mode(pad_mode), _dtype_code(dtype), ctypes.byref(out)))
    return int(out.value)


def workspace_min(shape, pad_mode: str, dtype) -> int:
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    _check(lib().hyenand_fftconv_workspace_min(nd, dims, _mode(pad_mode), _dtype_code(dtype),
                                               ctypes.byref(out)))
    return int(out.value)


def plan_name(shape, pad_mode: str, dtype) -> str:
    nd, dims = _dims(shape)
    buf = ctypes.create_string_buffer(64)
    _check(lib().hyenand_fftconv_plan_name(nd, dims, _mode(pad_mode), _dtype_code(dtype), buf, 64))
    return buf.value.decode()


def version() -> int:
    return int(lib().hyenand_version())


def _ptr(t) -> int:
    return int(t.data_ptr())


def _keep_for_stream(stream, *tensors) -> None:
    """Tensors this module allocates on the current stream but hands to work
    on another `stream`: mark them used there, so that torch's caching
    allocator does not give their memory to a later allocation on the
    current stream while that work is still pending."""
    import torch
    if stream is None:
        return
    for t in tensors:
        if t is not None and stream != torch.cuda.current_stream(t.device):
            t.record_stream(stream)


class Prepared:
    """One hyenand_fftconv call with its arguments checked and marshalled
    once; calling the object enqueues the work again on the same buffers and
    stream (for loops that repeat a call, where per-call Python work would
    otherwise delay the launches)."""

    def __init__(self, y, x1, x2, v, k, D, pad_mode: str = "linear", workspace=None, stream=None,
                 shared_k: bool = False):
        import torch
        shape = tuple(x1.shape)
        kshape = kernel_shape(shape, pad_mode, shared_k)
        for t, want in ((x1, shape), (x2, shape), (v, shape), (k, kshape), (y, shape)):
            if not t.is_cuda:
                raise ValueError("all tensors must be on the GPU")
            if tuple(t.shape) != want or t.dtype != x1.dtype:
                raise ValueError(f"x1, x2, v, y must share shape and dtype; k must be {kshape} "
                                 f"(pad_mode {pad_mode!r}, shared_k {shared_k})")
            if not t.is_contiguous():
                raise ValueError("tensors must be contiguous")
        if not D.is_cuda or D.dtype != x1.dtype or tuple(D.shape) != (shape[1],) or not D.is_contiguous():
            raise ValueError("D must be a contiguous [C] GPU tensor of the same dtype")
        nd, dims = _dims(shape)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        ws_ptr, ws_bytes = None, 0
        if workspace is not None:
            ws_ptr, ws_bytes = _ptr(workspace), workspace.numel() * workspace.element_size()
        self._fn = lib().hyenand_fftconv_shared_k if shared_k else lib().hyenand_fftconv
        self._args = (_ptr(x1), _ptr(x2), _ptr(v), _ptr(k), _ptr(D), _ptr(y), nd, dims, _mode(pad_mode),
                      _dtype_code(x1.dtype), ws_ptr, ws_bytes, ctypes.c_void_p(stream.cuda_stream))
        self._keep = (y, x1, x2, v, k, D, workspace, stream)  # the buffers outlive the object

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def fftconv_into(y, x1, x2, v, k, D, pad_mode: str = "linear", workspace=None,
                 stream=None, shared_k: bool = False) -> None:
    """y <- x2 * (k conv (x1*v) + D*(x1*v)); all tensors already allocated on
    the GPU.  shared_k: k is [C, L...], one kernel per channel for every sample."""
    Prepared(y, x1, x2, v, k, D, pad_mode, workspace, stream, shared_k)()


class PreparedModalConv:
    """One hyenand_fftconv_modal call with its arguments checked and
    marshalled once (see Prepared): y from x1, x2, v, D and the [C, M] modal
    filter parameters, the filter generated inside the transform kernels."""

    def __init__(self, y, x1, x2, v, log_mag, angle, res_re, res_im, D, pad_mode: str = "linear", workspace=None,
                 stream=None):
        import torch
        shape = tuple(x1.shape)
        for t in (x1, x2, v, y):
            if not t.is_cuda or tuple(t.shape) != shape or t.dtype != x1.dtype or not t.is_contiguous():
                raise ValueError("x1, x2, v, y must be contiguous GPU tensors of one shape and dtype")
        C, M = (int(n) for n in log_mag.shape)
        if C != shape[1]:
            raise ValueError("the modal parameters must be [C, M]")
        for t in (log_mag, angle, res_re, res_im):
            if not t.is_cuda or t.dtype != torch.float32 or tuple(t.shape) != (C, M) or not t.is_contiguous():
                raise ValueError("log_mag, angle, res_re, res_im must be contiguous fp32 [C, M] GPU tensors")
        if not D.is_cuda or D.dtype != x1.dtype or tuple(D.shape) != (C,) or not D.is_contiguous():
            raise ValueError("D must be a contiguous [C] GPU tensor of the same dtype")
        if workspace is None:
            nbytes = workspace_size(shape, pad_mode, x1.dtype)
            workspace = torch.empty(max(1, nbytes), dtype=torch.uint8, device=x1.device)
            _keep_for_stream(stream, workspace)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        nd, dims = _dims(shape)
        self._fn = lib().hyenand_fftconv_modal
        self._args = (_ptr(x1), _ptr(x2), _ptr(v), _ptr(log_mag), _ptr(angle), _ptr(res_re), _ptr(res_im), M,
                      _ptr(D), _ptr(y), nd, dims, _mode(pad_mode), _dtype_code(x1.dtype), _ptr(workspace),
                      workspace.numel() * workspace.element_size(), ctypes.c_void_p(stream.cuda_stream))
        self._keep = (y, x1, x2, v, log_mag, angle, res_re, res_im, D, workspace, stream)

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def fftconv_modal(x1, x2, v, log_mag, angle, res_re, res_im, D, pad_mode: str = "linear", workspace=None,
                  stream=None):
    """y = x2 * (k conv (x1*v) + D*(x1*v)) with k[c] the order-M modal filter
    of channel c (generated inside the transform kernels); torch-allocated y."""
    import torch
    y = torch.empty_like(x1)
    PreparedModalConv(y, x1, x2, v, log_mag, angle, res_re, res_im, D, pad_mode, workspace, stream)()
    _keep_for_stream(stream, y)
    return y


def kernel_spectrum_size(shape, pad_mode: str, dtype) -> int:
    """Bytes of the kept spectra of one kernel per channel for convolutions of
    this [B, C, L1, L2] shape (single-pass 2D plan only)."""
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    _check(lib().hyenand_kernel_spectrum_size(nd, dims, _mode(pad_mode), _dtype_code(dtype), ctypes.byref(out)))
    return int(out.value)


def kernel_spectrum(k, shape, pad_mode: str = "linear", stream=None):
    """Transform a static kernel k [C, L1, L2] once for convolutions of the
    given [B, C, L1, L2] shape; returns the spectra as a torch uint8 tensor
    (layout private to the library) for fftconv_spectrum."""
    import torch
    shape = tuple(shape)
    if not k.is_cuda or not k.is_contiguous() or tuple(k.shape) != (shape[1],) + shape[2:]:
        raise ValueError(f"k must be a contiguous GPU tensor of shape {(shape[1],) + shape[2:]}")
    khat = torch.empty(kernel_spectrum_size(shape, pad_mode, k.dtype), dtype=torch.uint8, device=k.device)
    if stream is None:
        stream = torch.cuda.current_stream(k.device)
    nd, dims = _dims(shape)
    _check(lib().hyenand_kernel_spectrum(_ptr(k), _ptr(khat), khat.numel(), nd, dims, _mode(pad_mode),
                                         _dtype_code(k.dtype), ctypes.c_void_p(stream.cuda_stream)))
    _keep_for_stream(stream, khat)
    return khat


def fftconv_spectrum(x1, x2, v, khat, D, pad_mode: str = "linear", stream=None):
    """y = x2 * (k conv (x1*v) + D*(x1*v)) for the static kernel whose spectra
    kernel_spectrum returned; torch-allocated y."""
    import torch
    shape = tuple(x1.shape)
    for t in (x1, x2, v):
        if not t.is_cuda or tuple(t.shape) != shape or t.dtype != x1.dtype or not t.is_contiguous():
            raise ValueError("x1, x2, v must be contiguous GPU tensors of one shape and dtype")
    if not D.is_cuda or D.dtype != x1.dtype or tuple(D.shape) != (shape[1],) or not D.is_contiguous():
        raise ValueError("D must be a contiguous [C] GPU tensor of the same dtype")
    if not khat.is_cuda or khat.dtype != torch.uint8:
        raise ValueError("khat must be the uint8 GPU tensor kernel_spectrum returned")
    y = torch.empty_like(x1)
    if stream is None:
        stream = torch.cuda.current_stream(x1.device)
    nd, dims = _dims(shape)
    _check(lib().hyenand_fftconv_spectrum(_ptr(x1), _ptr(x2), _ptr(v), _ptr(khat), khat.numel(), _ptr(D), _ptr(y),
                                          nd, dims, _mode(pad_mode), _dtype_code(x1.dtype),
                                          ctypes.c_void_p(stream.cuda_stream)))
    _keep_for_stream(stream, y)
    return y


NOALLOC_SCRATCH_BYTES = 128 << 20


def fftconv_noalloc_into(y, x1, x2, v, k, D, pad_mode: str = "linear", stream=None) -> None:
    """y <- x2 * (k conv (x1*v) + D*(x1*v)) through hyenand_fftconv_noalloc:
    no workspace argument, the library's static device scratch instead
    (calls overlapping on one GPU race on it)."""
    import torch
    shape = tuple(x1.shape)
    for t, want in ((x1, shape), (x2, shape), (v, shape), (k, kernel_shape(shape, pad_mode)), (y, shape)):
        if not t.is_cuda or tuple(t.shape) != want or t.dtype != x1.dtype or not t.is_contiguous():
            raise ValueError("x1, x2, v, y must be contiguous GPU tensors of one shape and dtype; "
                             f"k must be {kernel_shape(shape, pad_mode)}")
    if not D.is_cuda or D.dtype != x1.dtype or tuple(D.shape) != (shape[1],) or not D.is_contiguous():
        raise ValueError("D must be a contiguous [C] GPU tensor of the same dtype")
    if stream is None:
        stream = torch.cuda.current_stream(x1.device)
    nd, dims = _dims(shape)
    _check(lib().hyenand_fftconv_noalloc(_ptr(x1), _ptr(x2), _ptr(v), _ptr(k), _ptr(D), _ptr(y), nd, dims,
                                         _mode(pad_mode), _dtype_code(x1.dtype),
                                         ctypes.c_void_p(stream.cuda_stream)))


def fftconv(x1, x2, v, k, D, pad_mode: str = "linear", workspace=None, stream=None, shared_k: bool = False):
    """Allocate y (and, unless given, the workspace) with torch and run the op."""
    import torch
    y = torch.empty_like(x1)
    own = None
    if workspace is None:
        nbytes = workspace_size(tuple(x1.shape), pad_mode, x1.dtype, shared_k)
        if nbytes:
            workspace = own = torch.empty(nbytes, dtype=torch.uint8, device=x1.device)
    fftconv_into(y, x1, x2, v, k, D, pad_mode, workspace, stream, shared_k)
    _keep_for_stream(stream, y, own)
    return y


def backward_workspace_size(shape, pad_mode: str, dtype) -> int:
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    _check(lib().hyenand_fftconv_backward_workspace_size(nd, dims, _mode(pad_mode), _dtype_code(dtype),
                                                         ctypes.byref(out)))
    return int(out.value)


def backward_workspace_min(shape, pad_mode: str, dtype) -> int:
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    _check(lib().hyenand_fftconv_backward_workspace_min(nd, dims, _mode(pad_mode), _dtype_code(dtype),
                                                        ctypes.byref(out)))
    return int(out.value)


class PreparedBackward:
    """One hyenand_fftconv_backward call with its arguments checked and
    marshalled once (see Prepared)."""

    def __init__(self, gx1, gx2, gv, gk, gD, x1, x2, v, k, D, gy, pad_mode: str = "linear", workspace=None,
                 stream=None):
        import torch
        shape = tuple(x1.shape)
        kshape = kernel_shape(shape, pad_mode)
        for t in (x1, x2, v, k, gy, gx1, gx2, gv, gk):
            want = kshape if (t is k or t is gk) else shape
            if not t.is_cuda or tuple(t.shape) != want or t.dtype != x1.dtype or not t.is_contiguous():
                raise ValueError("x1, x2, v, gy, gx1, gx2, gv must be contiguous GPU tensors of one shape and "
                                 f"dtype; k and gk {kshape} (pad_mode {pad_mode!r})")
        for t in (D, gD):
            if not t.is_cuda or t.dtype != x1.dtype or tuple(t.shape) != (shape[1],) or not t.is_contiguous():
                raise ValueError("D and gD must be contiguous [C] GPU tensors of the same dtype")
        nd, dims = _dims(shape)
        if workspace is None:
            workspace = torch.empty(backward_workspace_size(shape, pad_mode, x1.dtype), dtype=torch.uint8,
                                    device=x1.device)
            _keep_for_stream(stream, workspace)
        if stream is None:
            stream = torch.cuda.current_stream(x1.device)
        self._fn = lib().hyenand_fftconv_backward
        self._args = (_ptr(x1), _ptr(x2), _ptr(v), _ptr(k), _ptr(D), _ptr(gy), _ptr(gx1), _ptr(gx2), _ptr(gv),
                      _ptr(gk), _ptr(gD), nd, dims, _mode(pad_mode), _dtype_code(x1.dtype), _ptr(workspace),
                      workspace.numel() * workspace.element_size(), ctypes.c_void_p(stream.cuda_stream))
        self._keep = (gx1, gx2, gv, gk, gD, x1, x2, v, k, D, gy, workspace, stream)

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def backward_into(gx1, gx2, gv, gk, gD, x1, x2, v, k, D, gy, pad_mode: str = "linear", workspace=None,
                  stream=None) -> None:
    """Gradients of a loss through y for dLoss/dy = gy, written into gx1, gx2,
    gv ([B, C, L...]), gk (shaped like k) and gD ([C]); all tensors already on
    the GPU."""
    PreparedBackward(gx1, gx2, gv, gk, gD, x1, x2, v, k, D, gy, pad_mode, workspace, stream)()


def backward(x1, x2, v, k, D, gy, pad_mode: str = "linear", workspace=None, stream=None):
    """(gx1, gx2, gv, gk, gD) with torch-allocated outputs."""
    import torch
    gx1, gx2, gv = (torch.empty_like(x1) for _ in range(3))
    gk = torch.empty_like(k)
    gD = torch.empty_like(D)
    backward_into(gx1, gx2, gv, gk, gD, x1, x2, v, k, D, gy, pad_mode, workspace, stream)
    _keep_for_stream(stream, gx1, gx2, gv, gk, gD)
    return gx1, gx2, gv, gk, gD


def operator_workspace_size(shape, pad_mode: str, dtype) -> int:
    nd, dims = _dims(shape)
    out = ctypes.c_size_t(0)
    _check(lib().hyenand_operator_workspace_size(nd, dims, _mode(pad_mode), _dtype_code(dtype), ctypes.byref(out)))
    return int(out.value)


class PreparedOperator:
    """One hyenand_operator call with its arguments checked and marshalled
    once (see Prepared)."""

    def __init__(self, y, q, kin, vin, k, D, w_in, w_out, eps_l2: float = 1e-6, eps_rms: float = 1e-6,
                 pad_mode: str = "linear", workspace=None, stream=None):
        import torch
        shape = tuple(q.shape)
        for t, want in ((q, shape), (kin, shape), (vin, shape), (y, shape),
                        (k, kernel_shape(shape, pad_mode))):
            if not t.is_cuda or tuple(t.shape) != want or t.dtype != q.dtype or not t.is_contiguous():
                raise ValueError("q, kin, vin, y must be contiguous GPU tensors of one shape and dtype; "
                                 f"k must be {kernel_shape(shape, pad_mode)}")
        for t in (D, w_in, w_out):
            if not t.is_cuda or t.dtype != q.dtype or tuple(t.shape) != (shape[1],) or not t.is_contiguous():
                raise ValueError("D, w_in and w_out must be contiguous [C] GPU tensors of the same dtype")
        if workspace is None:
            workspace = torch.empty(operator_workspace_size(shape, pad_mode, q.dtype), dtype=torch.uint8,
                                    device=q.device)
            _keep_for_stream(stream, workspace)
        nd, dims = _dims(shape)
        if stream is None:
            stream = torch.cuda.current_stream(q.device)
        self._fn = lib().hyenand_operator
        self._args = (_ptr(q), _ptr(kin), _ptr(vin), _ptr(k), _ptr(D), _ptr(w_in), _ptr(w_out), float(eps_l2),
                      float(eps_rms), _ptr(y), nd, dims, _mode(pad_mode), _dtype_code(q.dtype), _ptr(workspace),
                      workspace.numel() * workspace.element_size(), ctypes.c_void_p(stream.cuda_stream))
        self._keep = (y, q, kin, vin, k, D, w_in, w_out, workspace, stream)

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def operator(q, kin, vin, k, D, w_in, w_out, eps_l2: float = 1e-6, eps_rms: float = 1e-6,
             pad_mode: str = "linear", workspace=None, stream=None):
    """The HyenaND operator, Eq. (HyenaND): RMSNorm(Sigmoid(vin) * (k conv
    RMSNorm(l2(q) * SiLU(kin)) + D * .)) with torch-allocated y."""
    import torch
    y = torch.empty_like(q)
    PreparedOperator(y, q, kin, vin, k, D, w_in, w_out, eps_l2, eps_rms, pad_mode, workspace, stream)()
    _keep_for_stream(stream, y)
    return y


WINDOWS = {"gaussian": 0, "exponential": 1}


class PreparedSynth:
    """One hyenand_kernel_synth call with its arguments checked and
    marshalled once (see Prepared).  k is [B, C, grid...] when gamma and beta
    are given, else [C, grid...]; the grid is kernel_shape(shape, pad_mode)'s."""

    def __init__(self, k, shape, omega0, W1, Wh, Wout, window, gamma=None, beta=None, bias=None,
                 window_kind: str = "gaussian", pad_mode: str = "linear", stream=None):
        import torch
        shape = tuple(int(x) for x in shape)
        nd = len(shape) - 2
        B, C = shape[:2]
        Hf = int(omega0.shape[0])
        J = 1 if Wh is None else int(Wh.shape[0]) + 1
        if window_kind not in WINDOWS:
            raise ValueError(f"window_kind must be one of {sorted(WINDOWS)}")
        want = [(omega0, (Hf,)), (W1, (nd, Hf)), (Wout, (Hf, C)),
                (window, (nd, C) if window_kind == "gaussian" else (C,))]
        if Wh is not None:
            want.append((Wh, (J - 1, Hf, Hf)))
        if bias is not None:
            want.append((bias, (J, Hf)))
        if (gamma is None) != (beta is None):
            raise ValueError("gamma and beta go together")
        if gamma is not None:
            want += [(gamma, (B, J, Hf)), (beta, (B, J, Hf))]
        for t, sh in want:
            if not t.is_cuda or t.dtype != torch.float32 or tuple(t.shape) != sh or not t.is_contiguous():
                raise ValueError(f"parameters must be contiguous fp32 GPU tensors; expected shape {sh}, "
                                 f"got {tuple(t.shape)}")
        kshape = kernel_shape(shape, pad_mode, shared_k=gamma is None)
        if not k.is_cuda or tuple(k.shape) != kshape or not k.is_contiguous():
            raise ValueError(f"k must be a contiguous GPU tensor of shape {kshape}")
        nd_, dims = _dims(shape)
        if stream is None:
            stream = torch.cuda.current_stream(k.device)
        opt = lambda t: None if t is None else _ptr(t)
        self._fn = lib().hyenand_kernel_synth
        self._args = (_ptr(omega0), _ptr(W1), opt(Wh), opt(bias), opt(gamma), opt(beta), _ptr(Wout), _ptr(window),
                      WINDOWS[window_kind], Hf, J, _ptr(k), nd_, dims, _mode(pad_mode), _dtype_code(k.dtype),
                      ctypes.c_void_p(stream.cuda_stream))
        self._keep = (k, omega0, W1, Wh, Wout, window, gamma, beta, bias, stream)

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def kernel_synth(shape, omega0, W1, Wh, Wout, window, gamma=None, beta=None, bias=None,
                 window_kind: str = "gaussian", pad_mode: str = "linear", dtype=None, stream=None):
    """The HyenaND kernel K(x) for a convolution on tensors of `shape`
    ([B, C, L...]), with a torch-allocated k of `dtype` (fp32 by default)."""
    import torch
    dtype = dtype or torch.float32
    kshape = kernel_shape(shape, pad_mode, shared_k=gamma is None)
    k = torch.empty(kshape, dtype=dtype, device=omega0.device)
    PreparedSynth(k, shape, omega0, W1, Wh, Wout, window, gamma, beta, bias, window_kind, pad_mode, stream)()
    _keep_for_stream(stream, k)
    return k


class PreparedModal:
    """One hyenand_modal_filter call with its arguments checked and marshalled
    once (see Prepared): k [C, L] from the [C, M] poles and residues."""

    def __init__(self, k, log_mag, angle, res_re, res_im, stream=None):
        import torch
        C, M = (int(x) for x in log_mag.shape)
        for t in (log_mag, angle, res_re, res_im):
            if not t.is_cuda or t.dtype != torch.float32 or tuple(t.shape) != (C, M) or not t.is_contiguous():
                raise ValueError("log_mag, angle, res_re, res_im must be contiguous fp32 GPU tensors of one [C, M] shape")
        if not k.is_cuda or k.dim() != 2 or k.shape[0] != C or not k.is_contiguous():
            raise ValueError("k must be a contiguous [C, L] GPU tensor")
        if stream is None:
            stream = torch.cuda.current_stream(k.device)
        self._fn = lib().hyenand_modal_filter
        self._args = (_ptr(log_mag), _ptr(angle), _ptr(res_re), _ptr(res_im), M, _ptr(k), C, int(k.shape[1]),
                      _dtype_code(k.dtype), ctypes.c_void_p(stream.cuda_stream))
        self._keep = (k, log_mag, angle, res_re, res_im, stream)

    def __call__(self) -> None:
        status = self._fn(*self._args)
        if status != OK:
            _check(status)


def modal_filter(log_mag, angle, res_re, res_im, L: int, dtype=None, stream=None):
    """k [C, L] = Re sum_m R lambda^t (the modal long filter) with a
    torch-allocated k of `dtype` (fp32 by default)."""
    import torch
    k = torch.empty((log_mag.shape[0], int(L)), dtype=dtype or torch.float32, device=log_mag.device)
    PreparedModal(k, log_mag, angle, res_re, res_im, stream)()
    _keep_for_stream(stream, k)
    return k
