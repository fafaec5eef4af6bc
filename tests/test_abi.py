"""C-ABI library: loads, exports every declared symbol, validates arguments
and sizes workspaces on the host without touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_2607_19378_amd import hyenand as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hyenand.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(H.LIB_PATH):
        from paper_2607_19378_amd import build
        build.build()
    return H.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hyenand_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 7
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(H.EXPORTED)


def test_version_and_strings(L):
    assert L.hyenand_version() >= 100
    assert L.hyenand_status_string(0) == b"ok"
    assert L.hyenand_status_string(3) == b"workspace too small"
    assert L.hyenand_status_string(99) == b"unknown status"


FAKE = 1 << 40  # never dereferenced: every call below fails validation first


def call(L, shape, mode=0, dtype=0, ptrs=None, ws=None, ws_bytes=0, ndim=None):
    nd = len(shape) - 2 if ndim is None else ndim
    dims = (ctypes.c_int64 * len(shape))(*shape)
    p = ptrs or [FAKE + i * (1 << 36) for i in range(6)]
    return L.hyenand_fftconv(*[ctypes.c_void_p(x) for x in p], nd, dims, mode, dtype,
                             ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


def test_invalid_arguments(L):
    assert call(L, (1, 1, 16), ptrs=[0, FAKE, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30),
                                      FAKE + (4 << 30)]) == H.ERR_INVALID_ARGUMENT
    assert b"NULL" in L.hyenand_last_error()
    assert call(L, (1, 1, 16), ndim=0) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 1, 1, 1, 1, 16), ndim=4) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 0, 16)) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 1, 16), mode=3) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 1, 16), dtype=5) == H.ERR_INVALID_ARGUMENT
    # extents that are not powers of two beyond the single-pass kernels run
    # embedded in their transform grid, which needs a workspace
    assert call(L, (1, 1, 10000), mode=1) == H.ERR_WORKSPACE_TOO_SMALL
    assert call(L, (1, 1, 20, 20, 20), mode=1) == H.ERR_WORKSPACE_TOO_SMALL  # 8000 points: no mixed radix
    assert call(L, (1, 1, 300, 300)) == H.ERR_WORKSPACE_TOO_SMALL  # a 1024 x 1024 grid
    assert call(L, (1, 1, 300, 300), ws=FAKE + (40 << 36), ws_bytes=5 * (4 << 20)) == H.ERR_WORKSPACE_TOO_SMALL
    assert call(L, (1, 1, 600, 600)) == H.ERR_UNSUPPORTED  # a 2048-point axis: beyond every plan
    assert b"no plan" in L.hyenand_last_error()


def test_aliasing_rejected(L):
    base = FAKE
    n = 2 * 3 * 64 * 4
    # every call here must fail validation: the pointers are never valid
    assert call(L, (2, 3, 64), ptrs=[base, base + 2 * n, base + 4 * n, base + 6 * n, base + 8 * n,
                                     base + 2 * n + 16]) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps x2" in L.hyenand_last_error()
    assert call(L, (2, 3, 64), ptrs=[base, base + 2 * n, base + 4 * n, base + 6 * n, base + 10 * n,
                                     base + 10 * n - 16]) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps D" in L.hyenand_last_error()


def test_unaligned_pointer_rejected(L):
    base = FAKE
    n = 1 * 2 * 64 * 4
    ptrs = [base + 4, base + 2 * n, base + 4 * n, base + 6 * n, base + 8 * n, base + 10 * n]
    assert call(L, (1, 2, 64), ptrs=ptrs) == H.ERR_INVALID_ARGUMENT
    assert b"x1 is not 16-byte aligned" in L.hyenand_last_error()


def test_workspace_queries_are_host_only():
    assert H.workspace_size((1, 64, 4096), "linear", "f32") == 0
    assert H.plan_name((1, 64, 4096), "linear", "f32") == "fused1d"
    assert H.plan_name((8, 256, 64, 64), "linear", "f32") == "fused2d"
    assert H.plan_name((2, 2, 1, 64), "linear", "bf16") == "fused1d"      # unit axis squeezed
    assert H.plan_name((2, 2, 1, 1, 1), "circular", "f32") == "fused1d"  # single point
    # circular, extents with prime factors 2, 3, 5, 7: mixed-radix transforms
    # on the grid's own points
    assert H.plan_name((2, 4, 14, 14), "circular", "f32") == "mixed2d"
    assert H.plan_name((1, 1, 3), "circular", "f32") == "mixed1d"        # short lines
    assert H.plan_name((1, 1, 300), "circular", "f32") == "mixed1d"      # 300 against 1024 points
    # lines beyond 128 points with more than 5/12 of the power-of-two points:
    # that kernel (500 against 1024; 67: k periodic on 135 against 256)
    assert H.plan_name((1, 1, 500), "circular", "f32") == "fused1d_any"
    assert H.plan_name((1, 1, 67), "circular", "f32") == "fused1d_any"
    assert H.plan_name((1, 2, 5, 6, 7), "circular", "bf16") == "mixed3d"
    assert H.plan_name((1, 2, 63, 64), "circular", "f32") == "mixed2d"    # 4032 points
    assert H.workspace_size((1, 1, 3), "circular", "f32") == 0
    # a circular axis of 13 points: k repeated periodically on 25 points, the
    # 14-point axis on its own; half the points of the 32 x 32 power-of-two grid
    assert H.plan_name((2, 3, 13, 14), "circular", "f32") == "mixed2d"
    # 13 alone: 25 points, a short line
    assert H.plan_name((2, 3, 13), "circular", "f32") == "mixed1d"
    # beyond 4096 mixed-radix points
    assert H.plan_name((1, 1, 10000), "circular", "f32") == "embedded1d"
    assert H.plan_name((1, 1, 65, 65), "circular", "f32") == "embedded2d"   # 135 x 135 mixed, 256 x 256 pow2
    # other extents in the non-circular modes: transforms on the smallest power
    # of two >= 2L - 1, single pass
    assert H.plan_name((1, 1, 3), "linear", "f32") == "mixed1d"
    assert H.plan_name((1, 1, 100), "linear", "f32") == "fused1d_any"      # 200 points against 256
    assert H.plan_name((1, 1, 1000), "linear", "f32") == "fused1d_any"
    # 2D grids up to 2048 mixed-radix points: those kernels (27 x 27, 27 x 32)
    assert H.plan_name((2, 4, 14, 14), "centered", "f32") == "mixed2d"
    assert H.plan_name((2, 4, 14, 16), "linear", "bf16") == "mixed2d"
    assert H.plan_name((2, 4, 24, 40), "linear", "f32") == "fused2d_any"   # 48 x 80 against 64 x 128
    assert H.workspace_size((2, 4, 14, 14), "linear", "f32") == 0
    # beyond the single pass: embedded in the 256 x 256 grid; five embedded
    # tensors of 256^2 floats, then the circular multi-pass plan's workspace
    assert H.plan_name((1, 1, 100, 100), "linear", "f32") == "embedded2d"
    assert H.plan_name((1, 2, 48, 48, 48), "centered", "bf16") == "embedded3d"
    assert H.workspace_min((1, 1, 100, 100), "linear", "f32") == (
        5 * 256 * 256 * 4 + H.workspace_min((1, 1, 256, 256), "circular", "f32"))
    with pytest.raises(H.HyenandError):
        H.plan_name((1, 1, 600, 600), "linear", "f32")


def test_mixed_radix_plan_choice(monkeypatch):
    """HYENAND_PLAN=mixed prefers the mixed-radix kernels wherever they take
    the shape (4096 transform points at most), =nomixed avoids them."""
    monkeypatch.setenv("HYENAND_PLAN", "mixed")
    assert H.plan_name((2, 4, 14, 14), "centered", "f32") == "mixed2d"    # 27 x 27
    assert H.plan_name((2, 4, 1000), "linear", "bf16") == "mixed1d"       # 2000 points
    assert H.plan_name((2, 4, 13), "circular", "f32") == "mixed1d"
    assert H.plan_name((2, 4, 3000), "linear", "f32") == "fused1d_any"    # 6000 > 4096
    assert H.plan_name((2, 4, 64, 64), "linear", "f32") == "fused2d"      # powers of two: unchanged
    monkeypatch.setenv("HYENAND_PLAN", "nomixed")
    assert H.plan_name((2, 4, 14, 14), "circular", "f32") == "fused2d_any"
    assert H.plan_name((1, 2, 5, 6, 7), "circular", "f32") == "embedded3d"


def test_shared_kernel_workspace_query():
    """hyenand_fftconv_shared_k_workspace_size: room for C spectra of P0 x P1/2
    complex fp32 on the single-pass 2D plan with B >= 2, else the plain
    query's size."""
    assert H.workspace_size((8, 256, 64, 64), "linear", "f32", shared_k=True) == 256 * 128 * 64 * 8
    assert H.workspace_size((2, 3, 32, 64), "circular", "bf16", shared_k=True) == 3 * 32 * 32 * 8
    assert H.workspace_size((2, 1, 4, 4), "circular", "f32", shared_k=True) == 256  # rounded up
    for shape, mode in (((1, 256, 64, 64), "linear"),      # one sample: nothing to share
                        ((2, 4, 14, 14), "linear"),        # non-power-of-two grid
                        ((2, 4, 32, 32), "centered"),      # centred kernels
                        ((2, 4, 4096), "linear"),          # 1D
                        ((2, 3, 256, 256), "linear"),      # multi-pass
                        ((2, 3, 1 << 16), "linear")):      # four-step
        assert H.workspace_size(shape, mode, "f32", shared_k=True) == H.workspace_size(shape, mode, "f32")


def bcall(L, shape, mode=0, dtype=0, ptrs=None, ws=FAKE + (40 << 36), ws_bytes=1 << 20):
    nd = len(shape) - 2
    dims = (ctypes.c_int64 * len(shape))(*shape)
    p = ptrs or [FAKE + i * (1 << 36) for i in range(11)]
    return L.hyenand_fftconv_backward(*[ctypes.c_void_p(x) for x in p], nd, dims, mode, dtype,
                                      ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


def test_backward_validation(L):
    p = [FAKE + i * (1 << 36) for i in range(11)]
    q = list(p)
    q[6] = 0  # gx1
    assert bcall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert b"gx1 is NULL" in L.hyenand_last_error()
    q = list(p)
    q[7] = p[0] + 16  # gx2 inside x1
    assert bcall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert b"overlaps" in L.hyenand_last_error()
    q = list(p)
    q[8] = q[9]  # gv == gk
    assert bcall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    q = list(p)
    q[6] = p[6] + 4  # misaligned output
    assert bcall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert bcall(L, (2, 3, 16), ws=None, ws_bytes=0) == H.ERR_WORKSPACE_TOO_SMALL
    assert bcall(L, (2, 3, 16), ws_bytes=16) == H.ERR_WORKSPACE_TOO_SMALL
    assert bcall(L, (1, 2, 1 << 22)) == H.ERR_UNSUPPORTED       # 2^23 transform points
    assert bcall(L, (1, 2, 2048, 4)) == H.ERR_UNSUPPORTED       # 4096 points on an axis of a 2D grid
    # circular and linear, not a power of two: the mixed-radix single pass
    # needs the gD sums only (one float per line, a 256-byte block)
    assert bcall(L, (1, 2, 12), mode=1, ws_bytes=16) == H.ERR_WORKSPACE_TOO_SMALL
    assert bcall(L, (1, 2, 12), ws_bytes=16) == H.ERR_WORKSPACE_TOO_SMALL
    assert H.backward_workspace_min((1, 2, 12), "circular", "f32") == 256
    # beyond the mixed-radix grids (10000 points): embedded in the 32768-point
    # grid, nine embedded tensors of 2 x 32768 floats before the gD sums
    assert bcall(L, (1, 2, 10000), mode=1, ws_bytes=9 * 2 * 32768 * 4) == H.ERR_WORKSPACE_TOO_SMALL
    # multi-pass plans: the gD sums plus one line of three spectra at least
    assert bcall(L, (1, 2, 1 << 20)) == H.ERR_WORKSPACE_TOO_SMALL
    assert bcall(L, (1, 2, 128, 128), mode=1, ws_bytes=4096) == H.ERR_WORKSPACE_TOO_SMALL
    assert b"backward needs at least" in L.hyenand_last_error()


def test_backward_workspace_size(L):
    # single pass: one float per line, in a block rounded to 256 bytes
    assert H.backward_workspace_size((8, 256, 64, 64), "linear", "f32") == 8 * 256 * 4
    assert H.backward_workspace_size((3, 5, 16), "circular", "bf16") == 256
    assert H.backward_workspace_min((3, 5, 16), "circular", "bf16") == 256
    # multi-pass 2D, 512^2 transform grid: 32 sums per line (8 rows per
    # workgroup), then U, K, H of 256 rows x 272 (257 bins padded to 16)
    per = 3 * 256 * 272 * 8
    assert H.backward_workspace_min((1, 3, 256, 256), "linear", "f32") == 512 + per
    assert H.backward_workspace_size((1, 3, 256, 256), "linear", "f32") == 512 + 3 * per
    # four-step 1D, 2^21 points: 128 column tiles per line, three spectra of 2^20
    assert H.backward_workspace_min((1, 2, 1 << 20), "linear", "f32") == 1024 + 3 * (1 << 20) * 8
    with pytest.raises(H.HyenandError):
        H.backward_workspace_size((1, 1, 2048, 2048), "linear", "f32")


def test_centered_mode_queries():
    """pad_mode 2: the transform grid of the linear mode, a workspace that
    holds U (L0 rows) and a centered K (P0 rows) per line; the backward runs
    embedded in the transform grid."""
    assert H.plan_name((8, 256, 64, 64), "centered", "f32") == "fused2d"
    assert H.plan_name((1, 64, 4096), "centered", "f32") == "fused1d"
    assert H.plan_name((1, 4, 1 << 20), "centered", "bf16") == "fourstep1d"
    assert H.plan_name((1, 2, 128, 128, 128), "centered", "bf16") == "multipass3d"
    assert H.workspace_min((1, 3, 256, 256), "centered", "f32") == (256 + 512) * 272 * 8
    assert H.workspace_min((1, 3, 256, 256), "linear", "f32") == 2 * 256 * 272 * 8
    assert H.workspace_min((1, 2, 1 << 20), "centered", "f32") == 2 * (1 << 20) * 8
    # backward: nine tensors embedded in the 2 x 128 transform grid (1 KiB
    # each) and the circular backward's gD sums (one 256-byte block)
    assert H.backward_workspace_size((1, 2, 64), "centered", "f32") == 9 * 1024 + 256
    assert H.backward_workspace_min((1, 2, 64), "centered", "f32") == 9 * 1024 + 256
    assert H.kernel_shape((2, 3, 8, 4), "centered") == (2, 3, 15, 7)
    assert H.kernel_shape((2, 3, 8, 4), "centered", shared_k=True) == (3, 15, 7)


def test_centered_kernel_overlap_uses_double_grid(L):
    """y placed just past the [B, C, L] extent of k but inside its centered
    [B, C, 2L - 1] extent is rejected."""
    shape = (1, 2, 64)
    dims = (ctypes.c_int64 * 3)(*shape)
    p = [FAKE + i * (1 << 36) for i in range(6)]
    p[5] = p[3] + 2 * 64 * 4  # past 2 x 64 floats, inside 2 x 127
    args = [ctypes.c_void_p(x) for x in p]
    assert L.hyenand_fftconv(*args, 1, dims, 2, 0, None, 0, None) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps k" in L.hyenand_last_error()
    assert L.hyenand_fftconv(*args, 1, dims, 3, 0, None, 0, None) == H.ERR_INVALID_ARGUMENT
    assert b"pad_mode" in L.hyenand_last_error()


def ocall(L, shape, mode=0, dtype=0, ptrs=None, eps=(1e-6, 1e-6), ws=FAKE + (40 << 36), ws_bytes=1 << 20):
    nd = len(shape) - 2
    dims = (ctypes.c_int64 * len(shape))(*shape)
    p = ptrs or [FAKE + i * (1 << 36) for i in range(8)]
    a = [ctypes.c_void_p(x) for x in p]
    return L.hyenand_operator(*a[:7], ctypes.c_float(eps[0]), ctypes.c_float(eps[1]), a[7], nd, dims, mode, dtype,
                              ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


def test_operator_validation(L):
    """hyenand_operator rejects bad arguments before launching anything (every
    call here stops at validation)."""
    p = [FAKE + i * (1 << 36) for i in range(8)]
    for i in range(8):
        q = list(p)
        q[i] = 0
        assert ocall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
        assert b"is NULL" in L.hyenand_last_error()
    assert ocall(L, (2, 3, 16), eps=(-1.0, 1e-6)) == H.ERR_INVALID_ARGUMENT
    assert ocall(L, (2, 3, 16), eps=(1e-6, float("nan"))) == H.ERR_INVALID_ARGUMENT
    q = list(p)
    q[7] = p[2] + 32  # y inside vin
    assert ocall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps vin" in L.hyenand_last_error()
    q = list(p)
    q[5] = p[5] + 2  # w_in not aligned to a float
    assert ocall(L, (2, 3, 16), ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert ocall(L, (2, 3, 16), ws=None, ws_bytes=0) == H.ERR_WORKSPACE_TOO_SMALL
    assert ocall(L, (2, 3, 16), ws_bytes=64) == H.ERR_WORKSPACE_TOO_SMALL  # 2 x 16 scales need 256 bytes
    assert ocall(L, (1, 1 << 15, 2)) == H.ERR_UNSUPPORTED  # more channels than the output norm's tile
    assert ocall(L, (1, 2, 10000), mode=1) == H.ERR_UNSUPPORTED  # circular, no single-pass plan
    assert ocall(L, (1, 2, 100, 100)) == H.ERR_UNSUPPORTED  # embedded shapes: not in the operator


def test_operator_workspace_size(L):
    # scales [B, prod L] floats in a 256-byte block, then the convolution's workspace
    assert H.operator_workspace_size((8, 256, 64, 64), "linear", "f32") == 8 * 64 * 64 * 4
    assert H.operator_workspace_size((1, 3, 256, 256), "linear", "f32") == (
        256 * 256 * 4 + H.workspace_size((1, 3, 256, 256), "linear", "f32"))
    assert H.operator_workspace_size((2, 2, 4), "circular", "bf16") == 256


def test_shared_kernel_validation(L):
    """hyenand_fftconv_shared_k takes k as [C, L...]: y inside that smaller
    region still overlaps k; null pointers are rejected."""
    shape = (4, 3, 64)
    dims = (ctypes.c_int64 * 3)(*shape)
    p = [FAKE + i * (1 << 36) for i in range(6)]
    p[5] = p[3] + 3 * 64 * 4 - 16  # y starts 16 bytes before the end of k[C, L]
    args = [ctypes.c_void_p(x) for x in p]
    assert L.hyenand_fftconv_shared_k(*args, 1, dims, 0, 0, None, 0, None) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps k" in L.hyenand_last_error()
    q = [ctypes.c_void_p(x) for x in p[:3]] + [None] + [ctypes.c_void_p(x) for x in p[4:]]
    assert L.hyenand_fftconv_shared_k(*q, 1, dims, 0, 0, None, 0, None) == H.ERR_INVALID_ARGUMENT


def test_kernel_spectrum_validation(L):
    """Kept kernel spectra: sizes on the single-pass 2D plan (any B, since only
    C, the grid and the mode fix them), UNSUPPORTED elsewhere, and argument
    checks that fail before anything launches (fake pointers)."""
    assert H.kernel_spectrum_size((8, 256, 64, 64), "linear", "f32") == 256 * 128 * 64 * 8
    assert H.kernel_spectrum_size((1, 3, 32, 64), "circular", "bf16") == 3 * 32 * 32 * 8
    for shape, mode in (((2, 4, 4096), "linear"), ((2, 4, 32, 32), "centered"), ((2, 4, 14, 14), "linear"),
                        ((1, 3, 256, 256), "linear"), ((1, 2, 8, 8, 8), "circular")):
        with pytest.raises(H.HyenandError) as e:
            H.kernel_spectrum_size(shape, mode, "f32")
        assert e.value.status == H.ERR_UNSUPPORTED
    shape = (2, 3, 32, 32)
    dims = (ctypes.c_int64 * 4)(*shape)
    need = 3 * 64 * 32 * 8  # C x P0 x P1/2 complex fp32, P = 2 L (linear)
    k, khat = FAKE, FAKE + (1 << 36)
    vp = ctypes.c_void_p
    assert L.hyenand_kernel_spectrum(vp(k), vp(khat), need - 1, 2, dims, 0, 0, None) == H.ERR_WORKSPACE_TOO_SMALL
    assert L.hyenand_kernel_spectrum(None, vp(khat), need, 2, dims, 0, 0, None) == H.ERR_INVALID_ARGUMENT
    assert L.hyenand_kernel_spectrum(vp(k), vp(khat + 8), need, 2, dims, 0, 0, None) == H.ERR_INVALID_ARGUMENT
    assert L.hyenand_kernel_spectrum(vp(k), vp(k + 64), need, 2, dims, 0, 0, None) == H.ERR_INVALID_ARGUMENT
    assert b"khat overlaps k" in L.hyenand_last_error()
    d3 = (ctypes.c_int64 * 5)(2, 3, 8, 8, 8)
    assert L.hyenand_kernel_spectrum(vp(k), vp(khat), 1 << 30, 3, d3, 1, 0, None) == H.ERR_UNSUPPORTED
    p = [FAKE + i * (1 << 36) for i in range(6)]  # x1, x2, v, khat, D, y

    def conv(ptrs, nbytes=need, d=dims, nd=2, mode=0):
        return L.hyenand_fftconv_spectrum(*[vp(x) if x else None for x in ptrs[:4]], nbytes,
                                          *[vp(x) if x else None for x in ptrs[4:]], nd, d, mode, 0, None)
    assert conv(p, need - 256) == H.ERR_WORKSPACE_TOO_SMALL
    for i in range(6):
        q = list(p)
        q[i] = 0
        assert conv(q) == H.ERR_INVALID_ARGUMENT
    q = list(p)
    q[5] = p[3] + 16  # y over khat
    assert conv(q) == H.ERR_INVALID_ARGUMENT
    assert b"y overlaps khat" in L.hyenand_last_error()
    q = list(p)
    q[0] += 4
    assert conv(q) == H.ERR_INVALID_ARGUMENT
    assert conv(p, mode=2) == H.ERR_UNSUPPORTED


def synth(L, shape=(2, 4, 16), hidden=32, layers=1, wkind=0, mode=0, dtype=0, ptrs=None, k=None):
    """hyenand_kernel_synth with fake pointers: every call here must fail
    validation (nothing may launch)."""
    dims = (ctypes.c_int64 * len(shape))(*shape)
    p = ptrs or [FAKE + i * (1 << 36) for i in range(8)]
    kp = FAKE + (9 << 36) if k is None else k
    return L.hyenand_kernel_synth(*[ctypes.c_void_p(x) if x else None for x in p], wkind, hidden, layers,
                                  ctypes.c_void_p(kp), len(shape) - 2, dims, mode, dtype, None)


def test_synth_validation(L):
    base = [FAKE + i * (1 << 36) for i in range(8)]
    assert synth(L, hidden=48) == H.ERR_UNSUPPORTED
    assert b"hidden width" in L.hyenand_last_error()
    assert synth(L, layers=0) == H.ERR_UNSUPPORTED
    assert synth(L, layers=17) == H.ERR_UNSUPPORTED
    assert synth(L, wkind=2) == H.ERR_INVALID_ARGUMENT
    assert synth(L, mode=3) == H.ERR_INVALID_ARGUMENT
    assert synth(L, dtype=4) == H.ERR_INVALID_ARGUMENT
    assert synth(L, shape=(2, 0, 16)) == H.ERR_INVALID_ARGUMENT
    assert synth(L, shape=(2, 4, 16), ptrs=[0] + base[1:]) == H.ERR_INVALID_ARGUMENT  # omega0 NULL
    assert synth(L, layers=2, ptrs=base[:2] + [0] + base[3:]) == H.ERR_INVALID_ARGUMENT  # Wh NULL
    assert synth(L, ptrs=base[:5] + [0] + base[6:]) == H.ERR_INVALID_ARGUMENT  # gamma without beta
    assert b"gamma and beta" in L.hyenand_last_error()
    assert synth(L, ptrs=base[:1] + [base[1] + 2] + base[2:]) == H.ERR_INVALID_ARGUMENT  # W1 misaligned
    assert b"W1" in L.hyenand_last_error()
    assert synth(L, layers=2, ptrs=base[:2] + [base[2] + 4] + base[3:]) == H.ERR_INVALID_ARGUMENT  # Wh: 16 bytes
    assert b"Wh is not 16-byte aligned" in L.hyenand_last_error()
    assert synth(L, dtype=1, k=FAKE + (9 << 36) + 1) == H.ERR_INVALID_ARGUMENT  # bf16 k misaligned
    # k (2 x 4 x 16 fp32 = 512 bytes) running into Wout
    assert synth(L, k=base[6] - 256) == H.ERR_INVALID_ARGUMENT
    assert b"k overlaps Wout" in L.hyenand_last_error()
    # without FiLM k is [C, grid]: 4 x 16 fp32 = 256 bytes, so starting 252 bytes below Wout overlaps it
    nofilm = base[:4] + [0, 0] + base[6:]
    assert synth(L, ptrs=nofilm, k=base[6] - 252) == H.ERR_INVALID_ARGUMENT
    # centered: the grid has 2L - 1 = 31 points, so 4 x 31 floats reach Wout from 496 bytes below it
    assert synth(L, ptrs=nofilm, mode=2, k=base[6] - 492) == H.ERR_INVALID_ARGUMENT


def modal(L, C=4, Lt=64, order=16, dtype=0, ptrs=None, k=None):
    """hyenand_modal_filter with fake pointers: every call here must fail
    validation (nothing may launch)."""
    p = ptrs or [FAKE + i * (1 << 36) for i in range(4)]
    kp = FAKE + (9 << 36) if k is None else k
    return L.hyenand_modal_filter(*[ctypes.c_void_p(x) if x else None for x in p], order, ctypes.c_void_p(kp) if kp else None,
                                  C, Lt, dtype, None)


def test_modal_validation(L):
    base = [FAKE + i * (1 << 36) for i in range(4)]
    assert modal(L, C=0) == H.ERR_INVALID_ARGUMENT
    assert modal(L, Lt=0) == H.ERR_INVALID_ARGUMENT
    assert modal(L, order=0) == H.ERR_INVALID_ARGUMENT
    assert modal(L, order=257) == H.ERR_UNSUPPORTED
    assert modal(L, Lt=(1 << 29) + 1) == H.ERR_UNSUPPORTED
    assert modal(L, dtype=3) == H.ERR_INVALID_ARGUMENT
    assert modal(L, ptrs=[base[0], 0, base[2], base[3]]) == H.ERR_INVALID_ARGUMENT
    assert b"angle is NULL" in L.hyenand_last_error()
    assert modal(L, k=0) == H.ERR_INVALID_ARGUMENT
    assert modal(L, ptrs=[base[0] + 2] + base[1:]) == H.ERR_INVALID_ARGUMENT
    assert modal(L, dtype=1, k=FAKE + (9 << 36) + 1) == H.ERR_INVALID_ARGUMENT
    # k (4 x 64 fp32 = 1024 bytes) running into res_im
    assert modal(L, k=base[3] - 1020) == H.ERR_INVALID_ARGUMENT
    assert b"k overlaps res_im" in L.hyenand_last_error()


def test_embedded_backward_validation(L):
    """Centred and other-extent backward: k and gk take the kernel's shape in
    the overlap checks, and every call here fails validation."""
    p = [FAKE + i * (1 << 36) for i in range(11)]
    # centred [1, 2, 8]: gk is 2 x 15 floats = 120 bytes; placed 112 bytes
    # below gD's start it runs into gD (a data-sized gk, 64 bytes, would not)
    q = list(p)
    q[9] = p[10] - 112
    assert bcall(L, (1, 2, 8), mode=2, ptrs=q) == H.ERR_INVALID_ARGUMENT
    assert b"gD overlaps gk" in L.hyenand_last_error() or b"gk overlaps" in L.hyenand_last_error()
    assert bcall(L, (1, 2, 8), mode=2, ws_bytes=64) == H.ERR_WORKSPACE_TOO_SMALL
    assert bcall(L, (1, 2, 5, 7), mode=0, ws_bytes=64) == H.ERR_WORKSPACE_TOO_SMALL


def test_line_count_bounded(L):
    """B * C beyond what one launch of one workgroup per line can hold is
    refused on the host (no index or grid overflow on the GPU)."""
    assert call(L, (1 << 31, 1, 2)) == H.ERR_UNSUPPORTED
    assert b"lines" in L.hyenand_last_error()
    assert call(L, (1, 1 << 31, 2)) == H.ERR_UNSUPPORTED
    assert call(L, (1 << 11, 1 << 11, 2)) == H.ERR_UNSUPPORTED  # exactly 2^22 lines
    with pytest.raises(H.HyenandError):
        H.workspace_size((1 << 12, 1 << 10, 4), "linear", "f32")
    assert H.plan_name(((1 << 22) - 1, 1, 4), "linear", "f32") == "fused1d"


def test_embedded_grid_bounded():
    """An embedded plan whose grid tensor would exceed 2^31 elements has no
    plan (its elementwise launches would exceed 2^32 work-items)."""
    # 300 x 300 runs on a 1024 x 1024 grid: 2048 lines hold exactly 2^31
    # elements, 2049 one line more
    assert H.plan_name((1, 2048, 300, 300), "linear", "f32") == "embedded2d"
    with pytest.raises(H.HyenandError) as e:
        H.plan_name((1, 2049, 300, 300), "linear", "f32")
    assert e.value.status == H.ERR_UNSUPPORTED


def test_noalloc_rejects_beyond_its_scratch(L):
    """The no-allocation entry point refuses, on the host, shapes whose least
    workspace exceeds its static scratch (128 MiB per GPU)."""
    dims = (ctypes.c_int64 * 5)(1, 1, 256, 256, 256)
    p = [ctypes.c_void_p(FAKE + i * (1 << 36)) for i in range(6)]
    assert L.hyenand_fftconv_noalloc(*p, 3, dims, 0, 0, None) == H.ERR_UNSUPPORTED
    assert b"scratch" in L.hyenand_last_error()
    assert H.workspace_min((1, 1, 128, 128, 128), "linear", "bf16") <= H.NOALLOC_SCRATCH_BYTES
    assert H.workspace_min((1, 1, 1 << 20), "linear", "bf16") <= H.NOALLOC_SCRATCH_BYTES
    dims = (ctypes.c_int64 * 3)(1, 0, 64)
    assert L.hyenand_fftconv_noalloc(*p, 1, dims, 0, 0, None) == H.ERR_INVALID_ARGUMENT


def test_fused_modal_validation(L):
    """hyenand_fftconv_modal refuses, on the host, shapes beyond the
    four-step plan, orders above 32 and missing parameters."""
    p = [ctypes.c_void_p(FAKE + i * (1 << 36)) for i in range(10)]

    def call_modal(shape, mode=0, order=16, params=None):
        dims = (ctypes.c_int64 * len(shape))(*shape)
        pr = params if params is not None else p[3:7]
        return L.hyenand_fftconv_modal(p[0], p[1], p[2], *pr, order, p[7], p[8], len(shape) - 2, dims, mode, 0,
                                       p[9], 1 << 30, None)
    assert call_modal((1, 4, 4096)) == H.ERR_UNSUPPORTED      # single-pass shape
    assert b"four-step" in L.hyenand_last_error()
    assert call_modal((1, 4, 64, 64)) == H.ERR_UNSUPPORTED    # 2D
    assert call_modal((1, 4, 1 << 20), mode=2) == H.ERR_UNSUPPORTED  # centred
    assert call_modal((1, 4, 1 << 20), order=33) == H.ERR_UNSUPPORTED
    assert call_modal((1, 4, 1 << 20), order=0) == H.ERR_UNSUPPORTED
    assert call_modal((1, 4, 1 << 20), params=[p[3], None, p[5], p[6]]) == H.ERR_INVALID_ARGUMENT
    assert b"angle" in L.hyenand_last_error()
