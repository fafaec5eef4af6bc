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
    assert call(L, (1, 1, 16), mode=2) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 1, 16), dtype=5) == H.ERR_INVALID_ARGUMENT
    assert call(L, (1, 1, 12)) == H.ERR_UNSUPPORTED  # not a power of two
    assert b"power of two" in L.hyenand_last_error()


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
    with pytest.raises(H.HyenandError) as e:
        H.workspace_size((1, 1, 3), "linear", "f32")
    assert e.value.status == H.ERR_UNSUPPORTED
