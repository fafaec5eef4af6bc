"""A HIP error that earlier work left pending on the calling thread (here: a
failed hipSetDevice on an ordinal that does not exist, which touches no
device) is not reported as the library call's own: every entry point clears
it before it launches and checks each of its launches after."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _runtimes():
    paths = sorted({line.split()[-1] for line in open("/proc/self/maps").read().splitlines()
                    if "libamdhip64" in line and line.split()[-1].startswith("/")})
    assert paths, "no HIP runtime mapped"
    return [ctypes.CDLL(p) for p in paths]


@pytest.mark.parametrize("shape,shared_k", [((2, 3, 32, 32), True), ((2, 3, 4096), False),
                                            ((1, 2, 256, 256), False)])
def test_pending_error_of_earlier_work_is_not_reported(shape, shared_k):
    import torch
    from paper_2607_19378_amd import hyenand as H
    from gpu_util import log
    log(f"pending-error case {shape} shared_k={shared_k}")
    H.lib()
    rng = np.random.default_rng(3)
    x1, x2, v = (torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).cuda() for _ in range(3))
    kshape = (shape[1],) + shape[2:] if shared_k else shape
    k = torch.from_numpy(rng.standard_normal(kshape).astype(np.float32)).cuda()
    D = torch.from_numpy(rng.standard_normal(shape[1]).astype(np.float32)).cuda()
    ref = H.fftconv(x1, x2, v, k, D, shared_k=shared_k)
    torch.cuda.synchronize()
    for rt in _runtimes():
        assert rt.hipSetDevice(ctypes.c_int(4096)) != 0  # leaves an error pending
    y = H.fftconv(x1, x2, v, k, D, shared_k=shared_k)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)


def test_library_loaded_before_torch_touches_the_gpu():
    """A fresh process whose first use of the binding is a host-only query
    (which loads the library) and whose first GPU work comes after it: the
    library and torch must share one HIP runtime, or the library's launches
    find no device."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "from paper_2607_19378_amd import hyenand as H\n"
        "assert H.plan_name((2, 3, 32, 32), 'linear', 'f32') == 'fused2d'\n"
        "import torch\n"
        "x = torch.ones((2, 3, 32, 32), device='cuda')\n"
        "k = torch.ones((3, 32, 32), device='cuda')\n"
        "D = torch.zeros(3, device='cuda')\n"
        "y = H.fftconv(x, x, x, k, D, shared_k=True)\n"
        "torch.cuda.synchronize()\n"
        "assert abs(float(y[0, 0, 0, 0]) - 1.0) < 1e-4 and abs(float(y[1, 2, 31, 31]) - 1024.0) < 1e-2\n"
        "print('ok')\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, PYTHONPATH=root))
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr
