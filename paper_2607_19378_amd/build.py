"""Build libhyenand.so (HIP, gfx950) in-tree.

    python -m paper_2607_19378_amd.build
    python -m paper_2607_19378_amd.build --sanitize

compiles every csrc/*.hip translation unit with hipcc for gfx950 and links
them into paper_2607_19378_amd/libhyenand.so.  Always rebuilds.

--sanitize builds CPU-checking copies instead, under _build/sanitize/: the
library with its host code (argument validation, plan choice, workspace
arithmetic, chunking) under AddressSanitizer and UndefinedBehaviorSanitizer
(device code is built as usual), and the C oracle under both.  The CPU test
suite then runs on them with the sanitizer runtime preloaded:

    LD_PRELOAD=<clang's libclang_rt.asan-x86_64.so> ASAN_OPTIONS=detect_leaks=0 \
    HYENAND_LIBRARY=_build/sanitize/libhyenand.so \
    HYENAND_ORACLE_LIBRARY=_build/sanitize/liboracle.so \
    python -m pytest tests -m "not gpu"

(the command with the runtime's path filled in is printed at the end).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libhyenand.so")
BUILD_DIR = os.path.join(os.path.dirname(PKG), "_build", "hyenand")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 VALU forms are disabled on purpose: hipcc would otherwise emit
# v_pk_{add,mul,fma}_f32 from plain float code.  -fno-signed-zeros lets the
# compiler drop x + 0 where a transform's input is a compile-time zero (the
# zero-padded half of every linear-mode first pass); it changes no value, at
# most the sign of an exact zero.
FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall", "-fno-signed-zeros",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-pass-failed", "-I", os.path.join(os.path.dirname(PKG), "include")]


def source_hash() -> str:
    """Hash of every HIP source and header of the library.  Counter records
    under profiles/ carry it: they only describe the kernels they were taken on."""
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.hpp"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


SAN_DIR = os.path.join(os.path.dirname(PKG), "_build", "sanitize")
# host code only: each sanitizer flag goes to the host compilation
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
CLANG = os.environ.get("HYENAND_CLANG", "/opt/rocm/llvm/bin/clang")


def _compile(src: str, sanitize: bool = False) -> str:
    out_dir = SAN_DIR if sanitize else BUILD_DIR
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + (SAN_HOST if sanitize else []) + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in (r.stderr or "").splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def build(jobs: int | None = None, sanitize: bool = False) -> str:
    out_dir = SAN_DIR if sanitize else BUILD_DIR
    out = os.path.join(SAN_DIR, "libhyenand.so") if sanitize else OUT
    os.makedirs(out_dir, exist_ok=True)
    subprocess.run([sys.executable, os.path.join(CSRC, "gen_twiddles.py")], check=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda f: _compile(f, sanitize), srcs))
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_sanitized_oracle() -> str:
    """The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer,
    with the same compiler as the library's host code (one sanitizer runtime
    serves both)."""
    src = os.path.join(os.path.dirname(PKG), "oracle", "oracle.c")
    out = os.path.join(SAN_DIR, "liboracle.so")
    os.makedirs(SAN_DIR, exist_ok=True)
    subprocess.run([CLANG, "-O1", "-g", "-std=c99", "-fPIC", "-shared", "-Wall", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-o", out, src, "-lm", "-lpthread"],
                   check=True)
    return out


if __name__ == "__main__":
    if "--sanitize" in sys.argv[1:]:
        lib = build(sanitize=True)
        orc = build_sanitized_oracle()
        rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                            text=True, check=True).stdout.strip()
        print(lib)
        print(orc)
        print(f"LD_PRELOAD={rt} ASAN_OPTIONS=detect_leaks=0 HYENAND_LIBRARY={lib} HYENAND_ORACLE_LIBRARY={orc} "
              f"python -m pytest tests -m 'not gpu'")
    else:
        print(build())
