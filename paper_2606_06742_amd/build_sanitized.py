"""Host-sanitized build of the kmpath library (AddressSanitizer and
UndefinedBehaviorSanitizer on the host code only; the device code is built
as usual). Used by the CPU test that runs the C-ABI host tests (argument
validation, fold generator, workspace sizing) against it.

Usage: python -m paper_2606_06742_amd.build_sanitized  -> prints the path
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

from .build import CSRC, INCLUDE, ROOT, _jobs, hipcc, sources

OUT_DIR = os.path.join(ROOT, "_build", "sanitized")
LIB = os.path.join(OUT_DIR, "libkmpath_sanitized.so")
# every sanitizer flag applies to the host pass only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument"]


def runtime() -> str:
    """The compiler's AddressSanitizer runtime (to preload into python)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin",
                         "clang++")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang++"
    return subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                          capture_output=True, text=True, check=True).stdout.strip()


def build() -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    cc = hipcc()

    def one(src):
        obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
        cmd = [cc, *FLAGS, *HOST_SAN, "-I", INCLUDE, "-I", CSRC, "-x", "hip", "-c", src, "-o", obj]
        return obj, subprocess.run(cmd, capture_output=True, text=True)

    with ThreadPoolExecutor(max_workers=_jobs()) as ex:
        res = list(ex.map(one, sources()))
    bad = [r for _, r in res if r.returncode != 0]
    for r in bad:
        sys.stderr.write(r.stdout + r.stderr)
    if bad:
        raise RuntimeError("sanitized build failed")
    link = [cc, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
            "-Xarch_host", "-fsanitize=undefined", *[o for o, _ in res], "-o", LIB]
    r = subprocess.run(link, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("sanitized link failed")
    return LIB


if __name__ == "__main__":
    print(build())
