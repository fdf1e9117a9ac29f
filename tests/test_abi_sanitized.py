"""The C-ABI host tests (tests/test_abi.py: argument validation, the fold
generator, workspace sizing, host-side refusals of the single-step entry
points) run against a build of the library with AddressSanitizer and
UndefinedBehaviorSanitizer on its host code. No GPU is involved: every call
in those tests returns before the library touches a device."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs the ROCm compiler")
def test_abi_host_paths_under_asan_and_ubsan():
    from paper_2606_06742_amd import build_sanitized as bs
    lib = bs.build()
    env = dict(os.environ)
    env["KMPATH_LIB"] = lib
    env["LD_PRELOAD"] = bs.runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py"), "-k", "not refuses_missing"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in out and "runtime error" not in out
