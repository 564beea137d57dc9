"""The host-side ABI checks (tests/test_abi.py: configuration and argument
validation, workspace layout, binding, the error paths of every call) run
again against a build of the library whose host code is instrumented with
AddressSanitizer: no invalid host memory access on those paths.  CPU only;
the sanitizer runtime is clang's, preloaded into the child interpreter."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    found = sorted(glob.glob(
        "/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


@pytest.mark.slow
def test_abi_checks_under_address_sanitizer():
    runtime = _asan_runtime()
    if runtime is None:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    from paper_2605_07243_amd import build
    lib = build.build_host_asan()
    env = dict(os.environ, LD_PRELOAD=runtime, SPECBLOCK_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1")
    r = subprocess.run(
        [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
         "-m", "not gpu", os.path.join(ROOT, "tests", "test_abi.py")],
        env=env, capture_output=True, text=True, timeout=900, cwd=ROOT)
    log = r.stdout + r.stderr
    assert "AddressSanitizer" not in log, log[-4000:]
    assert r.returncode == 0, log[-4000:]
    assert " passed" in r.stdout, log[-2000:]
