"""The host runtime (C ABI, planner, generator, calibration reader) under
AddressSanitizer and UndefinedBehaviorSanitizer: builds the sanitizer variant of
the library (host code instrumented, device code as usual) and runs the
host-only library tests against it in a child process, failing on the first
report.  No GPU is used."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"
HOST_TESTS = ["tests/test_host_abi.py", "tests/test_host_crossgram.py", "tests/test_host_curvature.py",
              "tests/test_host_mask.py"]


@pytest.mark.timeout(900)
def test_host_runtime_under_asan_ubsan():
    if os.environ.get("DATTRI_LIB"):
        pytest.skip("already running against another build of the library")
    if not (os.path.exists("/opt/rocm/bin/hipcc") and os.path.exists(CLANG)):
        pytest.skip("hipcc / clang not available")
    from paper_2609_38767_amd import build
    lib = build.build(sanitize=True)
    rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    assert os.path.exists(rt), rt
    env = dict(os.environ, DATTRI_LIB=lib, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        *HOST_TESTS], cwd=ROOT, env=env, capture_output=True, text=True)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert " passed" in r.stdout, tail
