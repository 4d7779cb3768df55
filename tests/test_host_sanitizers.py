"""The C-ABI host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Builds api.hip's host code and the kernel packer with the host compiler,
-fsanitize=address,undefined and no recovery, linked against stand-in
launchers (no device code), and runs the host-side test files against that
library in a child process: the library and packer tests, plus
host_san_cases.py, which drives every entry point and whole composite chains
with fake device pointers.  Any sanitizer report fails the child.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CXX = os.environ.get("CXX", shutil.which("g++") or "c++")


def _runtime(name):
    path = subprocess.run([CXX, f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"), reason="needs the HIP headers")
def test_host_code_is_clean_under_asan_and_ubsan():
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("the host compiler has no AddressSanitizer runtime")
    sys.path.insert(0, ROOT)
    from paper_2408_03505_amd import build
    lib = build.build_host_sanitized(verbose=False)
    env = dict(os.environ)
    env.update(OPTIMUS_ENC_LIB=lib, LD_PRELOAD=asan,
               # the interpreter and torch are not instrumented: their own
               # allocations are neither leak-checked nor matched
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               CUDA_VISIBLE_DEVICES="", HIP_VISIBLE_DEVICES="")
    files = ["tests/test_library_cpu.py", "tests/test_schedule_cpu.py", "tests/host_san_cases.py"]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *files],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
    assert " passed" in r.stdout, tail
