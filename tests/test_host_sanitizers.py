"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The library's host side -- the C ABI's argument, config and shape checks,
the weight layout, the micro-batcher, the deficit router, the co-location
limits and the allocation-free entry point's capacity refusal -- is built a
second time with ASan + UBSan on its host pass (paper_2609_31551_amd/build.py,
sanitize=True; device code unchanged), and the host-only test files run
against that build in a child process with the sanitizer runtime preloaded.
Any sanitizer report aborts the child, so the test fails.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HOST_TESTS = ["tests/test_abi.py", "tests/test_batcher.py", "tests/test_router.py", "tests/test_colocate.py",
              "tests/test_zz_no_alloc.py"]


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(_asan_runtime() is None or not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc and the clang ASan runtime")
def test_host_code_is_clean_under_asan_and_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2609_31551_amd import build
    lib = build.build(verbose=False, sanitize=True)
    env = dict(os.environ, LD_PRELOAD=_asan_runtime(), EAS_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    probe = ("import ctypes; from paper_2609_31551_amd import eas; "
             "assert eas.LIB_PATH.endswith('libeas_asan.so'); "
             "ctypes.CDLL(None).__asan_report_load8; ctypes.CDLL(None).__ubsan_handle_add_overflow; print('ok')")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider"] + HOST_TESTS,
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    print(r.stdout[-1500:])
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert " passed" in r.stdout and "failed" not in r.stdout
