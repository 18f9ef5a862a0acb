"""The C ABI's host code (api.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: tests/sanitize/abi_host_check.c drives
its argument, overlap, ordering, codec, record, staging, stream, device,
capture and allocation-failure paths through a host-memory stand-in for the
HIP runtime (tests/sanitize/hip_double.cpp), and every allocation must be
freed by the end (LeakSanitizer)."""
import os
import shutil
import subprocess
import sys
from pathlib import Path

import pytest

HERE = Path(__file__).resolve().parent


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc and g++")
def test_abi_host_code_is_clean_under_asan_and_ubsan():
    sys.path.insert(0, str(HERE / "sanitize"))
    try:
        import build as san_build
        exe = san_build.build()
    finally:
        sys.path.pop(0)
    # verify_asan_link_order=0: the environment may preload a library of its
    # own ahead of the sanitizer runtime
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:detect_stack_use_after_return=1:"
                                        "verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
    assert "0 failed" in r.stdout
