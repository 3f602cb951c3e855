"""The host-side argument checks of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer:
tests/test_abi_cpu.py runs in a child process against the host-sanitized build of the library
(iso_abi.cpp instrumented, kernels not; paper_2607_19331_amd/build.py) with the sanitizer runtime
preloaded.  Any invalid access or undefined operation aborts the child.  No GPU is used: every
call in those tests is rejected on the host before anything is queued."""
import os
import subprocess
import sys

import pytest

from paper_2607_19331_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_under_host_sanitizers():
    rt = B.asan_runtime()
    if rt is None or not os.path.exists(B.SANITIZED_LIB):
        pytest.skip("no host-sanitized build (the toolchain has no AddressSanitizer runtime)")
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": rt,
        "ISO_LIB_PATH": B.SANITIZED_LIB,
        # the interpreter itself is not instrumented and keeps memory until exit
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout
