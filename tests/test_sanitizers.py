"""The C-ABI host code (argument checks, planner, handle and workspace
management) under AddressSanitizer and UndefinedBehaviorSanitizer, on the
CPU: the ABI tests run again in a child Python that loads libqlin_asan.so
(the same library with qlin.cpp and attn_abi.cpp instrumented, linked by
the build) with the sanitizer runtimes preloaded.  Any invalid access or
undefined behaviour in the checks they exercise aborts the child."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_ASAN = os.path.join(ROOT, "paper_2607_04244_amd", "libqlin_asan.so")


def _runtime(name):
    try:
        p = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True, timeout=30).stdout.strip()
    except (OSError, subprocess.SubprocessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_abi_checks_under_address_and_undefined_behaviour_sanitizers():
    if not os.path.exists(LIB_ASAN):
        pytest.skip("libqlin_asan.so is built by __graft_entry__.build()")
    rt = [_runtime("libasan.so"), _runtime("libubsan.so")]
    if None in rt:
        pytest.skip("g++ sanitizer runtimes not found")
    env = dict(os.environ, QLIN_LIB=LIB_ASAN, LD_PRELOAD=" ".join(rt),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi.py")], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout
