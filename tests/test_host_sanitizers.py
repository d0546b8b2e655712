"""The host-only translation unit (descriptor checks, byte accounting, INT4
packer) built with g++ under AddressSanitizer and UBSan, and driven through
its C ABI in a child process that preloads the sanitizer runtime."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    p = r.stdout.strip()
    return p if r.returncode == 0 and os.path.isabs(p) and os.path.exists(p) else None


def test_host_abi_under_asan_and_ubsan():
    from paper_2608_02703_amd import build
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("no libasan runtime for g++")
    lib = build.build_host(sanitize=True)
    env = dict(os.environ, LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "host_sanitizer_driver.py"),
                        lib], env=env, capture_output=True, text=True, timeout=300)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "AddressSanitizer" not in report and "runtime error" not in report, report[-4000:]
    assert "host ABI under sanitizers: ok" in r.stdout
