"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

``python -m paper_2412_05693_amd.build --sanitize`` (also run by the build
entry point) instruments the host side of the library -- argument, capacity
and order checks, context handling, launch setup -- and leaves the gfx950
device code as it is.  This test runs the CPU tests of the ABI and of the
benchmark's host logic in a child process that loads that build with the
sanitizer runtime preloaded; any report aborts the child.  It first checks that
the child really loaded the instrumented library and the runtime."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2412_05693_amd import build as B  # noqa: E402

PROBE = r"""
import sys
sys.path.insert(0, sys.argv[1])
from paper_2412_05693_amd import batchmax as bmx
maps = open("/proc/self/maps").read()
assert bmx.LIB_PATH.endswith("libbatchmax_san.so"), bmx.LIB_PATH
assert "libbatchmax_san.so" in maps and "libclang_rt.asan" in maps
print("sanitized library loaded")
"""


def _stale() -> bool:
    """The instrumented library is missing or older than a source file."""
    if not os.path.exists(B.LIB_SAN):
        return True
    built = os.path.getmtime(B.LIB_SAN)
    for d in (B.CSRC, B.INCLUDE):
        for f in os.listdir(d):
            if os.path.getmtime(os.path.join(d, f)) > built:
                return True
    return False


def _san_env():
    if _stale():
        B.build(sanitize=True)
    return B.sanitizer_env()


def test_sanitizer_build_is_loaded():
    r = subprocess.run([sys.executable, "-c", PROBE, ROOT], env=_san_env(), capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "sanitized library loaded" in r.stdout


def test_abi_and_bench_host_tests_under_sanitizers():
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py"),
                        os.path.join(ROOT, "tests", "test_bench_host.py")],
                       env=_san_env(), capture_output=True, text=True, timeout=900, cwd=ROOT)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error:" not in r.stderr
