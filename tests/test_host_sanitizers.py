"""The library's host side under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU): a sanitized build of every source (device code compiled as usual) and
a C driver (tests/c_consumer/host_stress.c) that runs validation, size
queries, set binding, the anchor count and the argument checks of every
compute entry point over thousands of problem shapes, up to the limits the
header states.  No call reaches a device.  Any sanitizer finding or failed
check makes the driver exit non-zero."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c_consumer"))
import build_sanitized  # noqa: E402


@pytest.mark.skipif(shutil.which("gcc") is None or not os.path.exists(build_sanitized.HIPCC),
                    reason="needs hipcc and a host toolchain")
def test_host_side_clean_under_asan_ubsan(tmp_path):
    exe = build_sanitized.build(str(tmp_path))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.startswith("ok "), r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
