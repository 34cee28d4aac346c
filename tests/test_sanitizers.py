"""Host sanitizer runs (no GPU needed).

- The CPU oracle's C source is compiled with AddressSanitizer and
  UndefinedBehaviorSanitizer into a driver (tests/sanitize/oracle_check.c)
  that runs every exported routine on a tiny grouped-query model in fp32 and
  bf16 and checks that a batch of rows equals the same rows one at a time.
- The library's host code (runtime, trainer handle, and the host side of
  every HIP source; device code is not instrumented) is built the same way
  and linked into a driver (tests/sanitize/runtime_check.cpp) that sizes
  regions, checks argument validation of every entry point and tears down a
  context whose device calls fail.  On a GPU the same driver also decodes
  (tests/test_gpu_sanitized_runtime.py).

Leak detection is on; any sanitizer report fails the run."""
import os
import shutil
import subprocess

import pytest

from paper_2606_03113_amd import build as b
from tests.sanitize import build as sb


def _run(exe):
    p = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=sb.env())
    return p.returncode, p.stdout + p.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_clean_under_asan_ubsan(tmp_path):
    rc, out = _run(sb.build_oracle_check(str(tmp_path / "oracle_check")))
    assert rc == 0 and "oracle sanitizer run: clean" in out, out[-4000:]


@pytest.mark.skipif(not (os.path.exists(b.HIPCC) and os.path.exists(sb.CLANG)), reason="ROCm compilers not installed")
def test_runtime_host_clean_under_asan_ubsan(tmp_path):
    rc, out = _run(sb.build_runtime_check(str(tmp_path / "runtime_check")))
    assert rc == 0 and "runtime sanitizer run: clean" in out, out[-4000:]
