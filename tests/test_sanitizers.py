"""Host sanitizer runs (no GPU needed).

- The CPU oracle's C source is compiled with AddressSanitizer and
  UndefinedBehaviorSanitizer into a driver (tests/sanitize/oracle_check.c)
  that runs every exported routine on a tiny grouped-query model in fp32 and
  bf16 and checks that a batch of rows equals the same rows one at a time.
- The library's host code (runtime, trainer handle, and the host side of
  every HIP source; device code is not instrumented) is built the same way
  and linked into a driver (tests/sanitize/runtime_check.cpp) that sizes
  regions, checks argument validation of every entry point and tears down a
  context whose device calls fail.

Leak detection is on; any sanitizer report fails the run."""
import os
import shutil
import subprocess

import pytest

from paper_2606_03113_amd import build as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_DIR = os.path.join(ROOT, "tests", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang++"
# host-side instrumentation only: device code is left as it is
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(exe):
    p = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=ENV)
    return p.returncode, p.stdout + p.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_clean_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_check")
    subprocess.check_call(["gcc", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-g", "-O1", "-fopenmp", "-ffp-contract=off",
                           os.path.join(SAN_DIR, "oracle_check.c"), "-lm", "-o", exe])
    rc, out = _run(exe)
    assert rc == 0 and "oracle sanitizer run: clean" in out, out[-4000:]


@pytest.mark.skipif(not (os.path.exists(b.HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not installed")
def test_runtime_host_clean_under_asan_ubsan(tmp_path):
    objs, procs = [], []
    for src in b.SOURCES:
        obj = str(tmp_path / (src + ".o"))
        cmd = [b.HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", *HOST_SAN,
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument",
               "-c", os.path.join(b.CSRC, src), "-o", obj]
        if src.endswith(".hip"):
            cmd[1:1] = ["-x", "hip"]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    drv = str(tmp_path / "runtime_check.o")
    procs.append(("runtime_check.cpp", subprocess.Popen(
        [CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-c", os.path.join(SAN_DIR, "runtime_check.cpp"), "-o", drv],
        stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        out = p.communicate(timeout=600)[0]
        if p.returncode != 0:
            failed.append((src, out[-2000:]))
    assert not failed, failed
    exe = str(tmp_path / "runtime_check")
    subprocess.check_call([b.HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, drv, "-o", exe])
    rc, out = _run(exe)
    assert rc == 0 and "runtime sanitizer run: clean" in out, out[-4000:]
