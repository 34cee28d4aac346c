"""Builds the host sanitizer drivers (test infrastructure).

runtime_check: the library's sources with AddressSanitizer and
UndefinedBehaviorSanitizer on their host side only (device code is compiled
as usual) linked with runtime_check.cpp.  oracle_check: the oracle's C
source compiled into oracle_check.c with both sanitizers.  `python -m
tests.sanitize.build` (or __graft_entry__.build) writes the runtime driver
next to this file, where the GPU test runs it."""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
from paper_2606_03113_amd import build as b  # noqa: E402

CLANG = "/opt/rocm/llvm/bin/clang++"
# host-side instrumentation only: device code is left as it is
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
RUNTIME_CHECK = os.path.join(HERE, "runtime_check")


def build_runtime_check(out: str = RUNTIME_CHECK) -> str:
    with tempfile.TemporaryDirectory() as tmp:
        objs, procs = [], []
        for src in b.SOURCES:
            obj = os.path.join(tmp, src + ".o")
            cmd = [b.HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", *HOST_SAN,
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument",
                   "-c", os.path.join(b.CSRC, src), "-o", obj]
            if src.endswith(".hip"):
                cmd[1:1] = ["-x", "hip"]
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
            objs.append(obj)
        drv = os.path.join(tmp, "runtime_check.o")
        procs.append(("runtime_check.cpp", subprocess.Popen(
            [CLANG, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
             "-c", os.path.join(HERE, "runtime_check.cpp"), "-o", drv],
            stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        failed = []
        for src, p in procs:
            text = p.communicate(timeout=900)[0].decode(errors="replace")
            if p.returncode != 0:
                failed.append(src + ":\n" + text[-2000:])
        if failed:
            raise RuntimeError("sanitizer build failed:\n" + "\n".join(failed))
        tmp_out = out + ".tmp%d" % os.getpid()
        subprocess.check_call([b.HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, drv, "-o", tmp_out])
        os.replace(tmp_out, out)
    return out


def build_oracle_check(out: str) -> str:
    subprocess.check_call(["gcc", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-g", "-O1", "-fopenmp", "-ffp-contract=off",
                           os.path.join(HERE, "oracle_check.c"), "-lm", "-o", out])
    return out


# sanitizer options for the drivers: leak detection on, the ROCm runtime's own
# allocations kept at exit suppressed
LSAN_SUPPRESSIONS = os.path.join(HERE, "lsan.supp")


def env() -> dict:
    return dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                LSAN_OPTIONS="suppressions=" + LSAN_SUPPRESSIONS, UBSAN_OPTIONS="print_stacktrace=1")


if __name__ == "__main__":
    print(build_runtime_check())
