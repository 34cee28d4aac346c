"""Builds the oracle's C library (gcc, OpenMP, IEEE arithmetic: no fast-math,
no floating-point contraction)."""
import os
import subprocess

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liblede_oracle.so")


def library_path() -> str:
    return _SO


def _has_avx2() -> bool:
    try:
        with open("/proc/cpuinfo") as f:
            return " avx2" in f.read()
    except OSError:
        return False


def build(force: bool = False, src: str | None = None, out: str | None = None) -> str:
    src = src or os.path.join(_HERE, "lede_oracle.c")
    out = out or _SO
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        flags = ["-O3", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]
        if _has_avx2():
            flags.append("-mavx2")  # wider vectors over independent rows only
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *flags, "-o", tmp, src, "-lm"])
        os.replace(tmp, out)
    return out
