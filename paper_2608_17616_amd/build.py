"""Build the HIP library libmone_ttl.so for gfx950, in the package directory.

    python -m paper_2608_17616_amd.build [--verbose]
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SOURCES = [os.path.join(PKG, "csrc", "mone_ttl.hip"), os.path.join(PKG, "csrc", "mone_swiglu.hip")]
DEPENDS = SOURCES + [os.path.join(PKG, "csrc", f) for f in
                     ("kernels.hpp", "host_common.hpp", "swiglu_kernels.hpp")] + [
                     os.path.join(ROOT, "include", f) for f in ("mone_ttl.h", "mone_swiglu.h")]
LIB = os.path.join(PKG, "libmone_ttl.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def build(verbose: bool = False, extra_flags: list[str] | None = None) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           # keep the compiler from emitting packed fp32 arithmetic
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include")]
    cmd += list(extra_flags or [])
    cmd += ["-o", tmp] + SOURCES
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    if verbose and res.stderr:
        print(res.stderr, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
