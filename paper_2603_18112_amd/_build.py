"""Build of libags.so for gfx950 with hipcc (in-tree, no JIT cache)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libags.so")
SOURCES = [os.path.join(CSRC, "ags_api.hip"), os.path.join(CSRC, "ags_kernels.hip"),
           os.path.join(CSRC, "ags_plan.cpp")]
HEADERS = [os.path.join(CSRC, "ags_internal.h"), os.path.join(INCLUDE, "ags.h"),
           os.path.join(INCLUDE, "ags_plan.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    # No packed fp32 instructions: the compiler emits plain fp32 VALU ops.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # Fused multiply-adds only where the source writes fmaf.
    "-ffp-contract=off",
    "-Wall", "-Wno-unused-result",
]


#: the HBM bandwidth probe the benchmark runs for context (a program, not
#: part of the library)
PROBE_SRC = os.path.join(CSRC, "hbm_probe.hip")
PROBE = os.path.join(LIBDIR, "hbm_probe")


def command(out: str = LIB):
    return [HIPCC, *FLAGS, "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", out]


def probe_command(out: str = PROBE):
    flags = [f for f in FLAGS if f not in ("-fPIC", "-shared")]
    return [HIPCC, *flags, PROBE_SRC, "-o", out]


def build(verbose: bool = False) -> str:
    """Compile libags.so; always rebuilds.  Returns the library path."""
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed to build libags.so")
    os.replace(tmp, LIB)
    tmp = PROBE + f".tmp{os.getpid()}"
    r = subprocess.run(probe_command(tmp), capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed to build hbm_probe")
    os.replace(tmp, PROBE)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True))
