"""Build the ARCHead HIP library for gfx950 (in-tree, no JIT cache).

``python -m paper_2608_02703_amd.build`` compiles csrc/host.cpp,
csrc/archead.hip and csrc/fidelity.hip with hipcc into
paper_2608_02703_amd/libarchead.so, and the
host-only translation unit with g++ (optionally under ASan/UBSan) into
libarchead_host.so for the CPU tests of the argument checks and packers.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libarchead.so")
HOST_LIB = os.path.join(PKG, "libarchead_host.so")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the library)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build failed ({r.returncode}):\n{' '.join(cmd)}\n"
                           f"{r.stdout}\n{r.stderr}")


def build_hip(verbose: bool = False, out: str = LIB, defines=()) -> str:
    tmp = out + ".tmp"
    cmd = [_hipcc(), *HIP_FLAGS, *[f"-D{d}" for d in defines], f"-I{INCLUDE}",
           os.path.join(CSRC, "host.cpp"), os.path.join(CSRC, "archead.hip"),
           os.path.join(CSRC, "fidelity.hip"), "-o", tmp]
    _run(cmd, verbose)
    os.replace(tmp, out)
    return out


def build_host(verbose: bool = False, sanitize: bool = False) -> str:
    out = HOST_LIB if not sanitize else os.path.join(PKG, "libarchead_host_asan.so")
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", f"-I{INCLUDE}",
           os.path.join(CSRC, "host.cpp"), "-o", out + ".tmp"]
    if sanitize:
        cmd[1:1] = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]
    _run(cmd, verbose)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False) -> None:
    build_host(verbose)
    build_hip(verbose)


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB, file=sys.stderr)
