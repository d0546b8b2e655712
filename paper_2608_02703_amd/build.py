"""Build the ARCHead HIP library for gfx950 (in-tree, no JIT cache).

``python -m paper_2608_02703_amd.build`` compiles every translation unit
under csrc/ (host.cpp and the .hip kernels) with hipcc, in parallel, into
objects under _build/, and links them into paper_2608_02703_amd/libarchead.so
(with rocBLAS and rocSOLVER, which the head-construction entry points call
for their dense GEMMs and the symmetric eigendecomposition); the host-only
translation unit is also built with g++ (optionally under ASan/UBSan) into
libarchead_host.so for the CPU tests of the argument checks and packers.

``build(reuse_objects=True)`` (or ARCHEAD_REUSE_OBJECTS=1) keeps an object
whose source, headers and flags are unchanged; the default rebuilds all.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libarchead.so")
HOST_LIB = os.path.join(PKG, "libarchead_host.so")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
LINK_LIBS = ["-L/opt/rocm/lib", "-lrocblas", "-lrocsolver", "-Wl,-rpath,/opt/rocm/lib"]


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


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + [os.path.join(CSRC, "host.cpp")]


def _headers_digest() -> bytes:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(CSRC, "*.cuh")) +
                    glob.glob(os.path.join(INCLUDE, "*.h"))):
        with open(p, "rb") as f:
            h.update(p.encode() + f.read())
    return h.digest()


def _compile(src, flags, reuse, verbose, hdr):
    os.makedirs(OBJDIR, exist_ok=True)
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    with open(src, "rb") as f:
        key = hashlib.sha256(f.read() + hdr + " ".join(flags).encode()).hexdigest()
    stamp = obj + ".key"
    if reuse and os.path.exists(obj) and os.path.exists(stamp) and open(stamp).read() == key:
        return obj
    cmd = [_hipcc(), *flags, "-c", src, "-o", obj + ".tmp"]
    _run(cmd, verbose)
    os.replace(obj + ".tmp", obj)
    with open(stamp, "w") as f:
        f.write(key)
    return obj


def build_hip(verbose: bool = False, out: str = LIB, defines=(), reuse_objects=None) -> str:
    if reuse_objects is None:
        reuse_objects = os.environ.get("ARCHEAD_REUSE_OBJECTS") == "1"
    flags = [*HIP_FLAGS, *[f"-D{d}" for d in defines], f"-I{INCLUDE}"]
    hdr = _headers_digest()
    srcs = sources()
    jobs = max(1, min(len(srcs), os.cpu_count() or 1, 16))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, flags, reuse_objects, verbose, hdr), srcs))
    tmp = out + ".tmp"
    _run([_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, *LINK_LIBS, "-o", tmp],
         verbose)
    os.replace(tmp, out)
    return out


def build_host(verbose: bool = False, sanitize: bool = False) -> str:
    out = HOST_LIB if not sanitize else os.path.join(PKG, "libarchead_host_asan.so")
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", f"-I{INCLUDE}",
           os.path.join(CSRC, "host.cpp"), "-o", out + ".tmp"]
    if sanitize:
        cmd[1:1] = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                    "-fno-sanitize-recover=undefined"]
    _run(cmd, verbose)
    os.replace(out + ".tmp", out)
    return out


def build(verbose: bool = False, reuse_objects=None) -> None:
    build_host(verbose)
    build_hip(verbose, reuse_objects=reuse_objects)


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB, file=sys.stderr)
