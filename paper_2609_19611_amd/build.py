"""Builds libdirigo_rocm.so (HIP, gfx950) and the host-emulation test library.

    python -m paper_2609_19611_amd.build

The HIP library holds the compiler, the C ABI and the kernels.  The host
emulation library (g++ only) runs the same plans and block code with one
host thread and is loaded only by CPU tests.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIBDIR = os.path.join(HERE, "lib")
LIB = os.path.join(LIBDIR, "libdirigo_rocm.so")
HOSTEMU = os.path.join(LIBDIR, "libdirigo_hostemu.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
             # Packed FP32 instructions stay off (no float code here, but the
             # flag keeps every build of this library on the same footing).
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_SOURCES = ["graph.cpp", "compile.cpp", "abi.cpp"]
HIP_SOURCES = ["kernels.hip"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build_hip(verbose: bool = False) -> str:
    os.makedirs(LIBDIR, exist_ok=True)
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in HOST_SOURCES + HIP_SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        jobs.append(([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj], obj))
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        list(ex.map(lambda j: _run(j[0]), jobs))
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *[o for _, o in jobs], "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


def build_hostemu(verbose: bool = False) -> str:
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = HOSTEMU + ".tmp"
    _run(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-Wall", "-Wno-unused-function",
          *[os.path.join(CSRC, s) for s in ("graph.cpp", "compile.cpp", "hostemu.cpp")], "-o", tmp])
    os.replace(tmp, HOSTEMU)
    if verbose:
        print("built", HOSTEMU)
    return HOSTEMU


def build_all(verbose: bool = False) -> None:
    with cf.ThreadPoolExecutor(max_workers=2) as ex:
        a = ex.submit(build_hip, verbose)
        b = ex.submit(build_hostemu, verbose)
        a.result()
        b.result()


if __name__ == "__main__":
    build_all(verbose=True)
    sys.exit(0)
