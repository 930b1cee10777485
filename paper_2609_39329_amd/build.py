"""Build libpatchkv.so (gfx950) in-tree with hipcc.

Each source is compiled to an object in parallel, then linked into
``paper_2609_39329_amd/lib/libpatchkv.so``. Packed-fp32 VALU instructions are
disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB_DIR = os.path.join(HERE, "lib")
LIB = os.path.join(LIB_DIR, "libpatchkv.so")
ARCH = "gfx950"

SOURCES = ["attention.hip", "attention_mx.hip", "stats.hip", "solve.hip", "capi.cpp"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# The C ABI layer holds no device code: plain host C++ against the HIP runtime headers.
HOST = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]
# Per-source extras. The attention kernels never see NaNs (masked scores are -inf),
# so they run with the IEEE mode bit off, which lets max() skip NaN quieting.
EXTRA = {s: ["-mno-amdgpu-ieee", "-fno-honor-nans"] for s in ("attention.hip", "attention_mx.hip")}


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libpatchkv)")


def host_cxx() -> str:
    for c in (os.environ.get("CXX"), shutil.which("g++"), shutil.which("c++")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("no host C++ compiler found")


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    if src.endswith(".hip"):
        cmd = [hipcc(), *COMMON, *DEVICE]
    else:
        cmd = [host_cxx(), *COMMON, *HOST]
    cmd += EXTRA.get(src, [])
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(OBJ, exist_ok=True)
    os.makedirs(LIB_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(min(len(SOURCES), 8)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # a library that links can still fail to load (a kernel whose host-side launch stub
    # the compiler did not emit leaves an undefined symbol): load it in a child process,
    # with every symbol resolved, before it replaces the previous build
    chk = [sys.executable, "-c", "import ctypes, os, sys; ctypes.CDLL(sys.argv[1], mode=os.RTLD_NOW)", tmp]
    r = subprocess.run(chk, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"the linked library does not load:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
