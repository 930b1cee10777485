"""Host AddressSanitizer build of the C ABI layer, for the CPU argument-validation tests.

The C ABI layer (capi.cpp, host code only) is compiled with AddressSanitizer by the
host compiler and linked with the regular device objects of build.py into
``lib/libpatchkv_asan.so``. The sanitizer runtime is not linked in: a process that
loads this library preloads it (see tests/test_abi_asan.py). Run build.py first.

    python paper_2609_39329_amd/build_asan.py
"""
from __future__ import annotations

import os
import subprocess
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
from paper_2609_39329_amd.build import (ARCH, COMMON, CSRC, HOST, LIB_DIR, OBJ,  # noqa: E402
                                        SOURCES, hipcc, host_cxx)

ASAN_LIB = os.path.join(LIB_DIR, "libpatchkv_asan.so")
SAN = ["-fsanitize=address", "-fno-omit-frame-pointer"]


def build_asan(verbose: bool = False) -> str:
    objs = [os.path.join(OBJ, os.path.splitext(f)[0] + ".o") for f in SOURCES if f.endswith(".hip")]
    if not all(os.path.exists(o) for o in objs):
        raise RuntimeError("build the library first (paper_2609_39329_amd/build.py)")
    capi = os.path.join(OBJ, "capi_asan.o")
    cmd = [host_cxx(), *COMMON, *HOST, *SAN, "-c", os.path.join(CSRC, "capi.cpp"), "-o", capi]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling capi.cpp with ASan failed:\n{r.stderr}")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", ASAN_LIB, *objs, capi]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking the ASan library failed:\n{r.stderr}")
    if verbose:
        print(f"built {ASAN_LIB}", file=sys.stderr)
    return ASAN_LIB


if __name__ == "__main__":
    build_asan(verbose=True)
