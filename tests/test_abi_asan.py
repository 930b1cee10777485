"""The C ABI's host-side argument validation under AddressSanitizer (CPU only).

tests/test_abi.py (every entry point fed invalid, null, misaligned and oversized
arguments, none of which may reach a launch) runs in a child process against the
host ASan build of the C ABI layer (paper_2609_39329_amd/build_asan.py), with the
sanitizer runtime preloaded. Any out-of-bounds access or use-after-free in the
validation code aborts the child.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ASAN_LIB = os.path.join(ROOT, "paper_2609_39329_amd", "lib", "libpatchkv_asan.so")


def _libasan():
    try:
        p = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True,
                           text=True).stdout.strip()
    except OSError:
        return None
    return os.path.realpath(p) if p and os.path.exists(p) else None


def test_abi_validation_under_asan():
    if not os.path.exists(ASAN_LIB):
        pytest.skip("ASan build missing (run paper_2609_39329_amd/build_asan.py)")
    rt = _libasan()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime on this host")
    env = dict(os.environ, PATCHKV_LIBRARY=ASAN_LIB, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:verify_asan_link_order=0:abort_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout
