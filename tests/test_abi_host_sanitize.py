"""The library's host-side argument validation under AddressSanitizer and
UndefinedBehaviorSanitizer (no GPU): the library is built with both sanitizers
on its host code (its device code, which never runs here, unoptimised to keep
the build short), and tests/c/abi_host_sanitize.c, built
with the same compiler's sanitizer runtime, calls every entry point with
arguments that break one rule each (null pointers, wrong rank, extents at and
past every size limit, non-finite or overflowing spacings and coefficients,
misalignment, overlapping outputs).  Every call must return its documented
status before queueing anything, with no sanitizer report."""
from __future__ import annotations

import os
import subprocess

import pytest

from paper_2607_18020_amd.csrc import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer", "-g"]


@pytest.mark.skipif(not (os.path.exists(B.HIPCC) and os.path.exists(CLANG)),
                    reason="hipcc / clang not available")
def test_validation_is_clean_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libfpde_host.so")
    cmd = [B.HIPCC, *B.FLAGS, "-Xarch_device", "-O0"]
    for f in SAN:  # host code only
        cmd += ["-Xarch_host", f]
    cmd += ["-o", lib, *B.SOURCES]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    exe = str(tmp_path / "abi_host_sanitize")
    cmd = [CLANG, "-std=c99", "-O1", *SAN, "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "c", "abi_host_sanitize.c"), lib,
           f"-Wl,-rpath,{tmp_path}", "-Wl,-rpath,/opt/rocm/lib", "-lm", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    # (leaks: the HIP runtime's own allocations at exit are not the library's)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout[-3000:], r.stderr[-3000:])
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi-host-sanitize:" in r.stdout and "ok" in r.stdout
