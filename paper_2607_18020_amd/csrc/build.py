"""Build libfpde.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2607_18020_amd.csrc.build [--save-temps]
Writes paper_2607_18020_amd/libfpde.so.  Packed-FP32 VALU ops are disabled
for all device code; float64 atomics use the native global_atomic_add_f64.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libfpde.so")
SOURCES = [os.path.join(HERE, "fpde.hip")]
HEADERS = [os.path.join(HERE, "fpde_engine.hpp"), os.path.join(HERE, "fpde_ops.hpp"),
           os.path.join(ROOT, "include", "fpde.h")]

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-munsafe-fp-atomics",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"), "-I", HERE,
]


def build(save_temps: bool = False, verbose: bool = False, out: str = LIB, extra=()) -> str:
    cmd = [HIPCC, *FLAGS, *extra, "-o", out + ".tmp", *SOURCES]
    if save_temps:
        cmd.insert(1, "-save-temps")
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True,
                       cwd=os.path.join(ROOT, "_build") if save_temps else None)
    # hipcc's host pass does not know the packed-fp32 feature and says so; drop that line
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln]
    if msgs and (verbose or r.returncode):
        print("\n".join(msgs), file=sys.stderr)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode})")
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    st = "--save-temps" in sys.argv
    if st:
        os.makedirs(os.path.join(ROOT, "_build"), exist_ok=True)
    print(build(save_temps=st, verbose=True))
