"""Build libfpde.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2607_18020_amd.csrc.build [--save-temps]
Writes paper_2607_18020_amd/libfpde.so.  Packed-FP32 VALU ops are disabled
for all device code; float64 atomics use the native global_atomic_add_f64;
floating-point contraction is off (the operators' fmaf are explicit).
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
    # no implicit fusing of a multiply and an add: the operators write their fmaf
    # explicitly, so each one is the same instruction sequence in every kernel
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"), "-I", HERE,
]


# The checking library (tests only): LDS filled with NaN before every march, and
# other tile shapes, chunk lengths and 2-D row widths than the product library
# (and the register-queue forward for heat and 3-D Poisson),
# so that a read of an LDS location nothing wrote turns into NaN, and so that
# the gradients can be compared bit for bit across tilings (a gather-form
# backward evaluates every node the same way whatever tile holds it).
CHECK_LIB = os.path.join(PKG, "libfpde_check.so")
CHECK_FLAGS = [
    "-DFPDE_LDS_POISON=1",
    "-DFPDE_NS3_FWD_TX=64", "-DFPDE_NS3_FWD_TY=8", "-DFPDE_NS3_BWD_TX=64", "-DFPDE_NS3_BWD_TY=16",
    "-DFPDE_NS3_MIN_BWD_BLOCKS=512", "-DFPDE_HEAT_FWD_TX=128", "-DFPDE_HEAT_BWD_TX=128",
    "-DFPDE_HEAT_MIN_BWD_BLOCKS=256", "-DFPDE_VJP_TY3=8", "-DFPDE_VJP_HEAT_TX=64",
    "-DFPDE_TX2=128", "-DFPDE_TX2_FWD=256", "-DFPDE_TX2_VG=256", "-DFPDE_BLOCKS2=512",
    "-DFPDE_FWD2_Q=4", "-DFPDE_HEAT_FWD_QUEUE=1", "-DFPDE_NS4_BWD_TX=64", "-DFPDE_NS4_BWD_TY=8",
    "-DFPDE_BWD2_QUEUE=1", "-DFPDE_NS4_MIN_BLOCKS=700", "-DFPDE_TM_REMAP=1",
]

_NOISE = "is not a recognized feature for this target"


def _command(out: str, extra=(), save_temps: bool = False):
    cmd = [HIPCC, *FLAGS, *extra, "-o", out + ".tmp", *SOURCES]
    if save_temps:
        cmd.insert(1, "-save-temps")
    return cmd


def _finish(p, out: str, verbose: bool) -> None:
    stdout, stderr = p.communicate()
    # hipcc's host pass does not know the packed-fp32 feature and says so; drop that line
    msgs = [ln for ln in (stdout + stderr).splitlines() if _NOISE not in ln]
    if msgs and (verbose or p.returncode):
        print("\n".join(msgs), file=sys.stderr)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed ({p.returncode}) for {out}")
    os.replace(out + ".tmp", out)


def build(save_temps: bool = False, verbose: bool = False, out: str = LIB, extra=(),
          check: bool = True) -> str:
    """Compile the product library (and, with check, the checking library in
    parallel)."""
    jobs = [(out, _command(out, extra, save_temps))]
    if check and out == LIB and not extra:
        jobs.append((CHECK_LIB, _command(CHECK_LIB, CHECK_FLAGS)))
    procs = []
    for o, cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((o, subprocess.Popen(
            cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
            cwd=os.path.join(ROOT, "_build") if save_temps and o == out else None)))
    for o, p in procs:
        _finish(p, o, verbose)
    return out


if __name__ == "__main__":
    st = "--save-temps" in sys.argv
    if st:
        os.makedirs(os.path.join(ROOT, "_build"), exist_ok=True)
    print(build(save_temps=st, verbose=True))
