"""Static instruction report of the gfx950 kernels, from their own assembly.

Compiles csrc/fpde.hip to device assembly with the library's flags and counts,
per kernel, the instruction classes that carry the design:

- plane loads streamed straight into LDS (``buffer_load_dword ... lds``) and
  LDS reads/writes (``ds_*``), the halo tiles of the 2.5-D march;
- DPP instructions (cross-lane row/quad permutes), the wavefront loss sum;
- global atomics: one float64 add per workgroup in the kernels that reduce the
  loss, none in the backward's gather, the boundary kernel or the vjp;
- no MFMA (the operator is a memory-bound stencil, not a contraction) and no
  packed-FP32 VALU (``v_pk_*_f32``, disabled for all device code);
- registers, LDS bytes and scratch from the compiler's own resource notes.

Usage: python -m paper_2607_18020_amd.isa_report [--out profiles/isa_kernels.md]
"""
from __future__ import annotations

import argparse
import os
import re
import subprocess
import sys
import tempfile
from typing import Dict, List

from paper_2607_18020_amd.csrc import build as B

KERNEL_PREFIXES = ("fwd_kernel", "fwdq_kernel", "bwd_kernel", "bwdq_kernel", "vjp_kernel", "bc_kernel",
                   "bc4_kernel", "tm_kernel", "zero_levels_kernel", "fill_f64_kernel")


def compile_asm(path: str) -> None:
    cmd = [B.HIPCC, *[f for f in B.FLAGS if f not in ("-fPIC", "-shared")], "--cuda-device-only",
           "-S", "-o", path, *B.SOURCES]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(r.stdout + r.stderr)


def _demangle(names: List[str]) -> Dict[str, str]:
    r = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True)
    out = r.stdout.splitlines() if r.returncode == 0 else names
    return {m: d.replace("fpde::", "").split("(")[0].replace("void ", "")
            for m, d in zip(names, out)}


def parse(asm: str) -> Dict[str, dict]:
    """Per kernel: instruction-class counts and resource notes (the notes the
    compiler prints after each function belong to the span up to the next one)."""
    lines = asm.splitlines()
    starts = [(i, m.group(1)) for i, ln in enumerate(lines)
              for m in [re.match(r"^(_Z\w+):", ln)] if m]
    names = _demangle([n for _, n in starts])
    kernels: Dict[str, dict] = {}
    for k, (i0, mangled) in enumerate(starts):
        name = names[mangled]
        if not name.startswith(KERNEL_PREFIXES):
            continue
        i1 = starts[k + 1][0] if k + 1 < len(starts) else len(lines)
        c = {"valu": 0, "salu": 0, "lds_dma": 0, "ds_read": 0, "ds_write": 0, "vmem_load": 0,
             "vmem_store": 0, "atomic": 0, "dpp": 0, "barrier": 0, "mfma": 0, "pk_f32": 0,
             "f64": 0, "scratch_ops": 0}
        res = {}
        for ln in lines[i0 + 1:i1]:
            s = ln.strip()
            m = re.match(r";\s*(NumVgprs|NumSgprs|ScratchSize|Occupancy|LDSByteSize):\s*(\d+)", s)
            if m:
                res.setdefault(m.group(1), int(m.group(2)))
                continue
            if not s or s.startswith((";", ".")) or s.endswith(":"):
                continue
            op = s.split()[0]
            if op.startswith("v_mfma"):
                c["mfma"] += 1
            if re.match(r"v_pk_\w+_f32", op):
                c["pk_f32"] += 1
            if op.startswith("v_"):
                c["valu"] += 1
                if "_f64" in op:
                    c["f64"] += 1
                if re.search(r"\b(quad_perm|row_\w+|wave_\w+)", s):
                    c["dpp"] += 1
            elif op.startswith("s_"):
                c["salu"] += 1
                if op == "s_barrier":
                    c["barrier"] += 1
            elif op.startswith("ds_"):
                c["ds_read" if "read" in op else "ds_write"] += 1
            elif op.startswith("scratch_"):
                c["scratch_ops"] += 1
            elif op.startswith(("buffer_", "global_", "flat_")):
                if "atomic" in op:
                    c["atomic"] += 1
                elif re.search(r"\blds\b", s):
                    c["lds_dma"] += 1
                elif "load" in op:
                    c["vmem_load"] += 1
                elif "store" in op:
                    c["vmem_store"] += 1
        c.update({"vgprs": res.get("NumVgprs"), "sgprs": res.get("NumSgprs"),
                  "lds_bytes": res.get("LDSByteSize"), "scratch": res.get("ScratchSize"),
                  "occupancy": res.get("Occupancy")})
        kernels[name] = c
    return kernels


def memory_stream(asm: str, kernel: str) -> List[str]:
    """The kernel's vector-memory operations, explicit barrier waits and
    barriers in code order: "D" a load into LDS, "L" a load into registers,
    "S" a store, "A" an atomic, "W<n>" an `s_waitcnt vmcnt(n) lgkmcnt(0)`
    directly before an `s_barrier`, "B" the barrier.  (Code order, not
    execution order: loops and branches are not followed.)"""
    lines = asm.splitlines()
    starts = [(i, m.group(1)) for i, ln in enumerate(lines)
              for m in [re.match(r"^(_Z\w+):", ln)] if m]
    names = _demangle([n for _, n in starts])
    for k, (i0, mangled) in enumerate(starts):
        if names[mangled] != kernel:
            continue
        i1 = starts[k + 1][0] if k + 1 < len(starts) else len(lines)
        body = [ln.strip() for ln in lines[i0 + 1:i1]]
        body = [s for s in body if s and not s.startswith((";", ".")) and not s.endswith(":")]
        out: List[str] = []
        for j, s in enumerate(body):
            op = s.split()[0]
            if op.startswith(("buffer_", "global_", "flat_")):
                if "atomic" in op:
                    out.append("A")
                elif re.search(r"\blds\b", s):
                    out.append("D")
                else:
                    out.append("L" if "load" in op else "S")
            elif op == "s_barrier":
                out.append("B")
            else:
                m = re.match(r"s_waitcnt vmcnt\((\d+)\) lgkmcnt\(0\)$", s)
                if m and j + 1 < len(body) and body[j + 1].startswith("s_barrier"):
                    out.append("W" + m.group(1))
        return out
    raise KeyError(kernel)


def _template_args(name: str) -> List[str]:
    args = name[name.index("<") + 1:name.rindex(">")]
    out, depth, cur = [], 0, ""
    for ch in args:
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        if ch == "," and depth == 0:
            out.append(cur.strip())
            cur = ""
        else:
            cur += ch
    out.append(cur.strip())
    return out


def reduces_loss(name: str) -> bool:
    """The kernels that add a float64 partial loss per workgroup: every forward,
    and the backward with its LOSS flag (bwd_kernel<OP, TX, TY, REV, LOSS, PER>)."""
    if name.startswith(("fwd_kernel", "fwdq_kernel")):
        return True
    return name.startswith("bwd_kernel") and _template_args(name)[4] == "true"


def violations(kernels: Dict[str, dict]) -> List[str]:
    """Design rules the assembly must keep."""
    bad = []
    for name, c in kernels.items():
        if c["mfma"]:
            bad.append(f"{name}: {c['mfma']} MFMA instructions")
        if c["pk_f32"]:
            bad.append(f"{name}: {c['pk_f32']} packed-FP32 instructions")
        if c["scratch_ops"]:
            bad.append(f"{name}: {c['scratch_ops']} scratch accesses (register spills)")
        if reduces_loss(name):
            if c["atomic"] != 1:
                bad.append(f"{name}: {c['atomic']} atomic instructions, expected one")
            if c["dpp"] == 0:
                bad.append(f"{name}: no DPP wavefront reduction")
        elif c["atomic"]:
            bad.append(f"{name}: {c['atomic']} atomics in a kernel without a loss")
    return bad


def report(kernels: Dict[str, dict], command: str, match=("",)) -> str:
    cols = ["vgprs", "lds_bytes", "scratch", "scratch_ops", "occupancy", "valu", "f64", "salu",
            "lds_dma", "ds_read", "ds_write", "vmem_load", "vmem_store", "atomic", "dpp",
            "barrier", "mfma", "pk_f32"]
    out = ["# Static instruction counts of the gfx950 kernels (their own assembly)", "",
           "Command (from the repository root, on any machine with hipcc):", "", "```",
           command, "```", "",
           "Counts are instructions in each kernel's code (not executed counts). "
           "`lds_dma`: buffer loads that write LDS directly (plane streaming); `dpp`: VALU "
           "instructions with a DPP cross-lane modifier (the wavefront loss sum); "
           "`atomic`: global atomics (one float64 add, executed by one thread per "
           "workgroup, in the kernels that reduce the loss); `scratch`: the private segment "
           "the compiler reserves (bytes), `scratch_ops`: instructions that use it (spills); "
           "`mfma`, `pk_f32`, `scratch_ops`: must be 0.",
           "", "| kernel | " + " | ".join(cols) + " |", "|---|" + "---|" * len(cols)]
    for name in sorted(kernels):
        if any(m in name for m in match):
            c = kernels[name]
            out.append(f"| `{name}` | " + " | ".join(str(c[k]) for k in cols) + " |")
    bad = violations(kernels)
    out += ["", f"Design-rule check over all {len(kernels)} kernels of the library: " +
            ("all pass." if not bad else "; ".join(bad))]
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--out", default=None, help="write the markdown report here")
    ap.add_argument("--match", action="append", default=None,
                    help="list only kernels whose name contains this (repeatable; the rule "
                         "check covers every kernel)")
    a = ap.parse_args(argv)
    with tempfile.TemporaryDirectory() as d:
        asm_path = os.path.join(d, "fpde.s")
        compile_asm(asm_path)
        kernels = parse(open(asm_path).read())
    match = a.match or [""]
    cmd = "python -m paper_2607_18020_amd.isa_report --out profiles/isa_kernels.md" + "".join(
        f" --match '{m}'" for m in (a.match or []))
    text = report(kernels, cmd, match)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    print(text)
    return 1 if violations(kernels) else 0


if __name__ == "__main__":
    sys.exit(main())
