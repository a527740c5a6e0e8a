"""rocprofv3 summaries for the benchmark: kernel timings and calibrated HBM traffic.

Usage (after the rocprofv3 runs listed in ``--help`` have produced their CSVs):

    python -m paper_2607_18020_amd.profiling --stats DIR --fetch DIR --write DIR \
        --bench-json FILE --commands FILE --path PATH --name STEM --out profiles/

(PATH: the ``bench.py --path`` the runs were taken with; STEM: the summary's
file name.)

Traffic calibration: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are scaled by
what the same counters read for the benchmark's stream kernel (y = 1 * x over
1 GiB: 1 GiB read, 1 GiB written), so the figures are bytes, whatever the
counters' own unit and coverage.  ``traffic_<STEM>.json`` records the workload,
the bench path and a hash of the kernel sources (comments and whitespace
ignored); ``bench.py`` reports the traffic of the record for its workload and
path only while that hash still matches.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
from collections import defaultdict
from typing import Dict, List

PKG = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("csrc/fpde.hip", "csrc/fpde_engine.hpp", "csrc/fpde_ops.hpp")
STREAM_KERNEL = "MulFunctor"  # the benchmark's 1 GiB y = 1 * x kernel
STREAM_BYTES = 1 << 30
# the library's kernels (name stems)
KERNELS = ("fwd_kernel", "fwdq_kernel", "bwd_kernel", "bwdq_kernel", "bc_kernel", "bc4_kernel", "vjp_kernel",
           "tm_kernel", "zero_levels_kernel", "fill_f64")


def _code_only(text: str) -> str:
    """The source without comments and with whitespace collapsed: edits to
    comments do not change what was measured."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash(root: str = PKG) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(root, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def _csv(path_glob: str) -> List[dict]:
    paths = sorted(glob.glob(path_glob, recursive=True))
    if not paths:
        raise FileNotFoundError(path_glob)
    with open(paths[0]) as f:
        return list(csv.DictReader(f))


def short_name(kernel: str) -> str:
    return kernel.split("(")[0].replace("void ", "").replace("fpde::", "")


def kernel_stats(stats_dir: str) -> Dict[str, dict]:
    rows = _csv(os.path.join(stats_dir, "**", "*kernel_stats.csv"))
    return {short_name(r["Name"]): {"calls": int(r["Calls"]), "avg_us": float(r["AverageNs"]) / 1e3,
                                    "min_us": float(r["MinNs"]) / 1e3, "max_us": float(r["MaxNs"]) / 1e3}
            for r in rows}


def counter_per_dispatch(pmc_dir: str, counter: str) -> Dict[str, List[float]]:
    rows = _csv(os.path.join(pmc_dir, "**", "*counter_collection.csv"))
    out: Dict[str, List[float]] = defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            out[short_name(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return out


def calibrated(pmc_dir: str, counter: str) -> Dict[str, dict]:
    """Per-kernel average counter (KiB/dispatch) and bytes via the stream kernel."""
    vals = counter_per_dispatch(pmc_dir, counter)
    stream = [v for k, vs in vals.items() if STREAM_KERNEL in k for v in vs]
    if not stream:
        raise RuntimeError(f"no {STREAM_KERNEL} dispatch in {pmc_dir}")
    ref_kib = max(stream)  # the 1 GiB dispatch (smaller fills share the name pattern)
    factor = STREAM_BYTES / ref_kib  # bytes per counted KiB
    out = {"_calibration": {"stream_kib": ref_kib, "bytes_per_kib": factor}}
    for k, vs in vals.items():
        if k.startswith(KERNELS):
            avg = sum(vs) / len(vs)
            out[k] = {"dispatches": len(vs), "avg_kib": avg, "bytes": avg * factor}
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--stats", required=True, help="rocprofv3 --kernel-trace --stats output dir")
    ap.add_argument("--fetch", required=True, help="rocprofv3 --pmc FETCH_SIZE output dir")
    ap.add_argument("--write", required=True, help="rocprofv3 --pmc WRITE_SIZE output dir")
    ap.add_argument("--bench-json", required=True, help="bench.py JSON line printed under --stats")
    ap.add_argument("--commands", required=True, help="text file with the three rocprofv3 commands")
    ap.add_argument("--out", required=True)
    ap.add_argument("--workload", default="ns_3d_tgv 256^3")
    ap.add_argument("--path", default="loss", choices=("loss", "residual", "fused"),
                    help="the bench.py --path the runs were taken with")
    ap.add_argument("--name", default="ns3d_256_fwd_bwd_bc", help="summary file stem")
    a = ap.parse_args()

    stats = kernel_stats(a.stats)
    fetch = calibrated(a.fetch, "FETCH_SIZE")
    write = calibrated(a.write, "WRITE_SIZE")
    bench = json.loads(open(a.bench_json).read().strip().splitlines()[-1])
    cmds = open(a.commands).read().strip()
    sha = source_hash()
    os.makedirs(a.out, exist_ok=True)

    kern = sorted(k for k in stats if k.startswith(KERNELS))
    lines = [f"# Kernel timings and HBM traffic, {a.workload}, bench.py --path {a.path}", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", "",
             f"Kernel sources hash (comments and whitespace ignored): `{sha}`.", "",
             "## rocprofv3 --kernel-trace --stats (same process as the bench line below)", "",
             "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for k in kern:
        s = stats[k]
        lines.append(f"| `{k}` | {s['calls']} | {s['avg_us']:.2f} | {s['min_us']:.2f} | {s['max_us']:.2f} |")
    lines += ["", "bench.py line printed by that run (HIP-event timings):", "", "```",
              json.dumps({k: bench[k] for k in ("value", "ms_per_step", "hbm_gbps", "kernel_us", "roofline")}),
              "```", "",
              "## HBM traffic (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE; KiB per dispatch)", "",
              f"Calibration: the 1 GiB stream kernel reads FETCH_SIZE = {fetch['_calibration']['stream_kib']:.0f} KiB "
              f"and WRITE_SIZE = {write['_calibration']['stream_kib']:.0f} KiB, so 1 counted KiB = "
              f"{fetch['_calibration']['bytes_per_kib']:.1f} B fetched and "
              f"{write['_calibration']['bytes_per_kib']:.1f} B written.", "",
              "| kernel | FETCH KiB | fetched MB | WRITE KiB | written MB |", "|---|---|---|---|---|"]
    traffic = {}
    for k in sorted(set(fetch) | set(write)):
        if k.startswith("_"):
            continue
        fb = fetch.get(k, {}).get("bytes", 0.0)
        wb = write.get(k, {}).get("bytes", 0.0)
        lines.append(f"| `{k}` | {fetch.get(k, {}).get('avg_kib', 0):.0f} | {fb / 1e6:.1f} | "
                     f"{write.get(k, {}).get('avg_kib', 0):.0f} | {wb / 1e6:.1f} |")
        traffic[k] = {"fetch_bytes": fb, "write_bytes": wb}
    with open(os.path.join(a.out, a.name + ".md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(os.path.join(a.out, f"traffic_{a.name}.json"), "w") as f:
        json.dump({"source_hash": sha, "workload": a.workload, "path": a.path, "kernels": traffic,
                   "calibration": {"fetch": fetch["_calibration"], "write": write["_calibration"]}},
                  f, indent=1)
    print("\n".join(lines))


if __name__ == "__main__":
    main()
