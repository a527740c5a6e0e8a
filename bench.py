"""Throughput of the differentiable FD residual operator on one MI355X.

One step = the whole hot path on one batch of resident synthetic input:
fpde_residual_fwd (fused stencil + loss) -> fpde_residual_bwd (interior
adjoint) -> fpde_bc_correct (boundary shell), queued on one stream.

Default workload: 3D Taylor-Green NS, one backward-Euler step, 256^3, 4 fields
(u, v, w, p) + 3 previous velocities.  Prints ONE JSON line.

Byte model (each input read once per pass, each output written once):
  fwd reads every field and const (the loss write is 8 bytes); bwd + bc read
  them again and write one gradient per field, so one step moves
  (2 (NF + NC) + NF) * 4 bytes per grid node (72 B/node for the 3D NS case).

The reported figure is the first of --runs runs of K back-to-back steps;
"runs" gives the median and quartiles over all of them (the paper's protocol
takes the median of five).  Beside the warm figure (steps back to back, as a
training loop calls the operator), "flushed" times steps one by one after reading 512 MB between them,
so that every input comes from HBM rather than the 256 MB memory-side cache;
"flushed_dirty" writes the 512 MB instead, so that the step also pays for
writing back the dirty lines that the write leaves in the caches.

--path fused times fpde_residual_value_and_grad, the same loss and gradient
from one read of the inputs ((2 NF + NC) * 4 B/node: 44 for the 3D NS case).

--path residual times the autograd form instead: fwd writing the residual
arrays (every node; zero off the residual set), then fpde_residual_vjp on
resident upstream sensitivities (read on the residual set), reading the fields
the Jacobian depends on and writing every gradient node.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "grid-points/s and achieved HBM GB/s (% of peak) for residual fwd+bwd"


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=None,
                   help="untimed warm-up steps (default: as many as take 0.5 s, at least 50: "
                        "a step back to back with others settles only after ~150 steps; after "
                        "20, the timed NS-3D steps read ~6%% slow)")
    p.add_argument("--config", default="ns_3d_tgv")
    p.add_argument("--seed", type=int, default=42)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-planes", type=int, default=0,
                   help="planes of the oracle sample along axis 0 (0: sized automatically)")
    p.add_argument("--bc-mode", type=int, default=0, choices=(0, 1),
                   help="0: interior residual set (the benchmark); 1: periodic wrap on every axis")
    p.add_argument("--path", default="loss", choices=("loss", "residual", "fused"),
                   help="loss: fwd+loss, bwd, bc (the benchmark); residual: fwd writing R, "
                        "then the explicit-sensitivity backward; fused: the one-pass value "
                        "and gradient")
    p.add_argument("--sample-every", type=int, default=10,
                   help="per-kernel HIP events on every n-th timed step (the others carry none)")
    p.add_argument("--runs", type=int, default=5,
                   help="the K timed steps are the first of this many runs of K steps; the "
                        "line adds the median and quartiles of ms per step over the runs")
    p.add_argument("--flushed-steps", type=int, default=20,
                   help="after the timed region, steps timed one by one with 512 MB read "
                        "(then written) between them (outside the events), so that no input is "
                        "left in the caches; reported beside the warm figure (0: skip)")
    return p.parse_args()


# fields the residual Jacobian depends on (what the explicit-sensitivity backward
# reads besides G): none for the linear operators, the velocity but not the
# pressure for NS
JAC_FIELDS = {1: 1, 2: 0, 3: 0, 4: 2, 5: 3, 6: 3, 7: 0, 8: 0, 9: 2}


def byte_model(wl, bc_mode=0, path="loss"):
    nf, nc, nr = len(wl.spec.fields), len(wl.spec.consts), len(wl.spec.residuals)
    N = wl.n_points
    M = N if bc_mode == 1 else wl.n_residual_points  # nodes the backward writes
    if path == "fused":
        vg = (nf + nc) * 4 * N + nf * 4 * N + 8
        return {"step": vg, "value_and_grad": vg, "per_node": (2 * nf + nc) * 4}
    if path == "residual":
        nfg = JAC_FIELDS[wl.op]
        fwd = (nf + nc + nr) * 4 * N + 8  # + the residual arrays (every node is written)
        vjp = nfg * 4 * N + nr * 4 * M + nf * 4 * N  # fields, G on the residual set, grads
        return {"step": fwd + vjp, "fwd": fwd, "vjp": vjp,
                "per_node": (2 * nf + nc + 2 * nr + nfg) * 4}
    return {
        "step": (2 * (nf + nc) + nf) * 4 * N + 8,
        "fwd": (nf + nc) * 4 * N + 8,
        "bwd": (nf + nc) * 4 * N + nf * 4 * M,
        "per_node": (2 * (nf + nc) + nf) * 4,
    }


def flushed_steps(torch, step, stream, n, flush_bytes=512 << 20, dirty=False):
    """Each of n steps timed alone (events on the step's stream) after a sweep
    over 512 MB that evicts the 256 MB memory-side cache and L2, the sweep
    outside the events: the step's inputs then come from HBM.  The sweep reads
    the buffer (the caches then hold clean lines), or with dirty=True writes it
    (the caches then hold dirty lines, written back while the step runs).
    Median and quartiles of the per-step milliseconds."""
    import statistics  # noqa: PLC0415
    buf = torch.empty(flush_bytes // 4, dtype=torch.float32, device="cuda")
    buf.fill_(1.0)
    ms = []
    for i in range(n):
        with torch.cuda.stream(stream):
            if dirty:
                buf.fill_(float(i))
            else:
                torch.sum(buf)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        b.synchronize()
        ms.append(a.elapsed_time(b))
    del buf
    q = statistics.quantiles(ms, n=4) if len(ms) > 1 else [ms[0]] * 3
    return {"steps": n, "ms_per_step_median": round(q[1], 4), "ms_q1": round(q[0], 4),
            "ms_q3": round(q[2], 4), "flush_bytes": flush_bytes,
            "flush": "write" if dirty else "read"}


def copy_gbps(torch, nbytes=1 << 30, reps=20):
    """Achievable-bandwidth reference: y = 1 * x over 1 GiB (reads 1 GiB, writes
    1 GiB).  Its rocprofv3 FETCH_SIZE / WRITE_SIZE readings calibrate the
    counters for the traffic figure."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    t0 = time.perf_counter()  # warm up for 0.25 s, as the steps do (after idle host work)
    while time.perf_counter() - t0 < 0.25:
        for _ in range(10):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    b.record()
    b.synchronize()
    s = a.elapsed_time(b) / 1e3 / reps
    del src, dst
    return 2 * nbytes / s / 1e9


# the kernels one timed call queues, where it queues several
TRAFFIC_KERNELS = {"value_and_grad": ("fill_f64", "bwd")}
OP_KERNEL_TAG = {1: "OpBurgers", 2: "OpHelmholtz", 3: "OpHeat", 4: "OpNS<2, false>",
                 5: "OpNS<3, true>", 6: "OpNS<3, false>", 7: "OpPoisson<2>", 8: "OpPoisson<3>",
                 9: "OpNST"}


def measured_traffic(cfg, op, kernels, path="loss"):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this
    bench path, summed over `kernels` (name stems such as "bwd", "fill_f64"), if
    it was taken on this workload with the current kernel sources; else None."""
    from paper_2607_18020_amd import profiling  # noqa: PLC0415
    fn = os.path.join(ROOT, "profiles", f"traffic_{path}.json")
    if not os.path.exists(fn):
        return None
    rec = json.load(open(fn))
    if rec.get("source_hash") != profiling.source_hash() or not rec.get("workload", "").startswith(cfg):
        return None
    if rec.get("path") != path:
        return None
    total = 0.0
    for stem in kernels:
        prefix = stem if stem.startswith("fill") else f"{stem}_kernel<{OP_KERNEL_TAG[op]}"
        hits = [v for name, v in rec.get("kernels", {}).items() if name.startswith(prefix)]
        if len(hits) != 1:
            return None
        total += hits[0]["fetch_bytes"] + hits[0]["write_bytes"]
    return round(total)


def cpu_baseline(W, wl_full, cfg, seed, planes, bc_mode=0, path="loss", min_s=10.0, gpu=None):
    """The oracle (single thread, float64) on a slab of the same workload, timed
    over repeated passes totalling at least min_s seconds.  When the slab is the
    whole grid and gpu = (loss, grads) of the timed steps is given (the loss and
    fused paths), the oracle's last pass also checks them: "parity" holds the
    loss's relative error and each gradient's max|err| / max|ref|."""
    import numpy as np  # noqa: PLC0415
    import oracle  # noqa: PLC0415  (CPU baseline leg only)
    shape = wl_full.shape
    if planes <= 0:
        # a slab of at most ~40M nodes (the whole grid for every configured
        # workload; tens of seconds of single-thread oracle work at most)
        per_plane = int(np.prod(shape[1:]))
        planes = max(3, min(shape[0], 40_000_000 // per_plane))
    sl = (slice(0, planes),) + tuple(slice(None) for _ in shape[1:])
    fields = [np.ascontiguousarray(f[sl], dtype=np.float64) for f in wl_full.fields]
    consts = [np.ascontiguousarray(c[sl], dtype=np.float64) for c in wl_full.consts]
    sshape = fields[0].shape
    args = (wl_full.op, sshape, wl_full.h, wl_full.coeffs, fields, consts)
    if path == "residual":
        G = [np.ascontiguousarray(g[sl], dtype=np.float64)
             for g in W.sensitivities(wl_full.op, shape, seed + 1)]

        def one():
            oracle.residual(*args, bc_mode=bc_mode)
            oracle.vjp(*args, G, bc_mode=bc_mode)
        what = "residuals + transposed-Jacobian action"
    else:
        def one():
            return (oracle.loss(*args, bc_mode=bc_mode),
                    oracle.grad(*args, dloss=1.0, bc_mode=bc_mode))
        what = "loss + full gradient"
    # repeated until at least min_s of CPU work has been timed (one pass at least)
    reps, t0 = 0, time.perf_counter()
    while True:
        out = one()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            break
    npts = int(np.prod(sshape))
    res = {"value": npts * reps / dt, "unit": "grid-points/s", "cores": 1, "kind": "oracle",
           "sample": f"{cfg} seed {seed}: first {planes} planes along axis 0 "
                     f"({'x'.join(map(str, sshape))} = {npts} nodes), {what}, "
                     f"float64, single thread, {reps} passes in {dt:.2f} s"}
    if gpu is not None and out is not None and planes == shape[0]:
        L_ref, g_ref = out
        L_gpu, g_gpu = gpu
        res["parity"] = {
            "loss_rel_err": abs(L_gpu - L_ref) / abs(L_ref),
            "grad_max_rel_err": [float(np.abs(a.astype(np.float64) - b).max() / np.abs(b).max())
                                 for a, b in zip(g_gpu, g_ref)],
            "bars": {"loss": 1e-5, "grad": 1e-4}}
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the operator's multi-GPU slab decomposition is a design, not built)",
              file=sys.stderr)
        sys.exit(2)
    import torch  # noqa: PLC0415

    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    from paper_2607_18020_amd import workloads as W  # noqa: PLC0415

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()
    cfg = args.config
    wl = W.make(cfg, seed=args.seed)
    dev = torch.device("cuda:0")
    fields = [torch.from_numpy(f).to(dev) for f in wl.fields]
    consts = [torch.from_numpy(c).to(dev) for c in wl.consts]
    grads = [torch.empty_like(f) for f in fields]
    loss = torch.empty((), dtype=torch.float64, device=dev)
    dl = torch.ones((), dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    op, h, co = wl.op, wl.h, wl.coeffs

    bcm = args.bc_mode

    # the entry points bound once to the resident tensors: each step issues only
    # the C calls (marshalling them in Python every time costs more host time
    # than a small grid's GPU time)
    kw = dict(bc_mode=bcm, stream=stream)
    fwd = B.bind("fwd", op, fields, consts, h, co, loss=loss, **kw)
    bwd = B.bind("bwd", op, fields, consts, h, co, dloss=dl, grads=grads, **kw)
    bc = B.bind("bc", op, fields, consts, h, co, dloss=dl, grads=grads, **kw)
    kernels = (("fwd", fwd), ("bwd", bwd), ("bc", bc))
    if args.path == "residual":
        R = [torch.empty_like(fields[0]) for _ in wl.spec.residuals]
        sens = [torch.from_numpy(g).to(dev) for g in W.sensitivities(op, wl.shape, args.seed + 1)]
        fwd_r = B.bind("fwd", op, fields, consts, h, co, residual_out=R, loss=loss, **kw)
        vjp = B.bind("vjp", op, fields, None, h, co, sens=sens, grads=grads, **kw)
        kernels = (("fwd", fwd_r), ("vjp", vjp))
    if args.path == "fused":
        value_and_grad = B.bind("value_and_grad", op, fields, consts, h, co, dloss=dl, loss=loss,
                                grads=grads, **kw)
        kernels = (("value_and_grad", value_and_grad),)  # (fill and march: one call)
    names = [n for n, _ in kernels]

    def step():
        for _, fn in kernels:
            fn()

    if args.warmup is not None:
        for _ in range(args.warmup):
            step()
        warmup = args.warmup
    else:  # steps in batches of 50 until 0.5 s of them have run
        warmup, t0 = 0, time.perf_counter()
        while warmup < 50 or time.perf_counter() - t0 < 0.5:
            for _ in range(50):
                step()
            warmup += 50
            torch.cuda.synchronize()
    torch.cuda.synchronize()

    # Timed region: K steps between two events.  A timestamp between two kernels
    # costs several microseconds of queue time, so per-kernel events sit on every
    # n-th step only; their averages give the per-kernel durations.
    K = args.steps
    every = max(1, args.sample_every)
    sampled = [k for k in range(K) if k % every == every - 1] or [K - 1]
    ev = {k: [torch.cuda.Event(enable_timing=True) for _ in range(len(kernels) + 1)]
          for k in sampled}
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for k in range(K):
        e = ev.get(k)
        if e is None:
            step()
            continue
        e[0].record(stream)
        for i, (_, fn) in enumerate(kernels):
            fn()
            e[i + 1].record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_s = t_start.elapsed_time(t_end) / 1e3
    per = {n: sum(ev[k][i].elapsed_time(ev[k][i + 1]) for k in sampled) / len(sampled) * 1e3
           for i, n in enumerate(names)}  # microseconds
    L = float(loss.item())
    if not (L == L) or L <= 0:
        raise RuntimeError(f"bad loss {L}")

    bm = byte_model(wl, bcm, args.path)
    N = wl.n_points
    ms = total_s / K * 1e3
    gbps = bm["step"] * K / total_s / 1e9
    dom = max((n for n in names if n in bm), key=lambda n: per[n])
    achieved = bm[dom] / (per[dom] * 1e-6) / 1e9
    roofline = {"bound": "hbm", "kernel": f"{dom} ({cfg})", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(cfg, wl.op, TRAFFIC_KERNELS.get(dom, (dom,)), args.path),
                "algorithmic_bytes_per_launch": bm[dom], "avg_launch_us": round(per[dom], 2)}
    # the same K steps timed again (no per-kernel events), for a median and
    # quartiles over runs beside the one figure the line reports
    run_ms = [ms]
    for _ in range(max(0, args.runs - 1)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(K):
            step()
        b.record(stream)
        b.synchronize()
        run_ms.append(a.elapsed_time(b) / K)
    import statistics  # noqa: PLC0415
    q = statistics.quantiles(run_ms, n=4) if len(run_ms) > 1 else [ms] * 3
    runs = {"n": len(run_ms), "ms_per_step_median": round(q[1], 5), "ms_q1": round(q[0], 5),
            "ms_q3": round(q[2], 5), "ms_per_step": [round(x, 5) for x in run_ms]}
    flushed = flushed_dirty = None
    if args.flushed_steps > 0:
        flushed = flushed_steps(torch, step, stream, args.flushed_steps)
        flushed["grid_points_per_s"] = N / (flushed["ms_per_step_median"] * 1e-3)
        flushed_dirty = flushed_steps(torch, step, stream, args.flushed_steps, dirty=True)
        flushed_dirty["grid_points_per_s"] = N / (flushed_dirty["ms_per_step_median"] * 1e-3)
    cpu = None
    if not args.no_cpu_baseline:
        gpu_out = None
        if args.path in ("loss", "fused"):  # the last timed step's loss and gradient
            gpu_out = (float(loss.item()), [g.cpu().numpy() for g in grads])
        cpu = cpu_baseline(W, wl, cfg, args.seed, args.cpu_planes, bcm, args.path, gpu=gpu_out)
    out = {
        "metric": METRIC,
        "value": N * K / total_s,
        "unit": "grid-points/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg}: {W.CONFIGS[cfg].description}",
                   "grid": list(wl.shape), "nodes": N,
                   "fields": list(wl.spec.fields), "consts": list(wl.spec.consts),
                   "seed": args.seed,
                   "step": {"loss": "fwd+loss, bwd, bc on one stream",
                            "residual": "fwd writing residuals, explicit-sensitivity vjp",
                            "fused": "one-pass loss + gradient (fill, bwd march with loss over every plane)"
                            }[args.path],
                   "path": args.path, "bc_mode": bcm},
        "hbm_gbps": round(gbps, 1),
        "hbm_frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4),
        "bytes_per_step": bm["step"],
        "kernel_us": {k: round(v, 2) for k, v in per.items()},
        "kernel_us_sampled_steps": len(sampled),
        "copy_gbps": round(copy_gbps(torch), 1),
        "runs": runs,
        "flushed": flushed,
        "flushed_dirty": flushed_dirty,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
