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

Protocol (the paper's: median of five runs, Sec. 4.1):
  1. W untimed warm-up steps;
  2. --runs runs of K back-to-back steps, each between two HIP events and
     nothing else: `value` and `ms_per_step` are the MEDIAN run, all runs are
     listed under "runs";
  3. "steady_state": 0.5 s more of untimed steps, then the same runs again.  A
     new load runs slower for its first few tens of ms, and with a short
     warm-up the runs of step 2 fall in that time;
  4. a separate pass per kernel of the step, after step 3: K steps with HIP
     events around that kernel only; its median over the K steps is the
     kernel's duration ("kernel_us"), from which `roofline` is computed for
     the dominant kernel;
  5. "flushed": steps timed one by one after reading 512 MB between them (every
     input then comes from HBM rather than the 256 MB memory-side cache);
     "flushed_dirty" writes the 512 MB instead, so the step also pays for
     writing back the dirty lines the write leaves in the caches;
  6. "workloads" (default config only; --no-workloads skips it): the same
     median-of-runs step time for the other workloads and paths, read-flushed
     steps, and a whole-grid parity check against the oracle for each;
  7. "cpu_baseline": the oracle on all host cores (whole-grid passes, threads
     each running the unchanged single-threaded oracle on an overlapping slab
     of axis 0) and on one core, the last pass checking the GPU's loss and
     gradient ("parity").
The process exits with status 3 after printing the line if any parity check
exceeds its bar.

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
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "grid-points/s and achieved HBM GB/s (% of peak) for residual fwd+bwd"
BARS = {"loss": 1e-5, "residual": 1e-5, "grad": 1e-4}  # max|err| / max|ref|
DEFAULT_CONFIG = "ns_3d_tgv"
# (config, path, bc_mode) of the "workloads" object, beside the headline case
EXTRA_CASES = (("burgers_1dt", "loss", 0), ("helmholtz_2d", "loss", 0), ("heat_3d", "loss", 0),
               ("ns_2d", "loss", 0), ("ns_2d", "fused", 0), ("ns_3d_tgv", "fused", 0),
               ("ns_3d_tgv", "residual", 0), ("ns_3d_tgv", "loss", 1), ("ns_3dt", "loss", 0),
               ("ns_3dt_large", "loss", 0), ("ns_3dt_large", "residual", 0))


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=None,
                   help="untimed warm-up steps (default: as many as take 0.5 s, at least 50)")
    p.add_argument("--config", default=DEFAULT_CONFIG)
    p.add_argument("--seed", type=int, default=42)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the other workloads and paths (the 'workloads' object)")
    p.add_argument("--cpu-planes", type=int, default=0,
                   help="planes of the oracle sample along axis 0 (0: sized automatically)")
    p.add_argument("--bc-mode", type=int, default=0, choices=(0, 1),
                   help="0: interior residual set (the benchmark); 1: periodic wrap on every axis")
    p.add_argument("--path", default="loss", choices=("loss", "residual", "fused"),
                   help="loss: fwd+loss, bwd, bc (the benchmark); residual: fwd writing R, "
                        "then the explicit-sensitivity backward; fused: the one-pass value "
                        "and gradient")
    p.add_argument("--runs", type=int, default=5,
                   help="runs of K timed steps; the line reports the median run")
    p.add_argument("--flushed-steps", type=int, default=20,
                   help="steps timed one by one with 512 MB read (then written) between them, "
                        "outside the events (0: skip)")
    return p.parse_args()


# fields the residual Jacobian depends on (what the explicit-sensitivity backward
# reads besides G): none for the linear operators, the velocity but not the
# pressure for NS
JAC_FIELDS = {1: 1, 2: 0, 3: 0, 4: 2, 5: 3, 6: 3, 7: 0, 8: 0, 9: 2, 10: 3}


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


def _quartiles(xs):
    if len(xs) == 1:
        return xs[0], xs[0], xs[0]
    q = statistics.quantiles(xs, n=4)
    return q[0], statistics.median(xs), q[2]


# --------------------------------------------------------------------------- the GPU side


class Case:
    """One workload and path bound to resident device tensors: `calls` are the
    (name, bound entry point) pairs one step queues on one stream."""

    def __init__(self, torch, B, W, cfg, seed, path, bc_mode):
        self.torch, self.cfg, self.path, self.bc_mode = torch, cfg, path, bc_mode
        self.wl = wl = W.make(cfg, seed=seed)
        dev = torch.device("cuda:0")
        self.fields = [torch.from_numpy(f).to(dev) for f in wl.fields]
        self.consts = [torch.from_numpy(c).to(dev) for c in wl.consts]
        # every output written once before the first step (no first-touch inside the timing)
        self.grads = [torch.zeros_like(f) for f in self.fields]
        self.loss = torch.zeros((), dtype=torch.float64, device=dev)
        self.dl = torch.ones((), dtype=torch.float64, device=dev)
        self.stream = s = torch.cuda.current_stream()
        op, h, co, f, c = wl.op, wl.h, wl.coeffs, self.fields, self.consts
        kw = dict(bc_mode=bc_mode, stream=s)
        self.R = self.sens = None
        if path == "residual":
            self.R = [torch.zeros_like(f[0]) for _ in wl.spec.residuals]
            self.sens = [torch.from_numpy(g).to(dev)
                         for g in W.sensitivities(op, wl.shape, seed + 1)]
            self.calls = (("fwd", B.bind("fwd", op, f, c, h, co, residual_out=self.R,
                                         loss=self.loss, **kw)),
                          ("vjp", B.bind("vjp", op, f, None, h, co, sens=self.sens,
                                         grads=self.grads, **kw)))
        elif path == "fused":
            self.calls = (("value_and_grad", B.bind("value_and_grad", op, f, c, h, co,
                                                    dloss=self.dl, loss=self.loss,
                                                    grads=self.grads, **kw)),)
        else:
            self.calls = (("fwd", B.bind("fwd", op, f, c, h, co, loss=self.loss, **kw)),
                          ("bwd", B.bind("bwd", op, f, c, h, co, dloss=self.dl, grads=self.grads,
                                         **kw)),
                          ("bc", B.bind("bc", op, f, c, h, co, dloss=self.dl, grads=self.grads,
                                        **kw)))
        self.names = [n for n, _ in self.calls]
        self.bm = byte_model(wl, bc_mode, path)

    def step(self):
        for _, fn in self.calls:
            fn()

    def _event(self):
        return self.torch.cuda.Event(enable_timing=True)

    def warm(self, steps=None, seconds=0.5):
        """`steps` untimed steps, or (steps None) batches of 50 for `seconds`."""
        torch = self.torch
        if steps is not None:
            for _ in range(steps):
                self.step()
            torch.cuda.synchronize()
            return steps
        n, t0 = 0, time.perf_counter()
        while n < 50 or time.perf_counter() - t0 < seconds:
            for _ in range(50):
                self.step()
            n += 50
            torch.cuda.synchronize()
        return n

    def runs(self, K, n):
        """n runs of K back-to-back steps, two events each: ms per step of every run."""
        torch = self.torch
        out = []
        for _ in range(n):
            a, b = self._event(), self._event()
            torch.cuda.synchronize()
            a.record(self.stream)
            for _ in range(K):
                self.step()
            b.record(self.stream)
            b.synchronize()
            out.append(a.elapsed_time(b) / K)
        return out

    def kernel_medians(self, K):
        """For each call of the step, K steps with events around that call only:
        its median duration in microseconds."""
        torch = self.torch
        med = {}
        for i, name in enumerate(self.names):
            ev = [(self._event(), self._event()) for _ in range(K)]
            torch.cuda.synchronize()
            for k in range(K):
                for j, (_, fn) in enumerate(self.calls):
                    if j == i:
                        ev[k][0].record(self.stream)
                        fn()
                        ev[k][1].record(self.stream)
                    else:
                        fn()
            torch.cuda.synchronize()
            med[name] = statistics.median(a.elapsed_time(b) for a, b in ev) * 1e3
        return med

    def flushed(self, n, flush_bytes=512 << 20, dirty=False):
        """Each of n steps timed alone after a sweep over 512 MB that evicts the
        memory-side cache and L2 (the sweep outside the events): reading the
        buffer leaves clean lines, writing it dirty ones that are written back
        while the step runs.  Median and quartiles of ms per step."""
        torch = self.torch
        buf = torch.empty(flush_bytes // 4, dtype=torch.float32, device="cuda")
        buf.fill_(1.0)
        ms = []
        for i in range(n):
            with torch.cuda.stream(self.stream):
                if dirty:
                    buf.fill_(float(i))
                else:
                    torch.sum(buf)
            a, b = self._event(), self._event()
            a.record(self.stream)
            self.step()
            b.record(self.stream)
            b.synchronize()
            ms.append(a.elapsed_time(b))
        del buf
        q1, q2, q3 = _quartiles(ms)
        return {"steps": n, "ms_per_step_median": round(q2, 4), "ms_q1": round(q1, 4),
                "ms_q3": round(q3, 4), "flush_bytes": flush_bytes,
                "flush": "write" if dirty else "read",
                "grid_points_per_s": self.wl.n_points / (q2 * 1e-3)}

    def outputs(self):
        """(loss, grads, residuals) of the last step, on the host."""
        self.torch.cuda.synchronize()
        R = [r.cpu().numpy() for r in self.R] if self.R is not None else None
        return float(self.loss.item()), [g.cpu().numpy() for g in self.grads], R

    def release(self):
        for name in ("fields", "consts", "grads", "R", "sens", "calls"):
            setattr(self, name, None)
        self.torch.cuda.empty_cache()


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
                 9: "OpNST", 10: "OpNS3T"}


def measured_traffic(cfg, op, kernels, path="loss"):
    """HBM bytes per launch from the committed rocprofv3 counter summary of this
    workload and bench path (profiles/traffic_*.json), summed over `kernels`
    (name stems such as "bwd", "fill_f64"), if it was taken with the current
    kernel sources; else None."""
    import glob  # noqa: PLC0415

    from paper_2607_18020_amd import profiling  # noqa: PLC0415
    rec = None
    for fn in sorted(glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json"))):
        r = json.load(open(fn))
        if r.get("path") == path and r.get("workload", "").split(" ")[0] == cfg:
            rec = r
    if rec is None or rec.get("source_hash") != profiling.source_hash():
        return None
    total = 0.0
    for stem in kernels:
        prefix = stem if stem.startswith("fill") else f"{stem}_kernel<{OP_KERNEL_TAG[op]}"
        hits = [v for name, v in rec.get("kernels", {}).items() if name.startswith(prefix)]
        if len(hits) != 1:
            return None
        total += hits[0]["fetch_bytes"] + hits[0]["write_bytes"]
    return round(total)


# --------------------------------------------------------------------------- the CPU side


def _rel(a, b):
    import numpy as np  # noqa: PLC0415
    s = float(np.abs(b).max())
    e = float(np.abs(np.asarray(a, dtype=np.float64) - b).max())
    return e / s if s > 0 else e


def _oracle_whole(wl, bc_mode, path, seed, W):
    """The oracle on the whole grid (float64, single thread): what the GPU path
    computes for this case, for the parity check."""
    import oracle  # noqa: PLC0415  (CPU baseline / parity leg only)
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    if path == "residual":
        G = W.sensitivities(wl.op, wl.shape, seed + 1)
        return {"R": oracle.residual(*args, bc_mode=bc_mode),
                "grads": oracle.vjp(*args, G, bc_mode=bc_mode)}
    return {"loss": oracle.loss(*args, bc_mode=bc_mode),
            "grads": oracle.grad(*args, dloss=1.0, bc_mode=bc_mode)}


def parity_of(gpu, ref):
    """Max errors of the GPU outputs (loss, grads, R) against the oracle's,
    relative to max|ref|, with the bars and a verdict."""
    L, g, R = gpu
    out = {}
    if "loss" in ref:
        out["loss_rel_err"] = abs(L - ref["loss"]) / abs(ref["loss"])
    if "R" in ref and R is not None:
        out["residual_max_rel_err"] = [_rel(a, b) for a, b in zip(R, ref["R"])]
    out["grad_max_rel_err"] = [_rel(a, b) for a, b in zip(g, ref["grads"])]
    ok = out.get("loss_rel_err", 0.0) <= BARS["loss"] and \
        all(e <= BARS["residual"] for e in out.get("residual_max_rel_err", [])) and \
        all(e <= BARS["grad"] for e in out["grad_max_rel_err"])
    out["bars"] = BARS
    out["ok"] = bool(ok)
    return out


def _slab_pass(oracle, wl, bc_mode, a, b):
    """Loss part and gradient of planes [a, b) of axis 0 from the unchanged
    single-threaded oracle on the slab [a - 2, b + 2) (wrapped on a periodic
    grid): the gradient at a node depends on the inputs within two nodes, so the
    slab's gradient on [a, b) is the whole grid's (with the whole grid's 1/M).
    Returns (sum of R^2 over the residual nodes of [a, b), gradient of [a, b))."""
    import numpy as np  # noqa: PLC0415
    n0 = wl.shape[0]
    if bc_mode == 1:
        idx = np.arange(a - 2, b + 2) % n0
        lo = 2
    else:
        s, e = max(0, a - 2), min(n0, b + 2)
        idx = np.arange(s, e)
        lo = a - s
    F = [np.ascontiguousarray(f[idx], dtype=np.float64) for f in wl.fields]
    C = [np.ascontiguousarray(c[idx], dtype=np.float64) for c in wl.consts]
    sshape = F[0].shape
    args = (wl.op, sshape, wl.h, wl.coeffs, F, C)
    M_full = wl.n_points if bc_mode == 1 else wl.n_residual_points
    M_slab = int(np.prod(sshape)) if bc_mode == 1 else int(np.prod([n - 2 for n in sshape]))
    R = oracle.residual(*args, bc_mode=bc_mode)
    own = slice(lo, lo + (b - a))
    ss = sum(float(np.sum(r[own] ** 2)) for r in R)  # zero off the residual set
    g = oracle.grad(*args, dloss=M_slab / M_full, bc_mode=bc_mode)  # scale 2 / M_full
    return ss, [x[own] for x in g]


def oracle_all_cores(wl, bc_mode, cores, min_s=5.0):
    """Whole-grid loss + gradient passes with `cores` threads, each calling the
    unchanged single-threaded oracle on an overlapping slab of axis 0 (the
    oracle is a C library; ctypes releases the interpreter lock during the
    call).  Repeated for at least min_s.  Returns (grid-points/s, passes,
    seconds, (loss, grads) of the last pass)."""
    import numpy as np  # noqa: PLC0415
    from concurrent.futures import ThreadPoolExecutor  # noqa: PLC0415

    import oracle  # noqa: PLC0415  (CPU baseline leg only)
    n0 = wl.shape[0]
    nsl = max(1, min(cores, n0))
    cuts = [round(i * n0 / nsl) for i in range(nsl + 1)]
    M_full = wl.n_points if bc_mode == 1 else wl.n_residual_points
    out = None
    with ThreadPoolExecutor(max_workers=cores) as ex:
        reps, t0 = 0, time.perf_counter()
        while True:
            parts = list(ex.map(lambda i: _slab_pass(oracle, wl, bc_mode, cuts[i], cuts[i + 1]),
                                range(nsl)))
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= min_s:
                break
    L = sum(p[0] for p in parts) / M_full
    grads = [np.concatenate([p[1][f] for p in parts], axis=0) for f in range(len(wl.fields))]
    out = (L, grads)
    return wl.n_points * reps / dt, reps, dt, out


def oracle_one_core(wl, bc_mode, path, seed, W, min_s=10.0):
    """Whole-grid passes of the unchanged oracle on one thread, for at least
    min_s.  Returns (grid-points/s, passes, seconds, oracle outputs of the last pass)."""
    reps, t0 = 0, time.perf_counter()
    while True:
        ref = _oracle_whole(wl, bc_mode, path, seed, W)
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            break
    return wl.n_points * reps / dt, reps, dt, ref


def host_cores():
    """Host cores this process may use, at most 16 (the host's share for one GPU
    on an eight-GPU machine)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def cpu_baseline(case, W, seed, gpu_out):
    """The oracle timed on the host beside the GPU run: all cores (the figure)
    and one core, both whole-grid passes; the one-core pass also checks the
    GPU's outputs of the timed steps."""
    wl, bcm, path = case.wl, case.bc_mode, case.path
    cores = host_cores()
    what = {"loss": "loss + full gradient", "fused": "loss + full gradient",
            "residual": "residuals + transposed-Jacobian action"}[path]
    res = {"unit": "grid-points/s", "kind": "oracle"}
    if path != "residual":
        v, reps, dt, _ = oracle_all_cores(wl, bcm, cores)
        res.update({"value": v, "cores": cores,
                    "sample": f"{case.cfg} seed {seed}: the whole grid "
                              f"({'x'.join(map(str, wl.shape))} = {wl.n_points} nodes), {what}, "
                              f"float64; {cores} threads each running the single-threaded oracle "
                              f"on an overlapping slab of axis 0; {reps} passes in {dt:.2f} s"})
    v1, reps1, dt1, ref = oracle_one_core(wl, bcm, path, seed, W)
    one = {"value": v1, "unit": "grid-points/s", "cores": 1, "kind": "oracle",
           "sample": f"{case.cfg} seed {seed}: the whole grid ({wl.n_points} nodes), {what}, "
                     f"float64, one thread, {reps1} passes in {dt1:.2f} s"}
    if path == "residual":  # the all-core split is for the loss and its gradient only
        res.update(one)
    else:
        res["single_core"] = one
    res["parity"] = parity_of(gpu_out, ref)
    return res


# --------------------------------------------------------------------------- main


def measure(case, K, runs, warmup):
    """Warm-up, the median-of-runs step time and the per-kernel medians."""
    w = case.warm(steps=warmup)
    run_ms = case.runs(K, runs)
    kus = case.kernel_medians(K)
    q1, med, q3 = _quartiles(run_ms)
    return w, run_ms, med, q1, q3, kus


def workloads_object(torch, B, W, seed, K, runs):
    """The other workloads and paths: median-of-runs step time, grid-points/s,
    byte-model bandwidth and whole-grid parity against the oracle."""
    out = {}
    for cfg, path, bcm in EXTRA_CASES:
        key = f"{cfg}/{path}/bc{bcm}"
        case = Case(torch, B, W, cfg, seed, path, bcm)
        # small grids: more steps per run so that a run spans at least ~20 ms
        k = K
        w, run_ms, med, q1, q3, kus = measure(case, k, runs, None)
        if med * k < 20.0:
            k = int(min(2000, max(K, 20.0 / med)))
            w2, run_ms, med, q1, q3, kus = measure(case, k, runs, 0)
        bm = case.bm
        # steps one by one after a 512 MB read: inputs from HBM, not from the
        # memory-side cache (the grids of 2-D workloads fit in it)
        fl = case.flushed(20)
        gpu_out = case.outputs()
        t0 = time.perf_counter()
        ref = _oracle_whole(case.wl, bcm, path, seed, W)
        rec = {"grid": list(case.wl.shape), "nodes": case.wl.n_points, "steps": k,
               "warmup": w, "ms_per_step": round(med, 5), "ms_q1": round(q1, 5),
               "ms_q3": round(q3, 5), "ms_per_step_runs": [round(x, 5) for x in run_ms],
               "grid_points_per_s": case.wl.n_points / (med * 1e-3),
               "bytes_per_step": bm["step"], "hbm_gbps": round(bm["step"] / (med * 1e-3) / 1e9, 1),
               "hbm_frac_of_peak": round(bm["step"] / (med * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
               "kernel_us": {n: round(v, 2) for n, v in kus.items()},
               "flushed_read": {
                   "steps": fl["steps"], "ms_per_step_median": fl["ms_per_step_median"],
                   "ms_q1": fl["ms_q1"], "ms_q3": fl["ms_q3"],
                   "hbm_frac_of_peak": round(bm["step"] / (fl["ms_per_step_median"] * 1e-3) / 1e9
                                             / HBM_PEAK_GBPS, 4)},
               "parity": parity_of(gpu_out, ref), "oracle_s": round(time.perf_counter() - t0, 2)}
        out[key] = rec
        case.release()
        print(f"bench: {key} {med:.4f} ms/step, parity ok={rec['parity']['ok']}",
              file=sys.stderr, flush=True)
    return out


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
    cfg, bcm, K = args.config, args.bc_mode, args.steps
    case = Case(torch, B, W, cfg, args.seed, args.path, bcm)
    # the headline: W warm-up steps, then the median of the runs of K steps
    warmup = case.warm(steps=args.warmup)
    run_ms = case.runs(K, args.runs)
    q1, med, q3 = _quartiles(run_ms)
    # the same runs once the GPU has settled on this load (the first few tens of
    # ms of a new load run slower), then the per-kernel pass in that state
    steady_warm = case.warm(seconds=0.5)
    steady_ms = case.runs(K, args.runs)
    sq1, smed, sq3 = _quartiles(steady_ms)
    kus = case.kernel_medians(K)
    L = float(case.loss.item())
    if not (L == L) or L <= 0:
        raise RuntimeError(f"bad loss {L}")
    bm, N = case.bm, case.wl.n_points
    gbps = bm["step"] / (med * 1e-3) / 1e9
    dom = max((n for n in case.names if n in bm), key=lambda n: kus[n])
    achieved = bm[dom] / (kus[dom] * 1e-6) / 1e9
    roofline = {"bound": "hbm", "kernel": f"{dom} ({cfg})", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(cfg, case.wl.op, TRAFFIC_KERNELS.get(dom, (dom,)),
                                            args.path),
                "algorithmic_bytes_per_launch": bm[dom], "avg_launch_us": round(kus[dom], 2),
                "timing": f"median over {K} steps, HIP events around this kernel only, "
                          "after the steady-state runs"}
    ksum = sum(kus.values())
    flushed = flushed_dirty = None
    if args.flushed_steps > 0:
        flushed = case.flushed(args.flushed_steps)
        flushed_dirty = case.flushed(args.flushed_steps, dirty=True)
    gpu_out = case.outputs()
    cgbps = round(copy_gbps(torch), 1)
    extra = None
    if not args.no_workloads and cfg == DEFAULT_CONFIG and args.path == "loss" and bcm == 0:
        extra = workloads_object(torch, B, W, args.seed, K, args.runs)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(case, W, args.seed, gpu_out)
    out = {
        "metric": METRIC,
        "value": N / (med * 1e-3),
        "unit": "grid-points/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": warmup,
        "ms_per_step": med,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg}: {W.CONFIGS[cfg].description}",
                   "grid": list(case.wl.shape), "nodes": N,
                   "fields": list(case.wl.spec.fields), "consts": list(case.wl.spec.consts),
                   "seed": args.seed,
                   "step": {"loss": "fwd+loss, bwd, bc on one stream",
                            "residual": "fwd writing residuals, explicit-sensitivity vjp",
                            "fused": "one-pass loss + gradient (fill, bwd march with loss over every plane)"
                            }[args.path],
                   "path": args.path, "bc_mode": bcm},
        "hbm_gbps": round(gbps, 1),
        "hbm_frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4),
        "bytes_per_step": bm["step"],
        "runs": {"n": len(run_ms), "statistic": "median", "ms_per_step": [round(x, 5) for x in run_ms],
                 "ms_q1": round(q1, 5), "ms_q3": round(q3, 5)},
        "kernel_us": {k: round(v, 2) for k, v in kus.items()},
        "steady_state": {"warm_steps": steady_warm, "statistic": "median",
                         "ms_per_step": round(smed, 5),
                         "ms_per_step_runs": [round(x, 5) for x in steady_ms],
                         "ms_q1": round(sq1, 5), "ms_q3": round(sq3, 5),
                         "grid_points_per_s": N / (smed * 1e-3),
                         "hbm_frac_of_peak": round(bm["step"] / (smed * 1e-3) / 1e9
                                                   / HBM_PEAK_GBPS, 4)},
        "kernel_us_check": {"sum_us": round(ksum, 2), "step_us": round(med * 1e3, 2),
                            "sum_le_step": bool(ksum <= med * 1e3),
                            "steady_step_us": round(smed * 1e3, 2),
                            "note": "events around one call also time its dispatch gap, and "
                                    "the forward's call launches the loss fill too, so the sum "
                                    "can exceed a back-to-back step by a few per cent"},
        "copy_gbps": cgbps,
        "flushed": flushed,
        "flushed_dirty": flushed_dirty,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "workloads": extra,
    }
    print(json.dumps(out), flush=True)
    checks = ([cpu["parity"]["ok"]] if cpu else []) + \
        ([r["parity"]["ok"] for r in extra.values()] if extra else [])
    if not all(checks):
        print("bench.py: a parity check exceeded its bar", file=sys.stderr)
        sys.exit(3)


if __name__ == "__main__":
    main()
