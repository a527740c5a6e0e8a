"""A NaN in one input node stays local: the operator reads a node's radius-1
star for a residual, and the gradient at a node gathers residuals of its own
star, so a NaN at node n0 reaches the residuals within Manhattan distance 1 of
n0 and the gradients within distance 2 (the loss, a sum over every residual,
is NaN).  Every other output is what the same call gives without the NaN.
Inputs are not checked for NaN or Inf; this is how they propagate, in the
oracle (CPU) and in the HIP path (GPU)."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W

CASES = [("ns_3d_tgv", (12, 14, 70)), ("heat_3d", (9, 10, 40)), ("ns_2d", (30, 300)),
         ("burgers_1dt", (20, 40))]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


def _with_nan(cfg, shape, field):
    wl = W.make(cfg, seed=47, shape=shape)
    n0 = tuple(n // 2 for n in shape)
    fields = [f.copy() for f in wl.fields]
    fields[field][n0] = np.float32(np.nan)
    dist = sum(np.abs(np.arange(n) - c).reshape([-1 if a == k else 1 for k in range(len(shape))])
               for a, (n, c) in enumerate(zip(shape, n0)))
    return wl, fields, n0, dist


@pytest.mark.parametrize("cfg,shape", CASES, ids=[c for c, _ in CASES])
def test_oracle_nan_input_stays_local(oracle_mod, cfg, shape):
    wl, fields, n0, dist = _with_nan(cfg, shape, field=0)
    o = oracle_mod
    R0 = o.residual(wl.op, shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    g0 = o.grad(wl.op, shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    R = o.residual(wl.op, shape, wl.h, wl.coeffs, fields, wl.consts)
    g = o.grad(wl.op, shape, wl.h, wl.coeffs, fields, wl.consts)
    assert np.isnan(o.loss(wl.op, shape, wl.h, wl.coeffs, fields, wl.consts))
    assert np.isnan(R[0][n0]) and np.isnan(g[0][n0])
    for r, r0 in zip(R, R0):
        assert not np.isnan(r[dist > 1]).any()
        assert np.array_equal(r[dist > 1], r0[dist > 1])
    for x, x0 in zip(g, g0):
        assert not np.isnan(x[dist > 2]).any()
        assert np.array_equal(x[dist > 2], x0[dist > 2])


@pytest.mark.gpu
@pytest.mark.parametrize("cfg,shape", CASES, ids=[c for c, _ in CASES])
def test_gpu_nan_input_stays_local(oracle_mod, cfg, shape):
    from tests import gpu_helpers as H  # noqa: PLC0415
    wl, fields, n0, dist = _with_nan(cfg, shape, field=0)
    print(f"case nan input {cfg} {shape} at {n0}", flush=True)
    R0, _, g0 = oracle_mod.on_workload(wl)  # the clean inputs
    R, L, g = H.run_gpu(dataclasses.replace(wl, fields=fields))
    assert np.isnan(L)
    assert np.isnan(R[0][n0]) and np.isnan(g[0][n0])
    sm = H.shell_mask(shape)
    for r, r0 in zip(R, R0):
        assert not np.isnan(r[dist > 1]).any()
        far = (dist > 1) & ~sm
        scale = float(np.abs(r0[~sm]).max())
        assert float(np.abs(r[far] - r0[far]).max()) <= H.TOL_RES * scale
    for x, x0 in zip(g, g0):
        assert not np.isnan(x[dist > 2]).any()
        far = dist > 2
        scale = float(np.abs(x0).max())
        assert float(np.abs(x[far] - x0[far]).max()) <= H.TOL_GRAD * scale
