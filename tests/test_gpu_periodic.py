"""GPU parity for periodic grids (bc_mode 1): every axis wraps, every node is a
residual node (M = N), the backward writes every node and the boundary
correction has nothing to do.  Compared with the oracle's periodic mode, element
by element."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

# several tiles along every axis, ragged last tiles (the lane past the last
# column must carry the wrapped residual), chunk seams along axis 0
CASES = [
    ("burgers_1dt", (5, 7)), ("burgers_1dt", (41, 300)),
    ("helmholtz_2d", (3, 3)), ("helmholtz_2d", (4, 259)), ("helmholtz_2d", (67, 513)),
    ("heat_3d", (3, 3, 3)), ("heat_3d", (5, 6, 7)), ("heat_3d", (19, 21, 70)),
    ("heat_3d", (9, 10, 300)),
    ("ns_2d", (6, 257)), ("ns_2d", (71, 600)),
    ("ns_3d_tgv", (3, 3, 3)), ("ns_3d_tgv", (4, 9, 66)), ("ns_3d_tgv", (19, 21, 70)),
    ("ns_3d_tgv", (40, 17, 129)), ("ns_3d_tgv", (7, 9, 300)), ("ns_3d_tgv", (42, 256, 256)),
    # tall 2-D grids: chunks of 14 rows, several passes of the unrolled row queue
    ("ns_2d", (13400, 40)), ("burgers_1dt", (20000, 30)),
]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


def _compare(oracle_mod, wl, dloss, what):
    R, L, g = H.run_gpu(wl, dloss=dloss, bc_mode=1)
    Rr = oracle_mod.residual(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, bc_mode=1)
    Lr = oracle_mod.loss(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, bc_mode=1)
    gr = oracle_mod.grad(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, dloss=dloss,
                         bc_mode=1)
    for b, (a, r) in enumerate(zip(R, Rr)):
        assert np.all(np.isfinite(a)), f"{what}: residual {b} not written everywhere"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_RES, f"{what}: residual {b} rel err {e:.3e}"
    assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (what, L, Lr)
    for f, (a, r) in enumerate(zip(g, gr)):
        assert np.all(np.isfinite(a)), f"{what}: grad {f} not written everywhere"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"


@pytest.mark.parametrize("cfg,shape", CASES, ids=[f"{c}-{'x'.join(map(str, s))}" for c, s in CASES])
def test_periodic_parity(oracle_mod, cfg, shape):
    wl = W.make(cfg, seed=43, shape=shape)
    print(f"case periodic {cfg} {shape}", flush=True)
    _compare(oracle_mod, wl, 0.7, f"periodic {cfg}{shape}")


@pytest.mark.parametrize("op", sorted(W.OPS))
def test_periodic_normal_inputs(oracle_mod, op):
    """The paper's N(0,1) verification inputs, on a wrapped grid."""
    shape = H.normal_shape(op)
    wl = W.normal_fields(op, shape, 44)
    print(f"case periodic op={op} {shape}", flush=True)
    _compare(oracle_mod, wl, 1.0, f"periodic normal op{op}")


def test_periodic_bwd_writes_every_node_and_bc_nothing():
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    for cfg, shape in (("ns_3d_tgv", (9, 12, 70)), ("ns_2d", (9, 260)), ("heat_3d", (3, 3, 3))):
        wl = W.make(cfg, seed=45, shape=shape)
        fields = [torch.from_numpy(f).cuda() for f in wl.fields]
        consts = [torch.from_numpy(c).cuda() for c in wl.consts]
        dl = torch.ones((), dtype=torch.float64, device="cuda")
        g = [torch.full_like(f, float("nan")) for f in fields]
        B.fpde_residual_bwd(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=g, bc_mode=1)
        torch.cuda.synchronize()
        assert all(torch.isfinite(x).all() for x in g)
        g = [torch.full_like(f, float("nan")) for f in fields]
        B.fpde_bc_correct(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=g, bc_mode=1)
        torch.cuda.synchronize()
        assert all(torch.isnan(x).all() for x in g)


@pytest.mark.parametrize("seed", [42, 43, 44, 45, 46])
def test_periodic_full_size_ns3d(oracle_mod, seed):
    """The 256^3 Taylor-Green workload on the wrapped grid, every node, for the
    paper's seeds."""
    wl = W.make("ns_3d_tgv", seed=seed)
    print(f"case periodic full ns_3d_tgv {wl.shape} seed {seed}", flush=True)
    _compare(oracle_mod, wl, 1.0, "periodic full ns_3d_tgv")
