"""GPU parity of the adjacent operators (steady 3D NS, 2D and 3D Poisson,
unsteady 2D and 3D NS on space-time grids): every entry point against the oracle,
node by node, in both boundary modes, on small, ragged and multi-chunk grids
and on the full-size workloads."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

CASES = [
    ("ns_3d_steady", (3, 3, 3)), ("ns_3d_steady", (5, 9, 66)), ("ns_3d_steady", (19, 21, 70)),
    ("ns_3d_steady", (40, 17, 129)), ("ns_3d_steady", (7, 9, 300)),
    ("poisson_2d", (3, 3)), ("poisson_2d", (5, 7)), ("poisson_2d", (41, 300)),
    ("poisson_2d", (67, 513)),
    ("poisson_3d", (3, 3, 3)), ("poisson_3d", (5, 6, 7)), ("poisson_3d", (19, 21, 70)),
    ("poisson_3d", (9, 10, 300)), ("poisson_3d", (42, 256, 256)),
    ("ns_2dt", (3, 3, 3)), ("ns_2dt", (4, 9, 66)), ("ns_2dt", (19, 21, 70)),
    ("ns_2dt", (40, 17, 129)), ("ns_2dt", (7, 9, 300)), ("ns_2dt", (42, 256, 256)),
    # 3D+t: several time levels, several tiles and chunks of each level, ragged tails
    ("ns_3dt", (3, 3, 3, 3)), ("ns_3dt", (4, 5, 9, 66)), ("ns_3dt", (6, 19, 21, 70)),
    ("ns_3dt", (5, 12, 17, 129)), ("ns_3dt", (4, 7, 9, 300)), ("ns_3dt", (9, 40, 20, 33)),
]
IDS = [f"{c}-{'x'.join(map(str, s))}" for c, s in CASES]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


def _dev(arrs):
    import torch  # noqa: PLC0415
    return [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in arrs]


def _ref(oracle_mod, wl, dloss, bc_mode):
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    return (oracle_mod.residual(*args, bc_mode=bc_mode), oracle_mod.loss(*args, bc_mode=bc_mode),
            oracle_mod.grad(*args, dloss=dloss, bc_mode=bc_mode))


def _check_grads(g, gr, what):
    for f, (a, r) in enumerate(zip(g, gr)):
        assert np.all(np.isfinite(a)), f"{what}: grad {f} has unwritten nodes"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape", CASES, ids=IDS)
def test_adjacent_fwd_bwd_bc(oracle_mod, cfg, shape, bc_mode):
    wl = W.make(cfg, seed=71, shape=shape)
    print(f"case adjacent {cfg} {shape} bc_mode={bc_mode}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=0.6, bc_mode=bc_mode)
    Rr, Lr, gr = _ref(oracle_mod, wl, 0.6, bc_mode)
    what = f"{cfg}{shape} bc{bc_mode}"
    if bc_mode == 0:
        H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=what)
        return
    for b, (a, r) in enumerate(zip(R, Rr)):
        assert H.max_rel_err(a, r) <= H.TOL_RES, (what, b)
    assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (what, L, Lr)
    _check_grads(g, gr, what)


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape", CASES, ids=IDS)
def test_adjacent_vjp_and_value_and_grad(oracle_mod, cfg, shape, bc_mode):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make(cfg, seed=72, shape=shape)
    G = W.sensitivities(wl.op, shape, 73)
    print(f"case adjacent vjp/vg {cfg} {shape} bc_mode={bc_mode}", flush=True)
    fields, consts, sens = _dev(wl.fields), _dev(wl.consts), _dev(G)
    gv = [torch.full_like(f, float("nan")) for f in fields]
    B.fpde_residual_vjp(wl.op, fields, wl.h, wl.coeffs, sens, grads=gv, bc_mode=bc_mode)
    gf = [torch.full_like(f, float("nan")) for f in fields]
    loss = torch.full((), float("nan"), dtype=torch.float64, device="cuda")
    dl = torch.tensor(0.6, dtype=torch.float64, device="cuda")
    B.fpde_residual_value_and_grad(wl.op, fields, consts, wl.h, wl.coeffs, dl, loss=loss,
                                   grads=gf, bc_mode=bc_mode)
    torch.cuda.synchronize()
    args = (wl.op, shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    what = f"{cfg}{shape} bc{bc_mode}"
    _check_grads([x.cpu().numpy() for x in gv], oracle_mod.vjp(*args, G, bc_mode=bc_mode),
                 "vjp " + what)
    Lr = oracle_mod.loss(*args, bc_mode=bc_mode)
    assert abs(loss.item() - Lr) <= H.TOL_RES * abs(Lr), (what, loss.item(), Lr)
    _check_grads([x.cpu().numpy() for x in gf],
                 oracle_mod.grad(*args, dloss=0.6, bc_mode=bc_mode), "value_and_grad " + what)


@pytest.mark.parametrize("op", [W.NS_3D_STEADY, W.POISSON_2D, W.POISSON_3D, W.NS_2DT, W.NS_3DT])
def test_adjacent_normal_inputs(oracle_mod, op):
    """N(0,1) fields (the paper's verification inputs), seeds 42-46."""
    shape = H.normal_shape(op)
    for seed in (42, 43, 44, 45, 46):
        wl = W.normal_fields(op, shape, seed)
        print(f"case adjacent normal op={op} seed={seed}", flush=True)
        R, L, g = H.run_gpu(wl, dloss=1.0)
        Rr, Lr, gr = _ref(oracle_mod, wl, 1.0, 0)
        H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"normal op{op} seed{seed}")


@pytest.mark.parametrize("cfg", list(W.ADJACENT_CONFIGS))
def test_adjacent_full_size_every_node(oracle_mod, cfg):
    """The full-size adjacent workloads, compared node by node."""
    wl = W.make(cfg, seed=42)
    print(f"case adjacent full {cfg} {wl.shape}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=1.0)
    Rr, Lr, gr = _ref(oracle_mod, wl, 1.0, 0)
    H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"full {cfg}")
