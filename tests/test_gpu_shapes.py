"""GPU parity on seeded random grid shapes.

For every operator, grids whose extents are drawn from a seeded generator
(small enough for the oracle to run in milliseconds, and ragged against the
tile widths, chunk lengths, row segments and time levels the kernels use), in
both boundary modes, through every entry point: the forward's loss and
residuals, bwd + bc, the one-pass value and gradient, and the
explicit-sensitivity backward, each compared with the oracle node by node.
Inputs: the paper's N(0,1) verification fields (App. A.7)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

MAX_NODES = 60_000
PER_OP = 6
# extent ranges by rank (log-uniform): the last axis spans the row segments and
# tile widths, the others several tiles, chunks and time levels
RANGES = {2: ((3, 80), (3, 1500)), 3: ((3, 30), (3, 48), (3, 320)),
          4: ((3, 8), (3, 18), (3, 24), (3, 150))}


def _shapes(op):
    rng = np.random.default_rng(2607 + op)
    out = []
    while len(out) < PER_OP:
        shape = tuple(int(round(np.exp(rng.uniform(np.log(lo), np.log(hi)))))
                      for lo, hi in RANGES[W.OPS[op].ndim])
        if int(np.prod(shape)) <= MAX_NODES and shape not in out:
            out.append(shape)
    return out


CASES = [(op, shape) for op in sorted(W.OPS) for shape in _shapes(op)]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


def _check_grads(got, ref, what):
    for f, (a, r) in enumerate(zip(got, ref)):
        assert np.all(np.isfinite(a)), f"{what}: grad {f} has unwritten nodes"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("op,shape", CASES,
                         ids=[f"op{op}-{'x'.join(map(str, s))}" for op, s in CASES])
def test_random_shape_every_entry_point(oracle_mod, op, shape, bc_mode):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    seed = 31 * op + sum(shape)
    wl = W.normal_fields(op, shape, seed)
    what = f"op{op} {shape} bc{bc_mode}"
    print(f"case random-shape {what}", flush=True)
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    Rr = oracle_mod.residual(*args, bc_mode=bc_mode)
    Lr = oracle_mod.loss(*args, bc_mode=bc_mode)
    gr = oracle_mod.grad(*args, dloss=0.8, bc_mode=bc_mode)

    # forward with residuals, then bwd + bc
    R, L, g = H.run_gpu(wl, dloss=0.8, bc_mode=bc_mode)
    if bc_mode == 0:
        H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=what)
    else:
        for b, (a, r) in enumerate(zip(R, Rr)):
            assert H.max_rel_err(a, r) <= H.TOL_RES, (what, b)
        assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (what, L, Lr)
        _check_grads(g, gr, what)

    fields = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in wl.fields]
    consts = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in wl.consts]
    # one-pass value and gradient
    gv = [torch.full_like(f, float("nan")) for f in fields]
    loss = torch.full((), float("nan"), dtype=torch.float64, device="cuda")
    dl = torch.tensor(0.8, dtype=torch.float64, device="cuda")
    B.fpde_residual_value_and_grad(wl.op, fields, consts, wl.h, wl.coeffs, dl, loss=loss,
                                   grads=gv, bc_mode=bc_mode)
    # explicit-sensitivity backward
    G = W.sensitivities(op, shape, seed + 1)
    gj = [torch.full_like(f, float("nan")) for f in fields]
    B.fpde_residual_vjp(wl.op, fields, wl.h, wl.coeffs,
                        [torch.from_numpy(x).cuda() for x in G], grads=gj, bc_mode=bc_mode)
    torch.cuda.synchronize()
    assert abs(loss.item() - Lr) <= H.TOL_RES * abs(Lr), (what, loss.item(), Lr)
    _check_grads([x.cpu().numpy() for x in gv], gr, "value_and_grad " + what)
    _check_grads([x.cpu().numpy() for x in gj],
                 oracle_mod.vjp(*args, G, bc_mode=bc_mode), "vjp " + what)
