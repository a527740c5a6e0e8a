"""GPU parity when input arrays alias each other.

The ABI forbids only outputs that overlap inputs; inputs may share memory (a
const that is one of the fields, two fields that are one array).  The kernels
read every input through its own buffer descriptor, so a shared array must
give exactly what separate copies of it give: each case passes the same
device tensor in several input slots and compares every entry point, node by
node, with the oracle on separate float32 copies of the same values.
Inputs: the paper's N(0,1) verification fields (App. A.7)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

# (op, shape, which input slots share an array): ("c", j) is const j and
# ("f", i) field i; every slot of a group reads the array of its first slot
CASES = [
    # backward-Euler NS with u_prev, v_prev, w_prev = u, v, w: no time term
    (W.NS_3D_BE, (13, 19, 75), [[("f", 0), ("c", 0)], [("f", 1), ("c", 1)], [("f", 2), ("c", 2)]]),
    # heat with u0 = u: R = -alpha lap u
    (W.HEAT_3D_BE, (11, 18, 140), [[("f", 0), ("c", 0)]]),
    # Helmholtz with f = u
    (W.HELMHOLTZ_2D, (37, 291), [[("f", 0), ("c", 0)]]),
    # steady 2-D NS with v = u (two differentiated fields on one array)
    (W.NS_2D_STEADY, (37, 291), [[("f", 0), ("f", 1)]]),
    # 3D+t NS with u = v = w
    (W.NS_3DT, (6, 9, 11, 75), [[("f", 0), ("f", 1), ("f", 2)]]),
]


def _shared(op, shape, groups, seed):
    """The workload with every group's slots holding the first slot's values (as
    separate numpy copies, for the oracle), and the slot map for the GPU."""
    wl = W.normal_fields(op, shape, seed)
    arrays = {("f", i): a for i, a in enumerate(wl.fields)}
    arrays.update({("c", j): a for j, a in enumerate(wl.consts)})
    source = {slot: slot for slot in arrays}
    for g in groups:
        for slot in g[1:]:
            arrays[slot] = arrays[g[0]].copy()
            source[slot] = g[0]
    wl.fields = [arrays[("f", i)] for i in range(len(wl.fields))]
    wl.consts = [arrays[("c", j)] for j in range(len(wl.consts))]
    return wl, source


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("op,shape,groups", CASES,
                         ids=[f"op{op}-{'x'.join(map(str, s))}" for op, s, _ in CASES])
def test_inputs_sharing_an_array(oracle_mod, op, shape, groups, bc_mode):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    what = f"aliasing op{op} {shape} bc{bc_mode}"
    print(f"case {what}", flush=True)
    wl, source = _shared(op, shape, groups, seed=50 + op)
    dev = torch.device("cuda:0")
    # one device tensor per distinct array; a slot that shares passes its source's
    distinct = {}
    for slot, src in source.items():
        if src not in distinct:
            kind, i = src
            distinct[src] = torch.from_numpy((wl.fields if kind == "f" else wl.consts)[i]).to(dev)
    fields = [distinct[source[("f", i)]] for i in range(len(wl.fields))]
    consts = [distinct[source[("c", j)]] for j in range(len(wl.consts))]
    assert len(distinct) < len(source)  # the case really shares memory

    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    Rr = oracle_mod.residual(*args, bc_mode=bc_mode)
    Lr = oracle_mod.loss(*args, bc_mode=bc_mode)
    gr = oracle_mod.grad(*args, dloss=0.7, bc_mode=bc_mode)

    R = [torch.full_like(fields[0], float("nan")) for _ in wl.spec.residuals]
    loss = B.fpde_residual_fwd(wl.op, fields, consts, wl.h, wl.coeffs, residual_out=R,
                               bc_mode=bc_mode)
    dl = torch.tensor(0.7, dtype=torch.float64, device=dev)
    grads = [torch.full_like(f, float("nan")) for f in fields]
    B.fpde_residual_bwd(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=grads, bc_mode=bc_mode)
    B.fpde_bc_correct(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=grads, bc_mode=bc_mode)
    gv = [torch.full_like(f, float("nan")) for f in fields]
    lv = torch.full((), float("nan"), dtype=torch.float64, device=dev)
    B.fpde_residual_value_and_grad(wl.op, fields, consts, wl.h, wl.coeffs, dl, loss=lv,
                                   grads=gv, bc_mode=bc_mode)
    torch.cuda.synchronize()

    Rn = [r.cpu().numpy() for r in R]
    for b, (a, r) in enumerate(zip(Rn, Rr)):
        assert H.max_rel_err(a, r) <= H.TOL_RES, (what, "residual", b)
    for L in (loss.item(), lv.item()):
        assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (what, L, Lr)
    for name, gs in (("bwd + bc", grads), ("value_and_grad", gv)):
        for f, (a, r) in enumerate(zip(gs, gr)):
            a = a.cpu().numpy()
            assert np.all(np.isfinite(a)), (what, name, f)
            assert H.max_rel_err(a, r) <= H.TOL_GRAD, (what, name, f)
