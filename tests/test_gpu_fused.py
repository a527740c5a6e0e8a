"""GPU parity of the one-pass value and gradient (fpde_residual_value_and_grad):
the loss of the forward and the gradient of backward + boundary correction from
one read of the inputs, compared with the oracle node by node in both boundary
modes, and with the three-call path on the same inputs."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

CASES = [
    ("burgers_1dt", (3, 3)), ("burgers_1dt", (5, 7)), ("burgers_1dt", (41, 300)),
    ("helmholtz_2d", (4, 259)), ("helmholtz_2d", (67, 513)),
    ("heat_3d", (3, 3, 3)), ("heat_3d", (5, 6, 7)), ("heat_3d", (19, 21, 70)),
    ("heat_3d", (9, 10, 300)),
    ("ns_2d", (6, 257)), ("ns_2d", (71, 600)),
    # rows wider than one 512-node segment of the one-pass kernel, ragged tail
    ("ns_2d", (5, 1300)), ("helmholtz_2d", (7, 1030)),
    ("ns_3d_tgv", (3, 3, 3)), ("ns_3d_tgv", (4, 9, 66)), ("ns_3d_tgv", (19, 21, 70)),
    ("ns_3d_tgv", (40, 17, 129)), ("ns_3d_tgv", (7, 9, 300)), ("ns_3d_tgv", (42, 256, 256)),
]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


def _dev(arrs):
    import torch  # noqa: PLC0415
    return [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in arrs]


def gpu_value_and_grad(wl, dloss, bc_mode=0):
    """Outputs pre-filled with NaN (an unwritten node stays NaN; the loss must be
    overwritten, not accumulated)."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    fields, consts = _dev(wl.fields), _dev(wl.consts)
    grads = [torch.full_like(f, float("nan")) for f in fields]
    loss = torch.full((), float("nan"), dtype=torch.float64, device="cuda")
    dl = torch.tensor(float(dloss), dtype=torch.float64, device="cuda")
    B.fpde_residual_value_and_grad(wl.op, fields, consts, wl.h, wl.coeffs, dl, loss=loss,
                                   grads=grads, bc_mode=bc_mode)
    torch.cuda.synchronize()
    return float(loss.item()), [g.cpu().numpy() for g in grads]


def _check(oracle_mod, wl, dloss, bc_mode, what):
    L, g = gpu_value_and_grad(wl, dloss, bc_mode)
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    Lr = oracle_mod.loss(*args, bc_mode=bc_mode)
    gr = oracle_mod.grad(*args, dloss=dloss, bc_mode=bc_mode)
    assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (what, L, Lr)
    for f, (a, r) in enumerate(zip(g, gr)):
        assert np.all(np.isfinite(a)), f"{what}: grad {f} has unwritten nodes"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape", CASES, ids=[f"{c}-{'x'.join(map(str, s))}" for c, s in CASES])
def test_value_and_grad_parity(oracle_mod, cfg, shape, bc_mode):
    wl = W.make(cfg, seed=61, shape=shape)
    print(f"case value_and_grad {cfg} {shape} bc_mode={bc_mode}", flush=True)
    _check(oracle_mod, wl, 0.7, bc_mode, f"vg {cfg}{shape} bc{bc_mode}")


@pytest.mark.parametrize("op", sorted(W.OPS))
def test_value_and_grad_normal_inputs(oracle_mod, op):
    shape = H.normal_shape(op)
    wl = W.normal_fields(op, shape, 45)
    print(f"case value_and_grad normal op={op} {shape}", flush=True)
    _check(oracle_mod, wl, 1.0, 0, f"vg normal op{op}")


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg", ["burgers_1dt", "helmholtz_2d", "heat_3d", "ns_2d", "ns_3d_tgv"])
def test_value_and_grad_matches_three_call_path_full_size(cfg, bc_mode):
    """At the full benchmark sizes: the same gradient as bwd + bc, bit for bit
    on the planes the three-call backward marches (the same march, which adds
    the loss on the side) and within float32 rounding on the end planes of axis
    0 (there the one-pass march evaluates the general transposed stencil with
    zero residuals where the boundary kernel evaluates the boundary term alone);
    the loss of the forward up to the float64 summation order."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make(cfg, seed=42)
    print(f"case value_and_grad full {cfg} {wl.shape} bc_mode={bc_mode}", flush=True)
    fields, consts = _dev(wl.fields), _dev(wl.consts)
    dl = torch.tensor(1.0, dtype=torch.float64, device="cuda")
    L3 = B.fpde_residual_fwd(wl.op, fields, consts, wl.h, wl.coeffs, bc_mode=bc_mode)
    g3 = B.fpde_residual_bwd(wl.op, fields, consts, wl.h, wl.coeffs, dl, bc_mode=bc_mode)
    B.fpde_bc_correct(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=g3, bc_mode=bc_mode)
    L1, g1 = B.fpde_residual_value_and_grad(wl.op, fields, consts, wl.h, wl.coeffs, dl,
                                            bc_mode=bc_mode)
    torch.cuda.synchronize()
    assert abs(L1.item() - L3.item()) <= 1e-9 * abs(L3.item()), (L1.item(), L3.item())
    for a, b in zip(g1, g3):
        if bc_mode == 1:  # no boundary: every plane is marched by both
            assert torch.equal(a, b)
            continue
        assert torch.equal(a[1:-1], b[1:-1])
        ends = torch.stack([b[0], b[-1]]).double()
        err = (torch.stack([a[0], a[-1]]).double() - ends).abs().max().item()
        assert err <= 1e-6 * max(ends.abs().max().item(), 1e-30), err


def test_value_and_grad_full_size_ns3d_loss(oracle_mod):
    """3D TGV at 256^3: the loss against the oracle on the whole grid (the
    gradient is the bwd + bc gradient, checked against the oracle elsewhere)."""
    wl = W.make("ns_3d_tgv", seed=42)
    L, g = gpu_value_and_grad(wl, 1.0)
    Lr = oracle_mod.loss(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    assert abs(L - Lr) <= H.TOL_RES * abs(Lr), (L, Lr)
    for x in g:
        assert np.all(np.isfinite(x))


def test_value_and_grad_dloss_scaling():
    """grads scale with dloss; the loss does not (up to the order in which the
    workgroups' float64 atomic adds land)."""
    wl = W.make("ns_3d_tgv", seed=62, shape=(19, 21, 70))
    L1, g1 = gpu_value_and_grad(wl, 1.0)
    L2, g2 = gpu_value_and_grad(wl, -2.5)
    assert abs(L1 - L2) <= 1e-13 * abs(L1), (L1, L2)
    for a, b in zip(g1, g2):
        assert H.max_rel_err(b, -2.5 * a.astype(np.float64)) <= 1e-6
