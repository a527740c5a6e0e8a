"""GPU parity of the explicit-sensitivity backward (fpde_residual_vjp): the
transposed residual Jacobian applied to upstream sensitivities G (Sec. 2.2),
compared node by node with the oracle's vjp on the same float32 inputs, in
both boundary modes, overwrite and accumulate; plus the autograd op built on it."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

# several tiles along every axis, ragged last tiles, chunk seams along axis 0,
# the smallest grids, wide rows
CASES = [
    ("burgers_1dt", (3, 3)), ("burgers_1dt", (5, 7)), ("burgers_1dt", (41, 300)),
    ("helmholtz_2d", (4, 259)), ("helmholtz_2d", (67, 513)),
    ("heat_3d", (3, 3, 3)), ("heat_3d", (5, 6, 7)), ("heat_3d", (19, 21, 70)),
    ("heat_3d", (9, 10, 300)),
    ("ns_2d", (6, 257)), ("ns_2d", (71, 600)),
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


def gpu_vjp(wl, G, bc_mode=0, init=None):
    """fpde_residual_vjp on cuda:0.  init None: overwrite mode, outputs pre-filled
    with NaN (an unwritten node stays NaN); else accumulate onto init."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    fields, sens = _dev(wl.fields), _dev(G)
    if init is None:
        grads = [torch.full_like(f, float("nan")) for f in fields]
    else:
        grads = _dev(init)
    B.fpde_residual_vjp(wl.op, fields, wl.h, wl.coeffs, sens, grads=grads,
                        accumulate=init is not None, bc_mode=bc_mode)
    torch.cuda.synchronize()
    return [g.cpu().numpy() for g in grads]


def _compare(got, ref, what):
    for f, (a, r) in enumerate(zip(got, ref)):
        assert np.all(np.isfinite(a)), f"{what}: grad {f} has unwritten nodes"
        e = H.max_rel_err(a, r)
        assert e <= H.TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape", CASES, ids=[f"{c}-{'x'.join(map(str, s))}" for c, s in CASES])
def test_vjp_parity(oracle_mod, cfg, shape, bc_mode):
    wl = W.make(cfg, seed=47, shape=shape)
    G = W.sensitivities(wl.op, shape, 48)
    print(f"case vjp {cfg} {shape} bc_mode={bc_mode}", flush=True)
    got = gpu_vjp(wl, G, bc_mode)
    ref = oracle_mod.vjp(wl.op, shape, wl.h, wl.coeffs, wl.fields, wl.consts, G, bc_mode=bc_mode)
    _compare(got, ref, f"vjp {cfg}{shape} bc{bc_mode}")


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("op", sorted(W.OPS))
def test_vjp_normal_inputs(oracle_mod, op, bc_mode):
    """N(0,1) fields and sensitivities (the paper's verification inputs)."""
    shape = H.normal_shape(op)
    wl = W.normal_fields(op, shape, 42)
    G = W.sensitivities(op, shape, 46)
    print(f"case vjp normal op={op} {shape} bc_mode={bc_mode}", flush=True)
    got = gpu_vjp(wl, G, bc_mode)
    ref = oracle_mod.vjp(op, shape, wl.h, wl.coeffs, wl.fields, wl.consts, G, bc_mode=bc_mode)
    _compare(got, ref, f"vjp normal op{op} bc{bc_mode}")


def test_vjp_ignores_sensitivities_off_the_residual_set():
    """Entries of G on the boundary shell are never read: NaN or huge values
    there give bitwise the result of zeros there."""
    for cfg, shape in (("ns_3d_tgv", (9, 12, 70)), ("ns_2d", (9, 260)), ("heat_3d", (5, 67, 3)),
                       ("burgers_1dt", (3, 300)), ("ns_3dt", (5, 6, 12, 70))):
        wl = W.make(cfg, seed=49, shape=shape)
        G = W.sensitivities(wl.op, shape, 50)
        sm = H.shell_mask(shape)
        Gz = [np.where(sm, np.float32(0), g) for g in G]
        Gn = [np.where(sm, np.float32(np.nan), g) for g in G]
        Gh = [np.where(sm, np.float32(3e38), g) for g in G]
        print(f"case vjp shell {cfg} {shape}", flush=True)
        a, b, c = gpu_vjp(wl, Gz), gpu_vjp(wl, Gn), gpu_vjp(wl, Gh)
        for x, y, z in zip(a, b, c):
            assert np.all(np.isfinite(x))
            assert np.array_equal(x, y) and np.array_equal(x, z), cfg


@pytest.mark.parametrize("bc_mode", [0, 1])
def test_vjp_accumulate(oracle_mod, bc_mode):
    """accumulate = 1 adds the action to what grads hold: bitwise the float32
    sum of the old values and the overwrite-mode result, at every node."""
    for cfg, shape in (("ns_3d_tgv", (19, 21, 70)), ("heat_3d", (9, 10, 300)),
                       ("ns_2d", (71, 600)), ("helmholtz_2d", (4, 259))):
        wl = W.make(cfg, seed=51, shape=shape)
        G = W.sensitivities(wl.op, shape, 52)
        rng = np.random.default_rng(53)
        init = [rng.standard_normal(shape).astype(np.float32) for _ in wl.fields]
        print(f"case vjp accumulate {cfg} {shape} bc_mode={bc_mode}", flush=True)
        over = gpu_vjp(wl, G, bc_mode)
        acc = gpu_vjp(wl, G, bc_mode, init=init)
        for a, o, i in zip(acc, over, init):
            assert np.array_equal(a, i + o), cfg
        ref = oracle_mod.vjp(wl.op, shape, wl.h, wl.coeffs, wl.fields, wl.consts, G,
                             bc_mode=bc_mode)
        _compare([a - i for a, i in zip(acc, init)], ref, f"acc {cfg}")


def test_vjp_is_deterministic():
    wl = W.make("ns_3d_tgv", seed=54, shape=(40, 33, 100))
    G = W.sensitivities(wl.op, wl.shape, 55)
    a, b = gpu_vjp(wl, G), gpu_vjp(wl, G)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# --------------------------------------------------------------------------- full size


@pytest.mark.parametrize("cfg", ["burgers_1dt", "helmholtz_2d", "heat_3d", "ns_2d", "ns_3d_tgv"])
def test_vjp_full_size_every_node(oracle_mod, cfg):
    wl = W.make(cfg, seed=42)
    G = W.sensitivities(wl.op, wl.shape, 56)
    print(f"case vjp full {cfg} {wl.shape}", flush=True)
    got = gpu_vjp(wl, G)
    ref = oracle_mod.vjp(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, G)
    _compare(got, ref, f"vjp full {cfg}")


@pytest.mark.parametrize("seed", [42, 43, 44, 45, 46])
def test_vjp_full_size_ns3d_seeds(oracle_mod, seed):
    """3D TGV at 256^3 in the launch configuration the benchmark times, every
    node against the whole-grid oracle, for the paper's seeds."""
    wl = W.make("ns_3d_tgv", seed=seed)
    G = W.sensitivities(wl.op, wl.shape, 57 + seed)
    print(f"case vjp full ns_3d_tgv {wl.shape} seed {seed}", flush=True)
    got = gpu_vjp(wl, G)
    ref = oracle_mod.vjp(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, G)
    _compare(got, ref, f"vjp full ns_3d_tgv seed {seed}")


@pytest.mark.parametrize("bc_mode", [0, 1])
def test_vjp_full_size_ns3d_matches_loss_gradient(bc_mode):
    """3D TGV at 256^3: the action on G = 2 R / M equals the loss gradient of
    bwd + bc, in both boundary modes."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=42)
    print(f"case vjp = loss gradient ns_3d_tgv {wl.shape} bc_mode={bc_mode}", flush=True)
    # property at full size: vjp(2 R / M) == d loss / d q (bwd + bc)
    fields = _dev(wl.fields)
    consts = _dev(wl.consts)
    R = [torch.zeros_like(fields[0]) for _ in wl.spec.residuals]
    B.fpde_residual_fwd(wl.op, fields, consts, wl.h, wl.coeffs, residual_out=R, bc_mode=bc_mode)
    M = wl.n_points if bc_mode == 1 else wl.n_residual_points
    sens = [(2.0 / M) * r for r in R]
    gv = B.fpde_residual_vjp(wl.op, fields, wl.h, wl.coeffs, sens, bc_mode=bc_mode)
    dl = torch.ones((), dtype=torch.float64, device="cuda")
    gl = B.fpde_residual_bwd(wl.op, fields, consts, wl.h, wl.coeffs, dl, bc_mode=bc_mode)
    B.fpde_bc_correct(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=gl, bc_mode=bc_mode)
    torch.cuda.synchronize()
    for a, b in zip(gv, gl):
        e = H.max_rel_err(a.cpu().numpy(), b.cpu().numpy().astype(np.float64))
        assert e <= H.TOL_GRAD, e


# --------------------------------------------------------------------------- autograd


@pytest.mark.parametrize("bc_mode", [0, 1])
def test_residual_autograd_op(oracle_mod, bc_mode):
    """Residual.apply returns R (zero off the residual set); any objective of R
    backpropagates through the vjp: d/dq sum_b <W_b, R_b> = J^T W."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=58, shape=(12, 20, 70))
    fields = [torch.from_numpy(f).cuda().requires_grad_() for f in wl.fields]
    consts = _dev(wl.consts)
    Wt = W.sensitivities(wl.op, wl.shape, 59)
    R = B.Residual.apply(wl.op, wl.h, wl.coeffs, consts, bc_mode, *fields)
    obj = sum((r * w).sum() for r, w in zip(R, _dev(Wt)))
    obj.backward()
    Rr = oracle_mod.residual(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts,
                             bc_mode=bc_mode)
    for a, r in zip(R, Rr):
        assert H.max_rel_err(a.detach().cpu().numpy(), r) <= H.TOL_RES
    ref = oracle_mod.vjp(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, Wt,
                         bc_mode=bc_mode)
    _compare([f.grad.cpu().numpy() for f in fields], ref, f"autograd bc{bc_mode}")


def test_residual_autograd_mse_matches_residual_loss():
    """The MSE objective written in torch over Residual's outputs has the
    gradient of the fused ResidualLoss op (same objective, two backward paths)."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    for bc_mode in (0, 1):
        wl = W.make("ns_2d", seed=60, shape=(71, 600))
        consts = _dev(wl.consts)
        f1 = [torch.from_numpy(f).cuda().requires_grad_() for f in wl.fields]
        f2 = [torch.from_numpy(f).cuda().requires_grad_() for f in wl.fields]
        M = wl.n_points if bc_mode == 1 else wl.n_residual_points
        R = B.Residual.apply(wl.op, wl.h, wl.coeffs, consts, bc_mode, *f1)
        (sum((r.double() ** 2).sum() for r in R) / M).backward()
        B.ResidualLoss.apply(wl.op, wl.h, wl.coeffs, consts, bc_mode, *f2).backward()
        for a, b in zip(f1, f2):
            e = H.max_rel_err(a.grad.cpu().numpy(), b.grad.cpu().numpy().astype(np.float64))
            assert e <= H.TOL_GRAD, (bc_mode, e)
