"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Small, ragged and full-size grids are compared element by element over every
node (residuals on the residual set, the loss, and the gradient on every node,
boundary shell included).  Full-size grids run in the same launch
configuration the benchmark times.
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

# (config, shape): several tiles along every axis plus ragged tails (2-D rows are
# 256-, 512- or 1024-node segments; 3-D tiles are 64, 128 or 256 nodes wide in x; chunks of planes
# along axis 0)
SMALL = [
    ("burgers_1dt", (3, 3)), ("burgers_1dt", (5, 7)), ("burgers_1dt", (41, 300)),
    ("burgers_1dt", (128, 256)),
    ("helmholtz_2d", (3, 3)), ("helmholtz_2d", (4, 259)), ("helmholtz_2d", (67, 513)),
    ("helmholtz_2d", (130, 1000)),
    ("heat_3d", (3, 3, 3)), ("heat_3d", (5, 6, 7)), ("heat_3d", (19, 21, 70)),
    ("heat_3d", (33, 40, 130)),
    ("ns_2d", (3, 3)), ("ns_2d", (6, 257)), ("ns_2d", (71, 600)), ("ns_2d", (300, 257)),
    ("ns_3d_tgv", (3, 3, 3)), ("ns_3d_tgv", (4, 9, 66)), ("ns_3d_tgv", (19, 21, 70)),
    ("ns_3d_tgv", (40, 17, 129)),
    # wider than one 256-node tile: side edges between tiles, ragged last tile
    ("heat_3d", (9, 10, 300)), ("heat_3d", (6, 7, 520)), ("ns_3d_tgv", (7, 9, 300)),
    # full-width planes: several chunks of several planes each along axis 0, so
    # the unrolled march, its tail and the seams between chunks are all exercised
    ("heat_3d", (42, 256, 256)), ("ns_3d_tgv", (42, 256, 256)), ("ns_3d_tgv", (75, 130, 200)),
    ("ns_2d", (700, 513)),
    # 2-D rows wider than one 1024-node forward row segment, ragged last segment
    ("ns_2d", (5, 2500)), ("helmholtz_2d", (9, 1100)), ("burgers_1dt", (6, 3000)),
    # tall 2-D grids: chunks of 14 or more rows, several passes of the forward's
    # unrolled row queue and its tail
    ("ns_2d", (13400, 40)), ("helmholtz_2d", (15000, 20)), ("burgers_1dt", (20000, 30)),
]


@pytest.fixture(scope="module")
def oracle_mod():
    import oracle  # noqa: PLC0415
    return oracle


@pytest.mark.parametrize("cfg,shape", SMALL, ids=[f"{c}-{'x'.join(map(str, s))}" for c, s in SMALL])
def test_parity_small_and_ragged(oracle_mod, cfg, shape):
    wl = W.make(cfg, seed=42, shape=shape)
    print(f"case {cfg} {shape}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=1.0)
    Rr, Lr, gr = oracle_mod.on_workload(wl, dloss=1.0)
    H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"{cfg}{shape}")


@pytest.mark.parametrize("op", sorted(W.OPS))
@pytest.mark.parametrize("seed", [42, 43, 44, 45, 46])
def test_parity_normal_inputs_seeds(oracle_mod, op, seed):
    """The paper's verification inputs (App. A.7): N(0,1) fields, seeds 42-46."""
    shape = H.normal_shape(op)
    wl = W.normal_fields(op, shape, seed)
    print(f"case op={op} seed={seed} {shape}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=1.0)
    Rr, Lr, gr = oracle_mod.on_workload(wl, dloss=1.0)
    H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"op{op} seed{seed}")


# degenerate coefficients: inviscid Burgers and NS (nu = 0), Helmholtz at k = 0
# (the Laplace operator), heat without diffusion (alpha = 0: pointwise), a huge
# time step (the time term all but vanishes), unequal spacings
DEGENERATE = [
    (W.BURGERS_1DT, (33, 130), W.Coeffs(nu=0.0), None),
    (W.HELMHOLTZ_2D, (33, 130), W.Coeffs(k=0.0), None),
    (W.HEAT_3D_BE, (9, 20, 70), W.Coeffs(dt=1e-3, alpha=0.0), None),
    (W.HEAT_3D_BE, (9, 20, 70), W.Coeffs(dt=1e6, alpha=0.1), (0.05, 0.02, 0.01)),
    (W.NS_2D_STEADY, (33, 130), W.Coeffs(nu=0.0), (0.03, 0.01)),
    (W.NS_3D_BE, (9, 20, 70), W.Coeffs(nu=0.0, dt=1e-2), (0.1, 0.05, 0.02)),
    (W.NS_3D_BE, (9, 20, 70), W.Coeffs(nu=0.01, dt=1e6), None),
]


@pytest.mark.parametrize("case", range(len(DEGENERATE)))
def test_parity_degenerate_coefficients(oracle_mod, case):
    op, shape, co, h = DEGENERATE[case]
    wl = W.normal_fields(op, shape, 50 + case, h=h, coeffs=co)
    print(f"case degenerate op={op} {shape} {co} h={h}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=1.0)
    Rr, Lr, gr = oracle_mod.on_workload(wl, dloss=1.0)
    H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"degenerate op{op} {co}")


@pytest.mark.parametrize("cfg", ["ns_2d", "ns_3d_tgv", "burgers_1dt"])
def test_dloss_scaling_and_call_order(oracle_mod, cfg):
    """dloss scales the gradient; bwd and bc write disjoint nodes (either order)."""
    shape = (23, 300) if W.OPS[W.CONFIGS[cfg].op].ndim == 2 else (11, 18, 67)
    wl = W.make(cfg, seed=44, shape=shape)
    dloss = -0.37
    _, L, g = H.run_gpu(wl, dloss=dloss, store_residual=False, order=("bc", "bwd"))
    gr = oracle_mod.grad(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, dloss=dloss)
    for a, b in zip(g, gr):
        assert H.max_rel_err(a, b) <= H.TOL_GRAD


def test_bwd_and_bc_cover_disjoint_node_sets():
    """bwd writes every node of planes 1..n0-2 of axis 0; bc writes planes 0 and n0-1."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    for cfg, shape in (("ns_3d_tgv", (9, 12, 70)), ("ns_2d", (9, 260)), ("heat_3d", (3, 3, 3))):
        wl = W.make(cfg, seed=45, shape=shape)
        fields = [torch.from_numpy(f).cuda() for f in wl.fields]
        consts = [torch.from_numpy(c).cuda() for c in wl.consts]
        dl = torch.ones((), dtype=torch.float64, device="cuda")
        ends = torch.zeros(shape, dtype=torch.bool, device="cuda")
        ends[0] = True
        ends[-1] = True
        g = [torch.full_like(f, float("nan")) for f in fields]
        B.fpde_residual_bwd(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=g)
        torch.cuda.synchronize()
        for x in g:
            assert torch.isnan(x[ends]).all() and torch.isfinite(x[~ends]).all()
        g = [torch.full_like(f, float("nan")) for f in fields]
        B.fpde_bc_correct(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=g)
        torch.cuda.synchronize()
        for x in g:
            assert torch.isfinite(x[ends]).all() and torch.isnan(x[~ends]).all()


def test_gradients_are_deterministic():
    """Gather form, no atomics: two runs give bitwise-identical gradients."""
    wl = W.make("ns_3d_tgv", seed=46, shape=(40, 33, 100))
    _, L1, g1 = H.run_gpu(wl, store_residual=False)
    _, L2, g2 = H.run_gpu(wl, store_residual=False)
    for a, b in zip(g1, g2):
        assert np.array_equal(a, b)
    assert abs(L1 - L2) <= 1e-12 * abs(L1)


def test_full_size_runs_are_deterministic():
    """3D TGV at 256^3, ten fwd + bwd + bc sequences on the same inputs: the
    gradients are bitwise identical every time (gather form, no atomics); the
    loss, summed with one float64 atomic per workgroup in whatever order the
    workgroups finish, spreads by at most 1e-9 relative."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=42)
    print(f"case determinism ns_3d_tgv {wl.shape}", flush=True)
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    dl = torch.ones((), dtype=torch.float64, device="cuda")
    first, losses = None, []
    for _ in range(10):
        g = [torch.full_like(x, float("nan")) for x in f]
        L = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs)
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g)
        B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g)
        losses.append(L.item())
        if first is None:
            first = g
        else:
            assert all(torch.equal(a, b) for a, b in zip(first, g))
    spread = (max(losses) - min(losses)) / abs(sum(losses) / len(losses))
    assert spread <= 1e-9, (spread, losses)


def test_autograd_function_matches_abi(oracle_mod):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=43, shape=(12, 20, 70))
    fields = [torch.from_numpy(f).cuda().requires_grad_() for f in wl.fields]
    consts = [torch.from_numpy(c).cuda() for c in wl.consts]
    loss = B.ResidualLoss.apply(wl.op, wl.h, wl.coeffs, consts, *fields)
    (2.5 * loss).backward()
    gr = oracle_mod.grad(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts, dloss=2.5)
    for f, ref in zip(fields, gr):
        assert H.max_rel_err(f.grad.cpu().numpy(), ref) <= H.TOL_GRAD
    Lr = oracle_mod.loss(wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    assert abs(loss.item() - Lr) <= H.TOL_RES * Lr


# --------------------------------------------------------------------------- full size


# the paper's seeds (App. A.7); each draws a new synthetic workload
SEEDS = [42, 43, 44, 45, 46]


@pytest.mark.parametrize("seed", SEEDS)
@pytest.mark.parametrize("cfg", ["burgers_1dt", "helmholtz_2d", "heat_3d", "ns_2d", "ns_3d_tgv"])
def test_parity_full_size_every_node(oracle_mod, cfg, seed):
    """Every workload at full size, in the launch configuration the benchmark
    times (the 256^3 Taylor-Green grid included: 16.8M nodes x 4 residuals and
    4 gradients), compared with the whole-grid oracle node by node."""
    wl = W.make(cfg, seed=seed)
    print(f"case full {cfg} {wl.shape} seed {seed}", flush=True)
    R, L, g = H.run_gpu(wl, dloss=1.0)
    Rr, Lr, gr = oracle_mod.on_workload(wl, dloss=1.0)
    H.assert_parity(wl, R, L, g, Rr, Lr, gr, what=f"full {cfg}")
