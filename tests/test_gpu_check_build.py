"""The checking build of the library against the product build.

libfpde_check.so is the same source compiled with every LDS array of the
marching kernels filled with NaN before the march, and with other tile shapes,
chunk lengths, 2-D row widths and 2-D row-queue depth.  On the same inputs:
- no output holds a NaN: no kernel reads an LDS location that no load or
  residual evaluation wrote;
- residuals and gradients are bitwise those of the product build: a node's
  residual and its gather are evaluated the same way whatever tile, chunk or
  row segment holds it, so tile edges, halos and chunk seams leave no trace;
- the losses agree to the float64 summation order of the per-workgroup sums.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W

pytestmark = pytest.mark.gpu

CASES = [
    ("ns_3d_tgv", (19, 21, 70)), ("ns_3d_tgv", (40, 17, 129)), ("ns_3d_tgv", (7, 9, 300)),
    ("ns_3d_tgv", (42, 256, 256)), ("heat_3d", (19, 21, 70)), ("heat_3d", (9, 10, 300)),
    ("ns_2d", (71, 600)), ("ns_2d", (13400, 40)), ("burgers_1dt", (41, 300)),
    ("helmholtz_2d", (67, 513)), ("ns_3d_steady", (19, 21, 70)), ("poisson_3d", (33, 40, 130)),
    ("poisson_2d", (30, 700)), ("ns_2dt", (9, 20, 70)), ("ns_3dt", (6, 19, 21, 70)),
    ("ns_3dt", (5, 12, 17, 300)),
]


def _run_all(wl, bc_mode):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    sens = [torch.from_numpy(x).cuda() for x in W.sensitivities(wl.op, wl.shape, 9)]
    dl = torch.tensor(1.25, dtype=torch.float64, device="cuda")
    R = [torch.full_like(f[0], float("nan")) for _ in wl.spec.residuals]
    L = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, residual_out=R, bc_mode=bc_mode)
    g = [torch.full_like(x, float("nan")) for x in f]
    B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g, bc_mode=bc_mode)
    B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g, bc_mode=bc_mode)
    Lv, gv = B.fpde_residual_value_and_grad(wl.op, f, c, wl.h, wl.coeffs, dl, bc_mode=bc_mode)
    gj = B.fpde_residual_vjp(wl.op, f, wl.h, wl.coeffs, sens, bc_mode=bc_mode)
    torch.cuda.synchronize()
    return (L.item(), Lv.item(), [x.cpu().numpy() for x in R], [x.cpu().numpy() for x in g],
            [x.cpu().numpy() for x in gv], [x.cpu().numpy() for x in gj])


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape", CASES, ids=[f"{c}-{'x'.join(map(str, s))}" for c, s in CASES])
def test_check_build_matches_product(cfg, shape, bc_mode):
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    if not os.path.exists(B.CHECK_LIB_PATH):  # (build() always builds it beside the product)
        pytest.skip(f"{B.CHECK_LIB_PATH} is not built")
    wl = W.make(cfg, seed=49, shape=shape)
    print(f"case check-build {cfg} {shape} bc_mode={bc_mode}", flush=True)
    prod = _run_all(wl, bc_mode)
    with B.library(B.CHECK_LIB_PATH):
        chk = _run_all(wl, bc_mode)
    for a, b in zip(prod[:2], chk[:2]):
        assert abs(a - b) <= 1e-12 * abs(a), (a, b)
    for what, xs, ys in (("residual", prod[2], chk[2]), ("bwd+bc", prod[3], chk[3]),
                         ("value_and_grad", prod[4], chk[4]), ("vjp", prod[5], chk[5])):
        for i, (x, y) in enumerate(zip(xs, ys)):
            assert not np.isnan(y).any(), f"{what} {i}: NaN in the checking build"
            assert np.array_equal(x, y), \
                f"{what} {i}: max diff {np.abs(x.astype(np.float64) - y).max():.3e}"
