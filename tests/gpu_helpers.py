"""Helpers shared by the GPU parity tests: run the HIP path, compare with the oracle."""
from __future__ import annotations

import numpy as np

# parity bar: residuals and loss within 1e-5 * max|ref|, gradients within 1e-4 * max|ref|
TOL_RES = 1e-5
TOL_GRAD = 1e-4


def normal_shape(op):
    """A ragged grid for the paper's N(0,1) verification inputs, by operator rank:
    several tiles and chunks with ragged tails (four axes: several time levels)."""
    from paper_2607_18020_amd import workloads as W  # noqa: PLC0415
    return {2: (37, 291), 3: (13, 19, 75), 4: (6, 9, 11, 75)}[W.OPS[op].ndim]


def interior(a):
    return a[tuple(slice(1, n - 1) for n in a.shape)]


def shell_mask(shape):
    m = np.ones(shape, bool)
    m[tuple(slice(1, n - 1) for n in shape)] = False
    return m


def run_gpu(wl, dloss=1.0, store_residual=True, order=("bwd", "bc"), bc_mode=0):
    """fwd (+ residuals) then bwd and bc on cuda:0; outputs pre-filled with NaN so
    that untouched nodes are visible.  Returns numpy (R list, loss, grads list)."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    dev = torch.device("cuda:0")
    fields = [torch.from_numpy(f).to(dev) for f in wl.fields]
    consts = [torch.from_numpy(c).to(dev) for c in wl.consts]
    R = None
    if store_residual:
        R = [torch.full_like(fields[0], float("nan")) for _ in wl.spec.residuals]
    loss = B.fpde_residual_fwd(wl.op, fields, consts, wl.h, wl.coeffs, residual_out=R,
                               bc_mode=bc_mode)
    dl = torch.tensor(float(dloss), dtype=torch.float64, device=dev)
    grads = [torch.full_like(f, float("nan")) for f in fields]
    for step in order:
        fn = B.fpde_residual_bwd if step == "bwd" else B.fpde_bc_correct
        fn(wl.op, fields, consts, wl.h, wl.coeffs, dl, grads=grads, bc_mode=bc_mode)
    torch.cuda.synchronize()
    Rn = [r.cpu().numpy() for r in R] if R is not None else None
    return Rn, float(loss.item()), [g.cpu().numpy() for g in grads]


def max_rel_err(got, ref):
    scale = float(np.abs(ref).max())
    err = float(np.abs(got.astype(np.float64) - ref).max())
    return err / scale if scale > 0 else err


def assert_parity(wl, R_gpu, L_gpu, g_gpu, R_ref, L_ref, g_ref, what=""):
    """Element-by-element comparison on the same float32 inputs."""
    sm = shell_mask(wl.shape)
    if R_gpu is not None:
        for b, (rg, rr) in enumerate(zip(R_gpu, R_ref)):
            assert np.all(rg[sm] == 0), f"{what}: residual {b} not zero off the residual set"
            e = max_rel_err(interior(rg), interior(rr))
            assert e <= TOL_RES, f"{what}: residual {b} rel err {e:.3e}"
    eL = abs(L_gpu - L_ref) / abs(L_ref)
    assert eL <= TOL_RES, f"{what}: loss {L_gpu!r} vs {L_ref!r} (rel {eL:.3e})"
    for f, (gg, gr) in enumerate(zip(g_gpu, g_ref)):
        assert np.all(np.isfinite(gg)), f"{what}: grad {f} has unwritten nodes"
        e = max_rel_err(gg, gr)
        assert e <= TOL_GRAD, f"{what}: grad {f} rel err {e:.3e}"
