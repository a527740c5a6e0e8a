"""Independent float64 PyTorch finite-difference reference (test helper).

The residuals are built the way the paper's eager PyTorch baseline builds them
(App. A.2): tensor slices of the interior shifted by one node, combined with
element-wise arithmetic; the gradient comes from ``torch.autograd``.  It shares
nothing with the C oracle: no stencil code, no Jacobian, no loop order.
"""
from __future__ import annotations

import torch


def _sh(q, a, s):
    idx = [slice(1, n - 1) for n in q.shape]
    idx[a] = slice(1 + s, q.shape[a] - 1 + s)
    return q[tuple(idx)]


def _d1(q, a, h):
    return (_sh(q, a, 1) - _sh(q, a, -1)) / (2 * h[a])


def _d2(q, a, h):
    return (_sh(q, a, 1) - 2 * _sh(q, a, 0) + _sh(q, a, -1)) / h[a] ** 2


def residuals(op, h, co, F, C):
    """Residual tensors on the interior (shape n-2 per axis)."""
    d = F[0].dim()
    c0 = lambda q: _sh(q, 0, 0)  # interior view
    if op == 1:  # Burgers, axis 0 = t, axis 1 = x
        u = F[0]
        return [_d1(u, 0, h) + c0(u) * _d1(u, 1, h) - co.nu * _d2(u, 1, h)]
    if op == 2:  # Helmholtz
        u, f = F[0], C[0]
        return [sum(_d2(u, a, h) for a in range(d)) + co.k ** 2 * c0(u) - c0(f)]
    if op == 3:  # implicit heat step
        u, u0 = F[0], C[0]
        return [(c0(u) - c0(u0)) / co.dt - co.alpha * sum(_d2(u, a, h) for a in range(d))]
    if op in (7, 8):  # Poisson
        u, f = F[0], C[0]
        return [sum(_d2(u, a, h) for a in range(d)) - c0(f)]
    if op in (9, 10):  # NS on a space-time grid: axis 0 = t, velocity component b on axis b + 1
        ds = d - 1  # spatial components
        vel, p = F[:ds], F[ds]
        out = []
        for b in range(ds):
            r = _d1(vel[b], 0, h) + sum(c0(vel[a]) * _d1(vel[b], a + 1, h) for a in range(ds)) \
                + _d1(p, b + 1, h) - co.nu * sum(_d2(vel[b], a + 1, h) for a in range(ds))
            out.append(r)
        out.append(sum(_d1(vel[a], a + 1, h) for a in range(ds)))
        return out
    if op in (4, 5, 6):  # incompressible NS, velocity component b on axis b
        vel, p = F[:d], F[d]
        out = []
        for b in range(d):
            r = sum(c0(vel[a]) * _d1(vel[b], a, h) for a in range(d)) + _d1(p, b, h) \
                - co.nu * sum(_d2(vel[b], a, h) for a in range(d))
            if op == 5:
                r = r + (c0(vel[b]) - c0(C[b])) / co.dt
            out.append(r)
        out.append(sum(_d1(vel[a], a, h) for a in range(d)))
        return out
    raise ValueError(op)


def loss_and_grad(op, h, co, fields, consts):
    F = [torch.tensor(f, dtype=torch.float64, requires_grad=True) for f in fields]
    C = [torch.tensor(c, dtype=torch.float64) for c in consts]
    R = residuals(op, h, co, F, C)
    L = sum((r ** 2).mean() for r in R)
    g = torch.autograd.grad(L, F)
    return [r.detach().numpy() for r in R], float(L.detach()), [x.numpy() for x in g]
