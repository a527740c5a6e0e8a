"""CPU oracle for the FD residual operator (ctypes binding).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The GPU product path never imports
this package.

All functions take and return float64 numpy arrays on the host.  Inputs given
in float32 are widened exactly.  ``coeffs`` is any object with attributes
``nu, k, dt, alpha``.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libfpde_oracle.so")
_lib = None

_DP = ctypes.POINTER(ctypes.c_double)


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b  # noqa: PLC0415
            _b.build()
        lib = ctypes.CDLL(_LIB_PATH)
        pp = ctypes.POINTER(_DP)
        common = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_long), _DP, ctypes.c_int,
                  _DP, pp, pp]
        lib.orc_op_info.argtypes = [ctypes.c_int] + [ctypes.POINTER(ctypes.c_int)] * 4
        lib.orc_residual.argtypes = common + [pp]
        lib.orc_loss.argtypes = common + [_DP]
        lib.orc_vjp.argtypes = common + [pp, pp]
        lib.orc_grad.argtypes = common + [ctypes.c_double, pp]
        for f in (lib.orc_op_info, lib.orc_residual, lib.orc_loss, lib.orc_vjp, lib.orc_grad):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def op_info(op: int):
    lib = _load()
    v = [ctypes.c_int() for _ in range(4)]
    st = lib.orc_op_info(op, *[ctypes.byref(x) for x in v])
    if st:
        raise ValueError(f"unknown op {op}")
    return tuple(x.value for x in v)  # ndim, n_fields, n_consts, n_residuals


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptrs(arrs: Sequence[np.ndarray]):
    t = (_DP * max(1, len(arrs)))()
    for i, a in enumerate(arrs):
        t[i] = a.ctypes.data_as(_DP)
    return t


class _Args:
    def __init__(self, op, shape, h, coeffs, fields, consts, bc_mode):
        self.op = int(op)
        self.ndim, self.nf, self.nc, self.nr = op_info(op)
        self.shape = tuple(int(s) for s in shape)
        self.fields = [_f64(f) for f in fields]
        self.consts = [_f64(c) for c in consts]
        for a in self.fields + self.consts:
            if a.shape != self.shape:
                raise ValueError(f"array shape {a.shape} != grid {self.shape}")
        if len(self.fields) != self.nf or len(self.consts) != self.nc:
            raise ValueError("wrong number of fields/consts")
        self.n = (ctypes.c_long * len(self.shape))(*self.shape)
        self.h = (ctypes.c_double * len(self.shape))(*[float(x) for x in h])
        self.coef = (ctypes.c_double * 4)(float(coeffs.nu), float(coeffs.k), float(coeffs.dt),
                                          float(coeffs.alpha))
        self.bc_mode = int(bc_mode)
        self.fp = _ptrs(self.fields)
        self.cp = _ptrs(self.consts)

    def head(self):
        return (self.op, len(self.shape), self.n, self.h, self.bc_mode, self.coef, self.fp, self.cp)


def _check(st: int, what: str):
    if st != 0:
        raise ValueError(f"oracle {what} failed with status {st}")


def residual(op, shape, h, coeffs, fields, consts=(), bc_mode=0) -> List[np.ndarray]:
    """Residual arrays R_b (full size; zero off the residual node set)."""
    a = _Args(op, shape, h, coeffs, fields, consts, bc_mode)
    R = [np.zeros(a.shape) for _ in range(a.nr)]
    _check(_load().orc_residual(*a.head(), _ptrs(R)), "residual")
    return R


def loss(op, shape, h, coeffs, fields, consts=(), bc_mode=0) -> float:
    """Sum over equations of the mean squared residual."""
    a = _Args(op, shape, h, coeffs, fields, consts, bc_mode)
    out = ctypes.c_double()
    _check(_load().orc_loss(*a.head(), ctypes.byref(out)), "loss")
    return out.value


def vjp(op, shape, h, coeffs, fields, consts, G, bc_mode=0) -> List[np.ndarray]:
    """Transpose-Jacobian action: grads[q] = sum_b J_bq^T G_b."""
    a = _Args(op, shape, h, coeffs, fields, consts, bc_mode)
    Gs = [_f64(g) for g in G]
    if len(Gs) != a.nr or any(g.shape != a.shape for g in Gs):
        raise ValueError("G must hold one full-size array per residual")
    out = [np.zeros(a.shape) for _ in range(a.nf)]
    _check(_load().orc_vjp(*a.head(), _ptrs(Gs), _ptrs(out)), "vjp")
    return out


def grad(op, shape, h, coeffs, fields, consts=(), dloss=1.0, bc_mode=0) -> List[np.ndarray]:
    """Gradient of dloss * loss w.r.t. every node of every field."""
    a = _Args(op, shape, h, coeffs, fields, consts, bc_mode)
    out = [np.zeros(a.shape) for _ in range(a.nf)]
    _check(_load().orc_grad(*a.head(), float(dloss), _ptrs(out)), "grad")
    return out


def on_workload(wl, dloss=1.0, bc_mode=0):
    """(residuals, loss, grads) of a ``workloads.Workload``."""
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    R = residual(*args, bc_mode=bc_mode)
    L = loss(*args, bc_mode=bc_mode)
    g = grad(*args, dloss=dloss, bc_mode=bc_mode)
    return R, L, g
