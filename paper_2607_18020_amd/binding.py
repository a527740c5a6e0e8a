"""ctypes binding of libfpde (include/fpde.h): argument marshalling only.

Every computation runs in the library's HIP kernels; this module turns torch
tensors into device pointers, grid/coefficient structs and a stream handle,
calls the C entry point and raises on a non-zero status.  There is no CPU
fallback: importing fails loudly when libfpde.so has not been built.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfpde.so")
# the checking build of the same sources (LDS poisoned with NaN, other tilings);
# tests only
CHECK_LIB_PATH = os.path.join(_HERE, "libfpde_check.so")

FPDE_OK = 0
STATUS_NAMES = {0: "FPDE_OK", -1: "FPDE_ERR_ARG", -2: "FPDE_ERR_SHAPE", -3: "FPDE_ERR_SPACING",
                -4: "FPDE_ERR_COEFF", -5: "FPDE_ERR_ALIGN", -6: "FPDE_ERR_HIP",
                -7: "FPDE_ERR_UNSUPPORTED"}
# the compute entry points; each also exists with a 4 suffix taking fpde_grid4
CALLS = ("fpde_residual_fwd", "fpde_residual_bwd", "fpde_bc_correct", "fpde_residual_vjp",
         "fpde_residual_value_and_grad")
EXPORTED = ("fpde_op_info",) + CALLS + tuple(c + "4" for c in CALLS) + \
    ("fpde_status_string", "fpde_version")


class FpdeGrid(ctypes.Structure):
    _fields_ = [("ndim", ctypes.c_int32), ("bc_mode", ctypes.c_int32),
                ("n", ctypes.c_int64 * 3), ("h", ctypes.c_double * 3)]


class FpdeGrid4(ctypes.Structure):
    """fpde_grid4: the grid with up to four axes (space-time 3D+t grids)."""
    _fields_ = [("ndim", ctypes.c_int32), ("bc_mode", ctypes.c_int32),
                ("n", ctypes.c_int64 * 4), ("h", ctypes.c_double * 4)]


class FpdeCoeffs(ctypes.Structure):
    _fields_ = [("nu", ctypes.c_double), ("k", ctypes.c_double), ("dt", ctypes.c_double),
                ("alpha", ctypes.c_double)]


class FpdeError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {_load().fpde_status_string(status).decode()} ({status})")


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_18020_amd.csrc.build`")
        lib = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        pp = ctypes.POINTER(ctypes.c_void_p)
        cp = ctypes.POINTER(FpdeCoeffs)
        lib.fpde_op_info.argtypes = [ctypes.c_int] + [ctypes.POINTER(ctypes.c_int)] * 4
        lib.fpde_op_info.restype = ctypes.c_int
        for sfx, grid in (("", FpdeGrid), ("4", FpdeGrid4)):
            gp = ctypes.POINTER(grid)
            sig = {"fpde_residual_fwd": [ctypes.c_int, gp, cp, pp, pp, pp, vp, vp],
                   "fpde_residual_bwd": [ctypes.c_int, gp, cp, pp, pp, vp, pp, vp],
                   "fpde_bc_correct": [ctypes.c_int, gp, cp, pp, pp, vp, pp, vp],
                   "fpde_residual_vjp": [ctypes.c_int, gp, cp, pp, pp, ctypes.c_int, pp, vp],
                   "fpde_residual_value_and_grad": [ctypes.c_int, gp, cp, pp, pp, vp, vp, pp, vp]}
            for name, args in sig.items():
                fn = getattr(lib, name + sfx)
                fn.argtypes = args
                fn.restype = ctypes.c_int
        lib.fpde_status_string.argtypes = [ctypes.c_int]
        lib.fpde_status_string.restype = ctypes.c_char_p
        lib.fpde_version.argtypes = []
        lib.fpde_version.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def lib():
    """The loaded ctypes library (raises ImportError if it is not built)."""
    return _load()


@contextlib.contextmanager
def library(path: str):
    """Within the block, the calls of this module go to another build of the C
    ABI at ``path`` (the tests compare the checking build with the product)."""
    global _lib, LIB_PATH
    saved = (_lib, LIB_PATH)
    _lib, LIB_PATH = None, path
    try:
        _load()
        yield
    finally:
        _lib, LIB_PATH = saved


def op_info(op: int):
    v = [ctypes.c_int() for _ in range(4)]
    st = _load().fpde_op_info(int(op), *[ctypes.byref(x) for x in v])
    if st != FPDE_OK:
        raise FpdeError(st, "fpde_op_info")
    return tuple(x.value for x in v)  # ndim, n_fields, n_consts, n_residuals


def make_grid(shape: Sequence[int], h: Sequence[float], bc_mode: int = 0):
    """fpde_grid for up to three axes, fpde_grid4 for four."""
    g = FpdeGrid4() if len(shape) == 4 else FpdeGrid()
    g.ndim = len(shape)
    g.bc_mode = int(bc_mode)
    for a, (n, hh) in enumerate(zip(shape, h)):
        g.n[a] = int(n)
        g.h[a] = float(hh)
    return g


def _entry(name: str, shape):
    """The C entry point for a grid of this rank (the 4-suffixed one for four axes)."""
    return getattr(_load(), name + ("4" if len(shape) == 4 else ""))


def make_coeffs(c) -> FpdeCoeffs:
    return FpdeCoeffs(float(getattr(c, "nu", 0.0)), float(getattr(c, "k", 0.0)),
                      float(getattr(c, "dt", 1.0)), float(getattr(c, "alpha", 0.0)))


def _ptr_array(tensors):
    arr = (ctypes.c_void_p * max(1, len(tensors)))()
    for i, t in enumerate(tensors):
        arr[i] = t.data_ptr()
    return arr


def _check_tensors(tensors, shape, what):
    dev = None
    for t in tensors:
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 \
                or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
            raise ValueError(f"{what}: need contiguous float32 CUDA tensors of shape {tuple(shape)}")
        dev = t.device if dev is None else dev
        if t.device != dev:
            raise ValueError(f"{what}: tensors on different devices ({dev}, {t.device})")
    # the kernels run on the current HIP device
    if dev is not None and dev.index != torch.cuda.current_device():
        raise ValueError(f"{what}: tensors on {dev}, current device is "
                         f"cuda:{torch.cuda.current_device()}")


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _used_on(stream, *tensors):
    """Tensors allocated here (on the current stream) and read or written by a
    call queued on another stream: tell the caching allocator, so that their
    memory is not handed out again before that stream has run the call."""
    if stream is not None and stream != torch.cuda.current_stream():
        for t in tensors:
            t.record_stream(stream)


def fpde_residual_fwd(op: int, fields, consts, h, coeffs, *, residual_out=None,
                      loss: Optional[torch.Tensor] = None, bc_mode: int = 0, stream=None):
    """Queue the fused forward stencil + loss; returns the float64 loss tensor."""
    shape = tuple(fields[0].shape)
    _check_tensors(list(fields) + list(consts), shape, "fpde_residual_fwd")
    dev = fields[0].device
    if loss is None:
        loss = torch.empty((), dtype=torch.float64, device=dev)
        _used_on(stream, loss)
    if loss.dtype != torch.float64 or loss.device != dev or loss.numel() != 1:
        raise ValueError("fpde_residual_fwd: loss must be a one-element float64 tensor on the "
                         "fields' device")
    res_arr = None
    if residual_out is not None:
        _check_tensors(residual_out, shape, "fpde_residual_fwd residual_out")
        res_arr = _ptr_array(residual_out)
    g, c = make_grid(shape, h, bc_mode), make_coeffs(coeffs)
    st = _entry("fpde_residual_fwd", shape)(int(op), ctypes.byref(g), ctypes.byref(c), _ptr_array(fields),
                                   _ptr_array(consts) if len(consts) else None, res_arr,
                                   loss.data_ptr(), _stream(stream))
    if st != FPDE_OK:
        raise FpdeError(st, "fpde_residual_fwd")
    return loss


def _grad_call(fn, name, op, fields, consts, h, coeffs, dloss, grads, bc_mode, stream):
    shape = tuple(fields[0].shape)
    _check_tensors(list(fields) + list(consts), shape, name)
    if grads is None:
        grads = [torch.empty_like(f) for f in fields]
        _used_on(stream, *grads)
    _check_tensors(grads, shape, name + " grads")
    if not isinstance(dloss, torch.Tensor):
        dloss = torch.tensor(float(dloss), dtype=torch.float64, device=fields[0].device)
        _used_on(stream, dloss)
    if dloss.dtype != torch.float64 or dloss.device != fields[0].device or dloss.numel() != 1:
        raise ValueError(f"{name}: dloss must be a one-element float64 tensor on the fields' device")
    g, c = make_grid(shape, h, bc_mode), make_coeffs(coeffs)
    st = fn(int(op), ctypes.byref(g), ctypes.byref(c), _ptr_array(fields),
            _ptr_array(consts) if len(consts) else None, dloss.data_ptr(), _ptr_array(grads),
            _stream(stream))
    if st != FPDE_OK:
        raise FpdeError(st, name)
    return grads


def fpde_residual_bwd(op: int, fields, consts, h, coeffs, dloss, *, grads=None, bc_mode: int = 0,
                      stream=None):
    """Queue the interior gather-form adjoint; returns the grads list."""
    return _grad_call(_entry("fpde_residual_bwd", fields[0].shape), "fpde_residual_bwd", op,
                      fields, consts, h, coeffs, dloss, grads, bc_mode, stream)


def fpde_bc_correct(op: int, fields, consts, h, coeffs, dloss, *, grads=None, bc_mode: int = 0,
                    stream=None):
    """Queue the boundary-shell correction; returns the grads list."""
    return _grad_call(_entry("fpde_bc_correct", fields[0].shape), "fpde_bc_correct", op,
                      fields, consts, h, coeffs, dloss, grads, bc_mode, stream)


def fpde_residual_value_and_grad(op: int, fields, consts, h, coeffs, dloss=1.0, *,
                                 loss: Optional[torch.Tensor] = None, grads=None,
                                 bc_mode: int = 0, stream=None):
    """Queue the one-pass loss + gradient (dloss known up front).  Returns
    (loss, grads): the float64 loss L and dloss * dL/dq for every field."""
    if loss is None:
        loss = torch.empty((), dtype=torch.float64, device=fields[0].device)
        _used_on(stream, loss)
    if loss.dtype != torch.float64 or loss.device != fields[0].device or loss.numel() != 1:
        raise ValueError("fpde_residual_value_and_grad: loss must be a one-element float64 "
                         "tensor on the fields' device")

    def fn(op_, g, c, fp, cp_, dl, gp, st):
        return _entry("fpde_residual_value_and_grad", fields[0].shape)(
            op_, g, c, fp, cp_, dl, loss.data_ptr(), gp, st)

    grads = _grad_call(fn, "fpde_residual_value_and_grad", op, fields, consts, h, coeffs, dloss,
                       grads, bc_mode, stream)
    return loss, grads


def fpde_residual_vjp(op: int, fields, h, coeffs, sens, *, grads=None, accumulate: bool = False,
                      bc_mode: int = 0, stream=None):
    """Queue the transposed-Jacobian action on upstream residual sensitivities
    ``sens`` (one full-size array per residual; read on the residual set only).
    Overwrites ``grads`` (allocated if None), or adds to them if ``accumulate``."""
    shape = tuple(fields[0].shape)
    _check_tensors(list(fields) + list(sens), shape, "fpde_residual_vjp")
    if grads is None:
        if accumulate:
            raise ValueError("fpde_residual_vjp: accumulate needs grads")
        grads = [torch.empty_like(f) for f in fields]
        _used_on(stream, *grads)
    _check_tensors(grads, shape, "fpde_residual_vjp grads")
    g, c = make_grid(shape, h, bc_mode), make_coeffs(coeffs)
    st = _entry("fpde_residual_vjp", shape)(int(op), ctypes.byref(g), ctypes.byref(c), _ptr_array(fields),
                                   _ptr_array(sens), int(bool(accumulate)), _ptr_array(grads),
                                   _stream(stream))
    if st != FPDE_OK:
        raise FpdeError(st, "fpde_residual_vjp")
    return grads


# ---------------------------------------------------------------------------
# Pre-marshalled calls.  Each call above validates its tensors and builds its
# ctypes arguments in Python, tens of microseconds of host time: more than the
# GPU time of the operator on small grids, where a loop of calls is then bound
# by the host.  bind(...) does that work once for fixed tensors and returns a
# callable that issues only the C call (which still validates its arguments).
# The callable keeps references to every tensor it was bound to, so their
# storage stays valid; their values may change between calls.

class BoundCall:
    """One entry point bound to fixed tensors, coefficients and stream."""

    def __init__(self, name, fn, args, keep, result):
        self.name, self._fn, self._args, self._keep, self.result = name, fn, args, keep, result

    def __call__(self):
        st = self._fn(*self._args)
        if st != FPDE_OK:
            raise FpdeError(st, self.name)
        return self.result


def bind(entry: str, op: int, fields, consts, h, coeffs, *, dloss=None, grads=None, loss=None,
         residual_out=None, sens=None, accumulate: bool = False, bc_mode: int = 0, stream=None):
    """Bind one entry point ("fwd", "bwd", "bc", "value_and_grad" or "vjp") to
    fixed tensors; the returned BoundCall queues the call each time it is
    called and returns what the unbound function returns (loss, grads or
    (loss, grads))."""
    shape = tuple(fields[0].shape)
    dev = fields[0].device
    consts = list(consts) if consts is not None else []
    _check_tensors(list(fields) + consts, shape, f"bind {entry}")
    g, c = make_grid(shape, h, bc_mode), make_coeffs(coeffs)
    fa = _ptr_array(fields)
    ca = _ptr_array(consts) if len(consts) else None
    sh = _stream(stream)
    lib = _load()
    keep = [g, c, fa, ca, list(fields), consts]
    if entry in ("fwd", "value_and_grad"):
        if loss is None:
            loss = torch.empty((), dtype=torch.float64, device=dev)
            _used_on(stream, loss)
        if loss.dtype != torch.float64 or loss.device != dev or loss.numel() != 1:
            raise ValueError(f"bind {entry}: loss must be a one-element float64 tensor on the "
                             "fields' device")
        keep.append(loss)
    if entry == "fwd":
        ra = None
        if residual_out is not None:
            _check_tensors(residual_out, shape, "bind fwd residual_out")
            ra = _ptr_array(residual_out)
            keep += [ra, list(residual_out)]
        args = (int(op), ctypes.byref(g), ctypes.byref(c), fa, ca, ra, loss.data_ptr(), sh)
        return BoundCall("fpde_residual_fwd", _entry("fpde_residual_fwd", shape), args, keep, loss)
    if grads is None:
        grads = [torch.empty_like(f) for f in fields]
        _used_on(stream, *grads)
    _check_tensors(grads, shape, f"bind {entry} grads")
    ga = _ptr_array(grads)
    keep += [ga, list(grads)]
    if entry == "vjp":
        _check_tensors(sens, shape, "bind vjp sensitivities")
        sa = _ptr_array(sens)
        keep += [sa, list(sens)]
        args = (int(op), ctypes.byref(g), ctypes.byref(c), fa, sa, int(bool(accumulate)), ga, sh)
        return BoundCall("fpde_residual_vjp", _entry("fpde_residual_vjp", shape), args, keep, grads)
    if not isinstance(dloss, torch.Tensor):
        dloss = torch.tensor(1.0 if dloss is None else float(dloss), dtype=torch.float64,
                             device=dev)
        _used_on(stream, dloss)
    if dloss.dtype != torch.float64 or dloss.device != dev or dloss.numel() != 1:
        raise ValueError(f"bind {entry}: dloss must be a one-element float64 tensor on the "
                         "fields' device")
    keep.append(dloss)
    if entry == "value_and_grad":
        args = (int(op), ctypes.byref(g), ctypes.byref(c), fa, ca, dloss.data_ptr(),
                loss.data_ptr(), ga, sh)
        return BoundCall("fpde_residual_value_and_grad",
                         _entry("fpde_residual_value_and_grad", shape), args, keep, (loss, grads))
    if entry not in ("bwd", "bc"):
        raise ValueError(f"bind: unknown entry point {entry!r}")
    name = "fpde_residual_bwd" if entry == "bwd" else "fpde_bc_correct"
    fn = _entry(name, shape)
    args = (int(op), ctypes.byref(g), ctypes.byref(c), fa, ca, dloss.data_ptr(), ga, sh)
    return BoundCall(name, fn, args, keep, grads)


class Residual(torch.autograd.Function):
    """Drop-in differentiable residual op: forward = the fused stencil writing
    the residual arrays (zero off the residual set), backward = the
    explicit-sensitivity transposed-Jacobian action on their gradients.

    Usage: ``R = Residual.apply(op, h, coeffs, consts, bc_mode, *fields)`` (a
    tuple with one tensor per residual); any objective of R can follow.
    """

    @staticmethod
    def forward(ctx, op, h, coeffs, consts, bc_mode, *fields):
        fields = [f.contiguous() for f in fields]
        ctx.op, ctx.h, ctx.coeffs, ctx.bc_mode = op, h, coeffs, bc_mode
        ctx.save_for_backward(*fields)
        nr = op_info(op)[3]
        R = [torch.empty_like(fields[0]) for _ in range(nr)]  # (every node is written)
        fpde_residual_fwd(op, fields, consts, h, coeffs, residual_out=R, bc_mode=bc_mode)
        return tuple(R)

    @staticmethod
    def backward(ctx, *gR):
        fields = list(ctx.saved_tensors)
        sens = [torch.zeros_like(fields[0]) if g is None else g.detach().float().contiguous()
                for g in gR]
        grads = fpde_residual_vjp(ctx.op, fields, ctx.h, ctx.coeffs, sens, bc_mode=ctx.bc_mode)
        return (None, None, None, None, None, *grads)


class ResidualLoss(torch.autograd.Function):
    """Drop-in differentiable loss op: forward = fused stencil + MSE loss,
    backward = interior adjoint + boundary correction with dloss = grad_output.

    Usage: ``loss = ResidualLoss.apply(op, h, coeffs, consts, *fields)``;
    ``ResidualLoss.apply(op, h, coeffs, consts, bc_mode, *fields)`` with an int
    ``bc_mode`` before the fields selects the boundary mode (0 by default).
    """

    @staticmethod
    def forward(ctx, op, h, coeffs, consts, *rest):
        bc_mode = 0
        ctx.n_lead = 4 + (len(rest) > 0 and not isinstance(rest[0], torch.Tensor))
        if ctx.n_lead == 5:
            bc_mode, rest = int(rest[0]), rest[1:]
        fields = [f.contiguous() for f in rest]
        ctx.op, ctx.h, ctx.coeffs, ctx.consts, ctx.bc_mode = op, h, coeffs, consts, bc_mode
        ctx.save_for_backward(*fields)
        return fpde_residual_fwd(op, fields, consts, h, coeffs, bc_mode=bc_mode)

    @staticmethod
    def backward(ctx, gout):
        fields = list(ctx.saved_tensors)
        dl = gout.detach().to(torch.float64).reshape(()).contiguous()
        kw = dict(bc_mode=ctx.bc_mode)
        grads = fpde_residual_bwd(ctx.op, fields, ctx.consts, ctx.h, ctx.coeffs, dl, **kw)
        fpde_bc_correct(ctx.op, fields, ctx.consts, ctx.h, ctx.coeffs, dl, grads=grads, **kw)
        return (None,) * ctx.n_lead + tuple(grads)
