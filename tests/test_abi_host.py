"""Host-side checks of the C ABI (no GPU): exports, op table, validation.

Every call here is invalid in at least one argument, so the library returns
before queueing any GPU work; the fake device addresses are never touched.
"""
from __future__ import annotations

import ctypes
import os
import re
import types

import pytest

from paper_2607_18020_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fpde.h")


@pytest.fixture(scope="module")
def B():
    from paper_2607_18020_amd import binding  # noqa: PLC0415
    try:
        binding.lib()
    except ImportError as e:  # pragma: no cover
        pytest.fail(f"libfpde.so missing: {e}")
    return binding


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fpde_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol(B):
    decl = _declared_functions()
    assert set(decl) == set(B.EXPORTED)
    lib = B.lib()
    for name in decl:
        assert hasattr(lib, name), name


def test_op_info_matches_workload_registry(B):
    for op, spec in W.OPS.items():
        ndim, nf, nc, nr = B.op_info(op)
        assert (ndim, nf, nc, nr) == (spec.ndim, len(spec.fields), len(spec.consts), len(spec.residuals))
    with pytest.raises(B.FpdeError):
        B.op_info(0)
    with pytest.raises(B.FpdeError):
        B.op_info(len(W.OPS) + 1)


def test_status_strings_and_version(B):
    lib = B.lib()
    for code, name in B.STATUS_NAMES.items():
        assert lib.fpde_status_string(code).decode().startswith(name)
    assert b"unknown" in lib.fpde_status_string(12345)
    assert b"gfx950" in lib.fpde_version()


# fake, 256-byte-aligned "device" addresses: never dereferenced (every call below is invalid)
BASE = 0x7F0000000000
STRIDE = 1 << 32


def _addr(i, off=0):
    return BASE + i * STRIDE + off


def _arr(vals):
    a = (ctypes.c_void_p * max(1, len(vals)))()
    for i, v in enumerate(vals):
        a[i] = v
    return a


def _call(B, fn, op, shape, h=None, coef=W.Coeffs(nu=0.01, k=1.0, dt=0.1, alpha=0.1),
          fields=None, consts=None, outs=None, scalar=None, bc_mode=0, ndim=None, sens=None,
          accumulate=0, loss=None, four=False):
    """One call of entry point `fn`; four-axis grids (or four=True) go through
    the entry points taking fpde_grid4."""
    spec = W.OPS[op]
    h = h if h is not None else (0.1,) * len(shape)
    four = four or len(shape) == 4
    g = B.make_grid(shape, h, bc_mode)
    if four and len(shape) < 4:
        g4 = B.FpdeGrid4()
        g4.ndim, g4.bc_mode = g.ndim, g.bc_mode
        for a in range(len(shape)):
            g4.n[a], g4.h[a] = g.n[a], g.h[a]
        g = g4
    lib = types.SimpleNamespace(**{n: getattr(B.lib(), n + ("4" if four else ""))
                                   for n in B.CALLS})
    if ndim is not None:
        g.ndim = ndim
    c = B.make_coeffs(coef)
    nf, nc, nr = len(spec.fields), len(spec.consts), len(spec.residuals)
    fields = fields if fields is not None else [_addr(i) for i in range(nf)]
    consts = consts if consts is not None else [_addr(10 + j) for j in range(nc)]
    scalar = _addr(30) if scalar is None else scalar
    if fn == "fwd":
        outs = outs if outs is not None else None
        return lib.fpde_residual_fwd(op, ctypes.byref(g), ctypes.byref(c), _arr(fields),
                                     _arr(consts) if nc else None,
                                     _arr(outs) if outs is not None else None, scalar, None)
    outs = outs if outs is not None else [_addr(20 + i) for i in range(nf)]
    if fn == "vjp":
        sens = sens if sens is not None else [_addr(40 + b) for b in range(nr)]
        return lib.fpde_residual_vjp(op, ctypes.byref(g), ctypes.byref(c), _arr(fields),
                                     _arr(sens), accumulate, _arr(outs), None)
    if fn == "vg":
        loss = _addr(31) if loss is None else loss
        return lib.fpde_residual_value_and_grad(op, ctypes.byref(g), ctypes.byref(c), _arr(fields),
                                                _arr(consts) if nc else None, scalar, loss,
                                                _arr(outs), None)
    f = lib.fpde_residual_bwd if fn == "bwd" else lib.fpde_bc_correct
    return f(op, ctypes.byref(g), ctypes.byref(c), _arr(fields), _arr(consts) if nc else None,
             scalar, _arr(outs), None)


ARG, SHAPE, SPACING, COEFF, ALIGN, UNSUP = -1, -2, -3, -4, -5, -7


@pytest.mark.parametrize("fn", ["fwd", "bwd", "bc", "vjp", "vg"])
def test_validation_status_codes(B, fn):
    op3, op2 = W.NS_3D_BE, W.NS_2D_STEADY
    s3 = (8, 9, 10)
    lib = B.lib()
    g = B.make_grid(s3, (0.1,) * 3)
    c = B.make_coeffs(W.Coeffs())
    z = _arr([_addr(0)] * 4)
    if fn == "fwd":  # unknown op, null grid
        assert lib.fpde_residual_fwd(0, ctypes.byref(g), ctypes.byref(c), z, z, None, _addr(30), None) == ARG
        assert lib.fpde_residual_fwd(op3, None, ctypes.byref(c), z, z, None, _addr(30), None) == ARG
    # wrong rank, too small, bad spacing, bad coefficients
    assert _call(B, fn, op3, s3, ndim=2) == SHAPE
    assert _call(B, fn, op3, (2, 9, 10)) == SHAPE
    assert _call(B, fn, op2, (9, 2)) == SHAPE
    assert _call(B, fn, op3, s3, h=(0.1, 0.0, 0.1)) == SPACING
    assert _call(B, fn, op3, s3, h=(0.1, float("nan"), 0.1)) == SPACING
    assert _call(B, fn, op3, s3, h=(0.1, 0.1, -1.0)) == SPACING
    assert _call(B, fn, op3, s3, coef=W.Coeffs(nu=0.01, dt=0.0)) == COEFF
    assert _call(B, fn, op3, s3, coef=W.Coeffs(nu=float("inf"), dt=0.1)) == COEFF
    assert _call(B, fn, W.HEAT_3D_BE, s3, coef=W.Coeffs(dt=-1.0, alpha=0.1)) == COEFF
    # null field / const pointers
    assert _call(B, fn, op3, s3, fields=[_addr(0), 0, _addr(2), _addr(3)]) == ARG
    if fn != "vjp":
        assert _call(B, fn, op3, s3, consts=[_addr(10), _addr(11), 0]) == ARG
    # misaligned field
    assert _call(B, fn, op3, s3, fields=[_addr(0), _addr(1, 2), _addr(2), _addr(3)]) == ALIGN
    # an unknown boundary mode
    assert _call(B, fn, op3, s3, bc_mode=7) == ARG
    # size limits: a plane of the non-marching axes below 2^29 nodes, every n_a below 2^31
    assert _call(B, fn, op3, (3, 1 << 14, 1 << 15)) == SHAPE
    assert _call(B, fn, op3, (3, 1 << 15, 1 << 14)) == SHAPE
    assert _call(B, fn, op2, (3, 1 << 29)) == SHAPE
    assert _call(B, fn, op2, (1 << 31, 5)) == SHAPE
    # every launch shape stays below 2^31 workgroups (so the node count below 2^36)
    assert _call(B, fn, op2, (1 << 26, 1 << 10)) == SHAPE
    assert _call(B, fn, op3, (1 << 20, 1 << 10, 1 << 10)) == SHAPE
    # the longest first axis the rank checks allow (the count is taken in 64 bits)
    assert _call(B, fn, op2, ((1 << 31) - 1, 3)) == SHAPE
    assert _call(B, fn, op3, ((1 << 31) - 1, 9, 9)) == SHAPE


@pytest.mark.parametrize("fn", ["fwd", "bwd", "bc", "vjp", "vg"])
def test_validation_four_axis_grids(B, fn):
    """fpde_grid4 and the entry points ending in 4: the 3D+t operator's grid,
    and every other op through the same calls."""
    op = W.NS_3DT
    s4 = (6, 7, 8, 9)
    assert _call(B, fn, op, s4, ndim=3) == SHAPE
    assert _call(B, fn, op, (2, 7, 8, 9)) == SHAPE
    assert _call(B, fn, op, (6, 7, 8, 2)) == SHAPE
    assert _call(B, fn, op, s4, h=(0.0, 0.1, 0.1, 0.1)) == SPACING  # the time step
    assert _call(B, fn, op, s4, h=(0.1, 0.1, 0.1, float("inf"))) == SPACING
    assert _call(B, fn, op, s4, coef=W.Coeffs(nu=float("nan"))) == COEFF
    assert _call(B, fn, op, s4, fields=[_addr(0), _addr(1), 0, _addr(3)]) == ARG
    assert _call(B, fn, op, s4, fields=[_addr(0), _addr(1), _addr(2, 2), _addr(3)]) == ALIGN
    assert _call(B, fn, op, s4, bc_mode=2) == ARG
    # a time level (the last three axes) below 2^29 nodes; the launches below 2^31 workgroups
    assert _call(B, fn, op, (3, 1 << 10, 1 << 10, 1 << 9)) == SHAPE
    assert _call(B, fn, op, (1 << 20, 1 << 8, 1 << 8, 1 << 8)) == SHAPE
    # the three-axis ops through fpde_grid4, and four axes refused by fpde_grid
    assert _call(B, fn, W.NS_3D_BE, (8, 9, 10), ndim=2, four=True) == SHAPE
    assert _call(B, fn, W.NS_3D_BE, (8, 9, 10), h=(0.1, 0.0, 0.1), four=True) == SPACING
    assert _call(B, fn, W.NS_2D_STEADY, (9, 2), four=True) == SHAPE
    assert _call(B, fn, W.NS_3D_BE, (8, 9, 10), ndim=4) == SHAPE


def test_output_checks(B):
    op = W.NS_3D_BE
    s3 = (8, 9, 10)
    nbytes = 8 * 9 * 10 * 4
    # fwd: null loss, misaligned loss, loss inside a field, residual aliasing a field
    assert _call(B, "fwd", op, s3, scalar=0) == ARG
    assert _call(B, "fwd", op, s3, scalar=_addr(30, 4)) == ALIGN
    assert _call(B, "fwd", op, s3, scalar=_addr(2, 64)) == ARG
    assert _call(B, "fwd", op, s3, outs=[_addr(20), _addr(21), _addr(1, 4 * 10), _addr(23)]) == ARG
    assert _call(B, "fwd", op, s3, outs=[_addr(20), 0, _addr(22), _addr(23)]) == ARG
    assert _call(B, "fwd", op, s3, outs=[_addr(20), _addr(20, nbytes - 4), _addr(22), _addr(23)]) == ARG
    # value_and_grad: null / misaligned loss, loss on dloss, inside a field, const or grad
    assert _call(B, "vg", op, s3, loss=0) == ARG
    assert _call(B, "vg", op, s3, loss=_addr(31, 4)) == ALIGN
    assert _call(B, "vg", op, s3, loss=_addr(30)) == ARG
    assert _call(B, "vg", op, s3, loss=_addr(2, 64)) == ARG
    assert _call(B, "vg", op, s3, loss=_addr(11, 8)) == ARG
    assert _call(B, "vg", op, s3, loss=_addr(22, nbytes - 8)) == ARG
    for fn in ("bwd", "bc", "vg"):
        # null / misaligned dloss, grads aliasing fields, consts, each other or dloss
        assert _call(B, fn, op, s3, scalar=0) == ARG
        assert _call(B, fn, op, s3, scalar=_addr(30, 4)) == ALIGN
        assert _call(B, fn, op, s3, outs=[_addr(20), _addr(0), _addr(22), _addr(23)]) == ARG
        assert _call(B, fn, op, s3, outs=[_addr(20), _addr(21), _addr(11, 8), _addr(23)]) == ARG
        assert _call(B, fn, op, s3, outs=[_addr(20), _addr(21), _addr(21), _addr(23)]) == ARG
        assert _call(B, fn, op, s3, outs=[_addr(20), _addr(21), _addr(22), _addr(30, 0)],
                     scalar=_addr(30, 16)) == ARG
        assert _call(B, fn, op, s3, outs=[_addr(20), _addr(21), _addr(22), _addr(23, 2)]) == ALIGN
    # vjp: accumulate flag, null / misaligned sensitivities, grads aliasing fields,
    # sensitivities or each other
    assert _call(B, "vjp", op, s3, accumulate=2) == ARG
    assert _call(B, "vjp", op, s3, accumulate=-1) == ARG
    assert _call(B, "vjp", op, s3, sens=[_addr(40), 0, _addr(42), _addr(43)]) == ARG
    assert _call(B, "vjp", op, s3, sens=[_addr(40), _addr(41, 2), _addr(42), _addr(43)]) == ALIGN
    assert _call(B, "vjp", op, s3, outs=[_addr(20), _addr(1, 8), _addr(22), _addr(23)]) == ARG
    assert _call(B, "vjp", op, s3, outs=[_addr(20), _addr(21), _addr(42, nbytes - 4), _addr(23)]) == ARG
    assert _call(B, "vjp", op, s3, outs=[_addr(20), _addr(20), _addr(22), _addr(23)]) == ARG
    assert _call(B, "vjp", op, s3, outs=[_addr(20), _addr(21), 0, _addr(23)]) == ARG
    assert _call(B, "vjp", op, s3, outs=[_addr(20), _addr(21), _addr(22), _addr(23, 2)]) == ALIGN


def test_product_path_shares_nothing_with_the_oracle():
    """The HIP path neither imports, includes nor links the oracle."""
    pkg = os.path.join(ROOT, "paper_2607_18020_amd")
    for dirpath, _, files in os.walk(pkg):
        for fn in files:
            if fn.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                src = open(os.path.join(dirpath, fn)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle\b", src, re.M), fn
                assert "fpde_oracle" not in src, fn
                assert "orc_" not in src, fn


def test_no_fallback_without_the_library_or_a_gpu(B, tmp_path):
    """The binding has no CPU path: without the built library every entry point
    raises ImportError, and host (CPU) tensors are refused before any call."""
    import torch  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=1, shape=(5, 6, 7))
    f = [torch.from_numpy(x) for x in wl.fields]
    c = [torch.from_numpy(x) for x in wl.consts]
    with pytest.raises(ImportError):
        with B.library(str(tmp_path / "libfpde_missing.so")):
            pass
    assert B.lib() is not None  # (the product library again after the block)
    with pytest.raises(ValueError, match="CUDA"):
        B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs)
    with pytest.raises(ValueError, match="CUDA"):
        B.fpde_residual_vjp(wl.op, f, wl.h, wl.coeffs, [x.clone() for x in f])
