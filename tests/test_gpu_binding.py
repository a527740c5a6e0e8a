"""The Python binding's argument checks (marshalling only): tensors that the C
ABI cannot take are refused before any call, with ValueError; ABI status codes
come back as FpdeError."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_18020_amd import workloads as W

pytestmark = pytest.mark.gpu


def _inputs():
    import torch  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=42, shape=(6, 7, 70))
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    return wl, f, c


def test_binding_refuses_unusable_tensors():
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl, f, c = _inputs()
    with pytest.raises(ValueError):  # a host tensor
        B.fpde_residual_fwd(wl.op, [f[0].cpu()] + f[1:], c, wl.h, wl.coeffs)
    with pytest.raises(ValueError):  # float64
        B.fpde_residual_fwd(wl.op, [f[0].double()] + f[1:], c, wl.h, wl.coeffs)
    with pytest.raises(ValueError):  # not contiguous
        B.fpde_residual_fwd(wl.op, [f[0].transpose(1, 2).contiguous().transpose(1, 2)] + f[1:],
                            c, wl.h, wl.coeffs)
    with pytest.raises(ValueError):  # shapes differ
        B.fpde_residual_fwd(wl.op, f, [c[0][:, :, :-1].contiguous()] + c[1:], wl.h, wl.coeffs)
    with pytest.raises(ValueError):  # loss of the wrong type
        B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs,
                            loss=torch.empty((), dtype=torch.float32, device="cuda"))
    dl_host = torch.ones((), dtype=torch.float64)
    with pytest.raises(ValueError):  # dloss on the host
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl_host)
    with pytest.raises(ValueError):  # value-and-grad loss on the host
        B.fpde_residual_value_and_grad(wl.op, f, c, wl.h, wl.coeffs, 1.0,
                                       loss=torch.empty((), dtype=torch.float64))
    with pytest.raises(ValueError):  # accumulate into nothing
        B.fpde_residual_vjp(wl.op, f, wl.h, wl.coeffs, [torch.zeros_like(f[0])] * 4,
                            accumulate=True)


def test_binding_reports_abi_status():
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl, f, c = _inputs()
    # grads aliasing a field: the library refuses with FPDE_ERR_ARG and queues nothing
    with pytest.raises(B.FpdeError) as e:
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, 1.0, grads=[f[0]] + f[1:])
    assert e.value.status == -1
    # a spacing of zero: FPDE_ERR_SPACING
    with pytest.raises(B.FpdeError) as e:
        B.fpde_residual_fwd(wl.op, f, c, (wl.h[0], 0.0, wl.h[2]), wl.coeffs)
    assert e.value.status == -3
    torch.cuda.synchronize()


@pytest.mark.parametrize("cfg", ["ns_3d_tgv", "ns_2d"])
def test_bound_calls_match_unbound(cfg):
    """bind(...) only moves the marshalling out of the call: the same kernels on
    the same tensors, so the same results (gradients bitwise; the loss up to
    the order of its float64 atomics)."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make(cfg, seed=44, shape=(9, 20, 70) if cfg == "ns_3d_tgv" else (30, 300))
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    dl = torch.tensor(0.75, dtype=torch.float64, device="cuda")
    L0 = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs)
    g0 = B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl)
    B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g0)
    Lv0, gv0 = B.fpde_residual_value_and_grad(wl.op, f, c, wl.h, wl.coeffs, dl)
    sens = [torch.from_numpy(x).cuda() for x in W.sensitivities(wl.op, wl.shape, 3)]
    gj0 = B.fpde_residual_vjp(wl.op, f, wl.h, wl.coeffs, sens)
    fwd = B.bind("fwd", wl.op, f, c, wl.h, wl.coeffs)
    bwd = B.bind("bwd", wl.op, f, c, wl.h, wl.coeffs, dloss=dl)
    bc = B.bind("bc", wl.op, f, c, wl.h, wl.coeffs, dloss=dl, grads=bwd.result)
    vg = B.bind("value_and_grad", wl.op, f, c, wl.h, wl.coeffs, dloss=dl)
    vj = B.bind("vjp", wl.op, f, None, wl.h, wl.coeffs, sens=sens)
    for _ in range(3):  # repeated calls reuse the bound arguments
        L1 = fwd()
        g1 = bwd()
        bc()
        Lv1, gv1 = vg()
        gj1 = vj()
        torch.cuda.synchronize()
        assert abs(L1.item() - L0.item()) <= 1e-12 * abs(L0.item())
        assert abs(Lv1.item() - Lv0.item()) <= 1e-12 * abs(Lv0.item())
        for a, b in zip(g1 + gv1 + gj1, g0 + gv0 + gj0):
            assert torch.equal(a, b)
    with pytest.raises(ValueError):
        B.bind("nonsense", wl.op, f, c, wl.h, wl.coeffs)


def test_calls_on_side_streams_run_concurrently_and_agree():
    """Every call is queued on the stream it is given: two problems queued on two
    side streams (default priority) at once give the results of the same calls
    on the current stream."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wls = [W.make("ns_3d_tgv", seed=45, shape=(30, 40, 130)),
           W.make("heat_3d", seed=46, shape=(30, 40, 130))]
    ins = [([torch.from_numpy(x).cuda() for x in wl.fields],
            [torch.from_numpy(x).cuda() for x in wl.consts]) for wl in wls]
    ref = []
    for wl, (f, c) in zip(wls, ins):
        L = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs)
        g = B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, 1.0)
        B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, 1.0, grads=g)
        ref.append((L, g))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    out = []
    for s in streams:  # inputs were written on the current stream
        s.wait_stream(torch.cuda.current_stream())
    for wl, (f, c), s in zip(wls, ins, streams):
        with torch.cuda.stream(s):  # (dloss filled on the stream that reads it)
            dl = torch.ones((), dtype=torch.float64, device="cuda")
            L = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, stream=s)
            g = B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl, stream=s)
            B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g, stream=s)
        out.append((L, g))
    torch.cuda.synchronize()
    for (L0, g0), (L1, g1) in zip(ref, out):
        assert abs(L1.item() - L0.item()) <= 1e-12 * abs(L0.item())
        for a, b in zip(g0, g1):
            assert torch.equal(a, b)


def test_side_stream_calls_keep_the_buffers_they_allocate():
    """The dloss scalar made from a Python float, and the loss and grads that the
    binding allocates for a call queued on another stream, stay reserved for that
    stream until it has run the call: new tensors filled on the current stream
    while the side stream is still busy do not take their memory."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make("ns_3d_tgv", seed=47, shape=(20, 30, 70))
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    dl = torch.full((), 0.5, dtype=torch.float64, device="cuda")
    L0 = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs)
    g0 = B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl)
    B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=g0)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # keep the side stream busy for a while
        busy = torch.empty(1 << 26, device="cuda")
        for _ in range(4):
            busy.fill_(1.0)
    # queued on s from the current stream's context
    L1 = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, stream=s)
    g1 = B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, 0.5, stream=s)
    B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, 0.5, grads=g1, stream=s)
    junk = [torch.full((), 1e30, dtype=torch.float64, device="cuda") for _ in range(64)]
    junk += [torch.full_like(f[0], 1e30) for _ in range(4)]
    torch.cuda.synchronize()
    del busy, junk
    assert abs(L1.item() - L0.item()) <= 1e-12 * abs(L0.item())
    for a, b in zip(g0, g1):
        assert torch.equal(a, b)


@pytest.mark.parametrize("cfg", ["ns_3d_tgv", "ns_2d", "heat_3d"])
def test_arrays_at_any_4_byte_offset(cfg):
    """The ABI asks only for 4-byte-aligned arrays: inputs, outputs and the
    sensitivities placed 4, 8 and 12 bytes past a 256-byte boundary (views into
    larger buffers) give bitwise the results of freshly allocated arrays, for
    every entry point."""
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    shape = (11, 20, 133) if len(W.CONFIGS[cfg].shape) == 3 else (37, 300)
    wl = W.make(cfg, seed=48, shape=shape)
    n = int(np.prod(shape))
    nf = len(wl.fields)
    nr = len(wl.spec.residuals)
    sens_np = W.sensitivities(wl.op, shape, 49)

    def placed(k, src=None):
        buf = torch.empty(n + 64, dtype=torch.float32, device="cuda")
        v = buf[k:k + n].view(shape)
        if src is not None:
            v.copy_(torch.from_numpy(src))
        return buf, v

    def run(off):
        keep = []
        def arr(src=None):
            if off is None:
                return torch.from_numpy(src).cuda() if src is not None else \
                    torch.empty(shape, dtype=torch.float32, device="cuda")
            b, v = placed(off, src)
            keep.append(b)
            return v
        f = [arr(x) for x in wl.fields]
        c = [arr(x) for x in wl.consts]
        R = [arr() for _ in range(nr)]
        L = B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, residual_out=R)
        g = [arr() for _ in range(nf)]
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, 1.0, grads=g)
        B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, 1.0, grads=g)
        gv = [arr() for _ in range(nf)]
        Lv, _ = B.fpde_residual_value_and_grad(wl.op, f, c, wl.h, wl.coeffs, 1.0, grads=gv)
        s = [arr(x) for x in sens_np]
        gs = [arr() for _ in range(nf)]
        B.fpde_residual_vjp(wl.op, f, wl.h, wl.coeffs, s, grads=gs)
        torch.cuda.synchronize()
        out = [x.cpu() for x in R + g + gv + gs]
        return out, L.item(), Lv.item()

    ref, L0, Lv0 = run(None)
    for off in (1, 2, 3):
        print(f"case {cfg} {shape} arrays at +{4 * off} bytes", flush=True)
        out, L, Lv = run(off)
        assert all(torch.equal(a, b) for a, b in zip(ref, out))
        assert abs(L - L0) <= 1e-12 * abs(L0) and abs(Lv - Lv0) <= 1e-12 * abs(Lv0)
