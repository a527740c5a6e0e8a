"""The three-call step captured in a HIP graph (torch.cuda.CUDAGraph over the
ABI's calls; the library queues no memset, so the graph holds kernel nodes
only) and replayed several times, with eager work and synchronisations between
the replays: every replay recomputes from the current inputs and matches an
eager run on them (gradients bitwise, the loss to the float64 atomic order)."""
from __future__ import annotations

import pytest

from paper_2607_18020_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg,shape", [("ns_3d_tgv", (30, 40, 130)), ("ns_2d", (200, 600)),
                                       ("heat_3d", (19, 21, 130)), ("ns_3dt", (6, 19, 21, 70))])
def test_graph_replays_match_eager(cfg, shape):
    import torch  # noqa: PLC0415
    from paper_2607_18020_amd import binding as B  # noqa: PLC0415
    wl = W.make(cfg, seed=47, shape=shape)
    print(f"case graph {cfg} {shape}", flush=True)
    f = [torch.from_numpy(x).cuda() for x in wl.fields]
    c = [torch.from_numpy(x).cuda() for x in wl.consts]
    dl = torch.tensor(0.5, dtype=torch.float64, device="cuda")
    loss = torch.empty((), dtype=torch.float64, device="cuda")
    grads = [torch.empty_like(x) for x in f]

    def step():
        B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, loss=loss)
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl, grads=grads)
        B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=grads)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    e_loss = torch.empty_like(loss)
    e_grads = [torch.empty_like(x) for x in f]
    for r in range(4):
        with torch.no_grad():  # new inputs, written eagerly between the replays
            f[0].mul_(1.0 + 0.01 * (r + 1))
            f[-1].add_(0.003)
        grads_before = [x.clone() for x in grads]
        g.replay()
        torch.cuda.synchronize()
        B.fpde_residual_fwd(wl.op, f, c, wl.h, wl.coeffs, loss=e_loss)
        B.fpde_residual_bwd(wl.op, f, c, wl.h, wl.coeffs, dl, grads=e_grads)
        B.fpde_bc_correct(wl.op, f, c, wl.h, wl.coeffs, dl, grads=e_grads)
        torch.cuda.synchronize()
        assert abs(loss.item() - e_loss.item()) <= 1e-12 * abs(e_loss.item()), (r, loss, e_loss)
        for a, b, old in zip(grads, e_grads, grads_before):
            assert torch.equal(a, b), r
            assert not torch.equal(a, old), r  # the replay recomputed
