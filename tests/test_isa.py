"""The kernels' own gfx950 assembly keeps the design (static, no GPU needed):
plane loads streamed straight into LDS and LDS stencil reads in the marching
kernels, a DPP wavefront sum and exactly one float64 atomic instruction in the
kernels that reduce the loss, no atomics in the gather-form backward, the
boundary kernel or the vjp, no MFMA, no packed-FP32 VALU and no register
spills anywhere."""
from __future__ import annotations

import os
import shutil

import pytest

from paper_2607_18020_amd import isa_report as R

pytestmark = pytest.mark.skipif(shutil.which(R.B.HIPCC) is None and not os.path.exists(R.B.HIPCC),
                                reason="hipcc not available")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    path = str(tmp_path_factory.mktemp("isa") / "fpde.s")
    R.compile_asm(path)
    return open(path).read()


@pytest.fixture(scope="module")
def kernels(asm):
    return R.parse(asm)


def test_design_rules(kernels):
    assert len(kernels) > 50
    assert R.violations(kernels) == []


def test_ns3d_kernels(kernels):
    fwd = kernels["fwd_kernel<OpNS<3, true>, 128, 4, false, false, 4>"]
    bwd = kernels["bwd_kernel<OpNS<3, true>, 128, 8, true, false, false>"]
    vg = kernels["bwd_kernel<OpNS<3, true>, 128, 8, true, true, false>"]
    bc = kernels["bc_kernel<OpNS<3, true> >"]
    for k in (fwd, bwd, vg):
        assert k["lds_dma"] > 0 and k["ds_read"] > 0 and k["barrier"] > 0
    assert fwd["atomic"] == 1 and fwd["dpp"] >= 6
    assert bwd["atomic"] == 0 and bwd["ds_write"] > 0  # residual tiles written to LDS
    assert vg["atomic"] == 1 and vg["dpp"] >= 6
    assert bc["atomic"] == 0
    # float64 arithmetic only where the divergence residual is summed and the loss accumulated
    assert 0 < fwd["f64"] < fwd["valu"] // 4


def test_2d_forward_has_no_lds_march(kernels):
    k = kernels["fwdq_kernel<OpNS<2, false>, 1024, 1, 6, false, false>"]
    assert k["lds_dma"] == 0 and k["atomic"] == 1 and k["dpp"] >= 6
    assert k["barrier"] <= 2  # only the workgroup sum of the loss


def _ring_stream_is_safe(P, NC, X, RD, CD, waits, steps=40):
    """Simulate the forward's operation stream (prologue: RD - 1 plane groups of
    P loads, then CD - 1 const groups; each step: P plane loads, NC const loads,
    X stores) and check that at the end of every step w, the wait for at most
    waits(w) operations in flight leaves none of the loads of plane w + 2
    (relative to the chunk's first plane), which step w + 1 reads first, in
    flight: operations retire in order."""
    ops, ends = [], []
    for j in range(RD - 1):
        ops += [("plane", j - 1)] * P
    ops += [("const",)] * ((CD - 1) * NC)
    for w in range(steps):
        ops += [("plane", w + RD - 2)] * P + [("const",)] * NC + [("store",)] * X
        ends.append(len(ops))
    for w in range(steps - 1):
        last = max(i for i, o in enumerate(ops[:ends[w]]) if o == ("plane", w + 2))
        if ends[w] - 1 - last < waits(w):
            return False
    return True


@pytest.mark.parametrize("store_r", [False, True])
@pytest.mark.parametrize("per", [False, True])
def test_eight_slot_forward_waits(asm, store_r, per):
    """The heat forward's 8-slot ring waits at each barrier, by an explicit
    count, only for the plane the next step reads first.  Those counts hold if
    the compiled kernel issues its memory operations as the count assumes: the
    prologue's RD - 1 plane groups before its CD - 1 const loads, and in every
    step the plane loads, the const loads and the stores, nothing merged or
    added.  Checked here on the kernel's own assembly, and the counts checked
    against a simulation of that stream."""
    TX, TY, NT, RD = 256, 4, 1024, 8
    CD = RD // 2
    P = ((TY + 2) * TX + 64 + 63) // 64 * 64 // NT + (((TY + 2) * TX + 64) % NT != 0)  # load rounds
    NC, X = 1, int(store_r)
    S = P + NC + X
    k_in = (S - P) + (RD - 4) * S
    early = [min((RD - 5 - w) * P + (CD - 1) * NC + (w + 1) * S, k_in) for w in range(RD - 4)]
    assert _ring_stream_is_safe(P, NC, X, RD, CD, lambda w: early[w] if w < RD - 4 else k_in)
    # the counts are tight: one more in flight at the steady barrier would not be safe
    assert not _ring_stream_is_safe(P, NC, X, RD, CD,
                                    lambda w: early[w] if w < RD - 4 else k_in + 1)
    name = f"fwd_kernel<OpHeat, {TX}, {TY}, {str(store_r).lower()}, {str(per).lower()}, {RD}>"
    s = R.memory_stream(asm, name)
    # the formula's counts are in the kernel; any other barrier wait is below the
    # smallest of them, and safe anywhere (the prologue's and the loss sum's
    # barriers wait for more)
    waits = {int(t[1:]) for t in s if t.startswith("W")}
    assert set(early) | {k_in} <= waits, (waits, early, k_in)
    assert all(n in set(early) | {k_in} or n < min(early) for n in waits), (waits, early, k_in)
    # prologue: the end planes' zero stores (non-periodic grids with residuals),
    # the plane groups, then the const loads, then the barrier
    pro = "".join(t for t in s[:s.index("B")] if not t.startswith("W")).lstrip("S")
    assert pro == "D" * ((RD - 1) * P) + "L" * ((CD - 1) * NC), pro
    # every step issues its plane loads first, then its const loads and stores
    # (the last step of a chunk may drop a const nothing reads); in code order a
    # step whose barrier has alternatives (early or steady count) is followed by
    # segments that hold only those waits
    counted = {f"W{n}" for n in set(early) | {k_in}}
    steps, seg = 0, []
    for t in s[s.index("B") + 1:]:
        if t == "A":  # the loss sum's atomic (blocks placed after it belong to the march)
            seg = []
        elif t == "B":
            body = "".join(x for x in seg if not x.startswith("W"))
            if body and any(x in counted for x in seg):  # a march step
                assert body.startswith("D" * P) and body.count("D") == P, body
                assert body[P:] in ("L" * NC + "S" * X, "S" * X), body
                steps += 1
            seg = []
        else:
            seg.append(t)
    assert steps >= RD  # the unrolled march and its tail
