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
def kernels(tmp_path_factory):
    path = str(tmp_path_factory.mktemp("isa") / "fpde.s")
    R.compile_asm(path)
    return R.parse(open(path).read())


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
