"""Host-side parts of bench.py (no GPU): the byte model, the all-core CPU
baseline, whose slab passes must reproduce the whole-grid oracle, the parity
verdict, the choice of the profile record behind roofline.traffic, and the
refusal of more than one GPU."""
from __future__ import annotations

import numpy as np
import pytest

import bench
from paper_2607_18020_amd import workloads as W


@pytest.mark.parametrize("bc_mode", [0, 1])
@pytest.mark.parametrize("cfg,shape,cores", [("ns_3d_tgv", (23, 12, 17), 5),
                                             ("ns_3d_tgv", (7, 9, 10), 6),
                                             ("heat_3d", (19, 8, 9), 3),
                                             ("ns_2d", (30, 21), 4),
                                             ("burgers_1dt", (9, 40), 8)])
def test_slab_oracle_matches_whole_grid(oracle_mod, cfg, shape, cores, bc_mode):
    """Overlapping axis-0 slabs, each through the unchanged oracle: the loss and
    the gradient at every node equal the whole-grid oracle's (up to the order
    of the float64 loss sum)."""
    wl = W.make(cfg, seed=42, shape=shape)
    _, reps, _, (L, g) = bench.oracle_all_cores(wl, bc_mode, cores, min_s=0.0)
    assert reps == 1
    args = (wl.op, wl.shape, wl.h, wl.coeffs, wl.fields, wl.consts)
    Lr = oracle_mod.loss(*args, bc_mode=bc_mode)
    gr = oracle_mod.grad(*args, dloss=1.0, bc_mode=bc_mode)
    assert L == pytest.approx(Lr, rel=1e-13)
    for a, b in zip(g, gr):
        assert a.shape == b.shape
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13 * np.abs(b).max())


def test_byte_model_ns3d():
    wl = W.make("ns_3d_tgv", seed=42, shape=(10, 11, 12))
    N, M = wl.n_points, wl.n_residual_points
    bm = bench.byte_model(wl)
    assert bm["per_node"] == 72
    assert bm["fwd"] == 28 * N + 8 and bm["bwd"] == 28 * N + 16 * M
    assert bench.byte_model(wl, path="fused")["per_node"] == 44


def test_parity_verdict():
    ref = {"loss": 2.0, "grads": [np.ones(4)]}
    ok = bench.parity_of((2.0 * (1 + 5e-6), [np.ones(4) * (1 + 5e-5)], None), ref)
    bad = bench.parity_of((2.0 * (1 + 2e-5), [np.ones(4)], None), ref)
    assert ok["ok"] and not bad["ok"]


def test_measured_traffic_only_for_matching_records(tmp_path, monkeypatch):
    """roofline.traffic comes from the profile record of the same workload and
    bench path, summed over the named kernels, and only while the record's
    kernel-source hash is the current one."""
    import json  # noqa: PLC0415

    from paper_2607_18020_amd import profiling  # noqa: PLC0415
    (tmp_path / "profiles").mkdir()
    rec = {"source_hash": "abc", "workload": "ns_3d_tgv 256^3", "path": "loss",
           "kernels": {"bwd_kernel<OpNS<3, true>, 128, 8, true, false, false>":
                       {"fetch_bytes": 100.0, "write_bytes": 20.0},
                       "fill_f64_kernel": {"fetch_bytes": 1.0, "write_bytes": 0.0}}}
    (tmp_path / "profiles" / "traffic_x.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(profiling, "source_hash", lambda root=None: "abc")
    op = W.CONFIGS["ns_3d_tgv"].op
    assert bench.measured_traffic("ns_3d_tgv", op, ["bwd"]) == 120
    assert bench.measured_traffic("ns_3d_tgv", op, ["bwd", "fill_f64"]) == 121
    assert bench.measured_traffic("ns_3d_tgv", op, ["bwd"], path="fused") is None
    assert bench.measured_traffic("heat_3d", op, ["bwd"]) is None
    assert bench.measured_traffic("ns_3d_tgv", op, ["fwd"]) is None  # no such kernel
    monkeypatch.setattr(profiling, "source_hash", lambda root=None: "changed")
    assert bench.measured_traffic("ns_3d_tgv", op, ["bwd"]) is None


def test_more_than_one_gpu_is_refused():
    """bench.py measures one GPU: --gpus above 1 exits with status 2 and says
    so, before touching a GPU."""
    import os  # noqa: PLC0415
    import subprocess  # noqa: PLC0415
    import sys  # noqa: PLC0415
    root = os.path.dirname(os.path.abspath(bench.__file__))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
