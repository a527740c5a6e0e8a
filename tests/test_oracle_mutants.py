"""The oracle pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a copy of the oracle's C source (a flipped
sign, a transposed operand, a wrong normaliser, a dropped Jacobian term, a
coefficient off by one part in 1e7, a spacing taken from the wrong axis, a
derivative taken along the wrong axis, a source term's sign), builds the copy on
the CPU and runs the pin suite (the pins and the cross-operator reductions)
against it in a fresh process.  The pin suite must fail for every mutant.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "ns_neighbour_sign": ("gr[b][nb(g, iv, m, a, +1)] += gm * F[a][m] * i2h;",
                          "gr[b][nb(g, iv, m, a, +1)] -= gm * F[a][m] * i2h;"),
    "ns_local_term_wrong_field": ("gr[a][m] += gm * D1(g, cb, iv, m, a);",
                                  "gr[b][m] += gm * D1(g, cb, iv, m, a);"),
    "ns_advection_transposed": ("for (a = 0; a < d; a++) r += F[a][m] * D1(g, cb, iv, m, a);",
                                "for (a = 0; a < d; a++) r += F[b][m] * D1(g, F[a], iv, m, a);"),
    "loss_scale_all_nodes": ("x.dscale = 2.0 * dloss / (double)g.M;",
                             "x.dscale = 2.0 * dloss / (double)g.N;"),
    "burgers_viscous_1e-7": ("du[m] += gm * 2.0 * c->nu / (h1 * h1);",
                             "du[m] += gm * 2.0 * c->nu / (h1 * h1 * 1.0000001);"),
    "ns_dropped_pressure_term": ("dp[nb(g, iv, m, b, -1)] -= gm / (2.0 * g->h[b]);", ""),
    "heat_diffusion_sign": ("R[0] = (u[m] - C[0][m]) / c->dt - c->alpha * lap;",
                            "R[0] = (u[m] - C[0][m]) / c->dt + c->alpha * lap;"),
    "d1_spacing_axis0": ("/ (2.0 * g->h[a]);\n}\n\nstatic double D2",
                         "/ (2.0 * g->h[0]);\n}\n\nstatic double D2"),
    "ns_dropped_time_term": ("if (unsteady) gr[b][m] += gm / c->dt;", ""),
    "periodic_wrap_off_by_one": ("if (i >= g->n[a]) i -= g->n[a];",
                                 "if (i >= g->n[a]) i -= g->n[a] - 1;"),
    # the space-time NS operators (2D+t, 3D+t)
    "spacetime_time_adjoint_sign": ("gr[b][nb(g, iv, m, 0, +1)] += gm / (2.0 * g->h[0]);",
                                    "gr[b][nb(g, iv, m, 0, +1)] -= gm / (2.0 * g->h[0]);"),
    "spacetime_last_axis_dropped": ("for (a = 0; a < d; a++) R[d] += D1(g, F[a], iv, m, a + 1);",
                                    "for (a = 0; a + 1 < d; a++) R[d] += D1(g, F[a], iv, m, a + 1);"),
    "spacetime_advection_axis": ("for (a = 0; a < d; a++) r += F[a][m] * D1(g, cb, iv, m, a + 1);",
                                 "for (a = 0; a < d; a++) r += F[a][m] * D1(g, cb, iv, m, a);"),
    "poisson_source_sign": ("R[0] = lap - C[0][m];", "R[0] = lap + C[0][m];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(os.path.join(ROOT, "oracle", "fpde_oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    for sub in ("oracle", "tests", "paper_2607_18020_amd"):
        shutil.copytree(os.path.join(ROOT, sub), tmp_path / sub,
                        ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    csrc = tmp_path / "oracle" / "fpde_oracle.c"
    csrc.write_text(src.replace(old, new))
    subprocess.run(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o",
                    str(tmp_path / "oracle" / "libfpde_oracle.so"), str(csrc), "-lm"], check=True)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        str(tmp_path / "tests" / "test_oracle_pins.py"),
                        str(tmp_path / "tests" / "test_oracle_reductions.py"), "--rootdir", str(tmp_path)],
                       cwd=tmp_path, capture_output=True, text=True, timeout=300)
    assert r.returncode == 1, f"pins did not catch mutant {name}:\n{r.stdout[-2000:]}"
    assert "failed" in r.stdout
