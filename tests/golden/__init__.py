"""Reader for the hand-worked golden fixtures in this folder.

Each ``*.txt`` file is a tiny operator instance whose residuals, loss and
gradient were worked out by hand from the residual definitions (the derivation
is in the file's comment header).  Format, one record per line:
``op <id>``, ``shape <n...>``, ``h <h...>``, ``coeffs nu=.. k=.. dt=.. alpha=..``,
``field <name> <values...>``, ``const <name> <values...>``,
``residual <name> <values...>``, ``loss <value>``, ``grad <name> <values...>``.
Values are listed in C order (last axis fastest).
"""
from __future__ import annotations

import glob
import os
import types

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def load(path: str):
    rec = types.SimpleNamespace(fields=[], consts=[], residuals=[], grads=[], loss=None)
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, *rest = line.split()
        if key == "op":
            rec.op = int(rest[0])
        elif key == "shape":
            rec.shape = tuple(int(x) for x in rest)
        elif key == "h":
            rec.h = tuple(float(x) for x in rest)
        elif key == "coeffs":
            kv = dict(x.split("=") for x in rest)
            rec.coeffs = types.SimpleNamespace(**{k: float(v) for k, v in kv.items()})
        elif key in ("field", "const", "residual", "grad"):
            arr = np.array([float(x) for x in rest[1:]], dtype=np.float64).reshape(rec.shape)
            {"field": rec.fields, "const": rec.consts, "residual": rec.residuals,
             "grad": rec.grads}[key].append(arr)
        elif key == "loss":
            rec.loss = float(rest[0])
        else:
            raise ValueError(f"{path}: unknown record {key}")
    rec.name = os.path.basename(path)
    return rec


def all_fixtures():
    return sorted(glob.glob(os.path.join(HERE, "*.txt")))
