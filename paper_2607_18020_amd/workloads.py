"""Seeded synthetic workloads for the FD residual operators.

This module holds the operator registry (op ids, field/const names, grid
spacings, PDE coefficients) and the seeded input generators.  It contains none
of the residual or adjoint arithmetic: only sums of Fourier modes and Gaussian
noise that stand in for the grid-aligned network outputs the operator consumes
(the paper feeds the operator with fields produced by a neural field generator,
Sec. 2 intro; its trained fields are not available, so seeded fields of the same
shape and smoothness are used instead).

Every generator is a pure function of (config, seed, shape): it draws all of its
random numbers from ``numpy.random.default_rng(seed)``, evaluates the fields in
float64 and rounds them once to float32.  The float32 arrays are the canonical
inputs; the CPU oracle receives them widened exactly to float64.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Operator ids shared by the C ABI and the oracle (numbers only).
BURGERS_1DT = 1
HELMHOLTZ_2D = 2
HEAT_3D_BE = 3
NS_2D_STEADY = 4
NS_3D_BE = 5
NS_3D_STEADY = 6
POISSON_2D = 7
POISSON_3D = 8
NS_2DT = 9
NS_3DT = 10

OP_NAMES = {
    BURGERS_1DT: "burgers_1dt",
    HELMHOLTZ_2D: "helmholtz_2d",
    HEAT_3D_BE: "heat_3d_be",
    NS_2D_STEADY: "ns_2d_steady",
    NS_3D_BE: "ns_3d_be",
    NS_3D_STEADY: "ns_3d_steady",
    POISSON_2D: "poisson_2d",
    POISSON_3D: "poisson_3d",
    NS_2DT: "ns_2dt",
    NS_3DT: "ns_3dt",
}


@dataclasses.dataclass(frozen=True)
class OpSpec:
    """Static description of one operator: which arrays it reads and writes."""

    op: int
    ndim: int
    fields: Tuple[str, ...]      # differentiated inputs, in ABI order
    consts: Tuple[str, ...]      # non-differentiated inputs, in ABI order
    residuals: Tuple[str, ...]   # residual equations, in ABI order


OPS: Dict[int, OpSpec] = {
    BURGERS_1DT: OpSpec(BURGERS_1DT, 2, ("u",), (), ("R",)),
    HELMHOLTZ_2D: OpSpec(HELMHOLTZ_2D, 2, ("u",), ("f",), ("R",)),
    HEAT_3D_BE: OpSpec(HEAT_3D_BE, 3, ("u",), ("u0",), ("R",)),
    NS_2D_STEADY: OpSpec(NS_2D_STEADY, 2, ("u", "v", "p"), (), ("R_u", "R_v", "R_c")),
    NS_3D_BE: OpSpec(NS_3D_BE, 3, ("u", "v", "w", "p"), ("u_prev", "v_prev", "w_prev"),
                     ("R_u", "R_v", "R_w", "R_c")),
    NS_3D_STEADY: OpSpec(NS_3D_STEADY, 3, ("u", "v", "w", "p"), (), ("R_u", "R_v", "R_w", "R_c")),
    POISSON_2D: OpSpec(POISSON_2D, 2, ("u",), ("f",), ("R",)),
    POISSON_3D: OpSpec(POISSON_3D, 3, ("u",), ("f",), ("R",)),
    # space-time grid (t, x, y): velocity component b on array axis b + 1
    NS_2DT: OpSpec(NS_2DT, 3, ("u", "v", "p"), (), ("R_u", "R_v", "R_c")),
    # space-time grid (t, x, y, z): velocity component b on array axis b + 1
    NS_3DT: OpSpec(NS_3DT, 4, ("u", "v", "w", "p"), (), ("R_u", "R_v", "R_w", "R_c")),
}

# the operators of the five benchmark workloads; the others are the adjacent
# operators that share their kernels
CORE_OPS = (BURGERS_1DT, HELMHOLTZ_2D, HEAT_3D_BE, NS_2D_STEADY, NS_3D_BE)


@dataclasses.dataclass(frozen=True)
class Coeffs:
    """PDE coefficients; an operator ignores the members it does not use."""

    nu: float = 0.0
    k: float = 0.0
    dt: float = 1.0
    alpha: float = 0.0


@dataclasses.dataclass
class Workload:
    """One concrete operator instance: arrays plus everything the ABI needs."""

    name: str
    op: int
    shape: Tuple[int, ...]
    h: Tuple[float, ...]
    coeffs: Coeffs
    fields: List[np.ndarray]   # float32, C-contiguous
    consts: List[np.ndarray]   # float32, C-contiguous

    @property
    def spec(self) -> OpSpec:
        return OPS[self.op]

    @property
    def n_points(self) -> int:
        return int(np.prod(self.shape))

    @property
    def n_residual_points(self) -> int:
        return int(np.prod([s - 2 for s in self.shape]))


@dataclasses.dataclass(frozen=True)
class Config:
    """A named workload: operator, full-size grid, domain and coefficients."""

    name: str
    op: int
    shape: Tuple[int, ...]
    coeffs: Coeffs
    description: str


# The five workloads: 1D+t Burgers, 2D Helmholtz, one implicit 3D heat step,
# 2D steady incompressible NS (the paper's worked ldc_2d example, Sec. 2.1) and
# one backward-Euler step of 3D Taylor-Green NS.
CONFIGS: Dict[str, Config] = {
    "burgers_1dt": Config("burgers_1dt", BURGERS_1DT, (128, 256),
                          Coeffs(nu=0.01 / math.pi),
                          "1D viscous Burgers, space-time grid nt=128 x nx=256, t in [0,1], x in [-1,1]"),
    "helmholtz_2d": Config("helmholtz_2d", HELMHOLTZ_2D, (1024, 1024),
                           Coeffs(k=4.0 * math.pi),
                           "2D Helmholtz 1024^2 on [0,1]^2, k=4pi, 5-point Laplacian"),
    "heat_3d": Config("heat_3d", HEAT_3D_BE, (256, 256, 256),
                      Coeffs(dt=1e-3, alpha=0.1),
                      "3D heat, one implicit step, 256^3 on [0,1]^3, dt=1e-3, alpha=0.1"),
    "ns_2d": Config("ns_2d", NS_2D_STEADY, (2048, 2048),
                    Coeffs(nu=0.01),
                    "2D steady incompressible NS (u,v,p), 2048^2 on [0,1]^2, nu=0.01"),
    "ns_3d_tgv": Config("ns_3d_tgv", NS_3D_BE, (256, 256, 256),
                        Coeffs(nu=0.01, dt=1e-2),
                        "3D Taylor-Green NS (u,v,w,p), one backward-Euler step, 256^3 on [0,2pi)^3, nu=0.01, dt=1e-2"),
    # adjacent operators (same kernels, other point functions)
    "ns_3d_steady": Config("ns_3d_steady", NS_3D_STEADY, (256, 256, 256), Coeffs(nu=0.01),
                           "3D steady incompressible NS (u,v,w,p), 256^3 on [0,1]^3, nu=0.01"),
    "poisson_2d": Config("poisson_2d", POISSON_2D, (1024, 1024), Coeffs(),
                         "2D Poisson 1024^2 on [0,1]^2, 5-point Laplacian"),
    "poisson_3d": Config("poisson_3d", POISSON_3D, (256, 256, 256), Coeffs(),
                         "3D Poisson 256^3 on [0,1]^3, 7-point Laplacian"),
    "ns_2dt": Config("ns_2dt", NS_2DT, (64, 512, 512), Coeffs(nu=0.01),
                     "2D+t unsteady incompressible NS (u,v,p) on a space-time grid 64 x 512^2, "
                     "t in [0,1], (x,y) on [0,2pi)^2, nu=0.01, central time differences"),
    # the paper's 3D Taylor-Green operator on its space-time grid (32^3 x 10 points),
    # and on ~42M space-time points, the largest grid of its kernel-scaling study
    "ns_3dt": Config("ns_3dt", NS_3DT, (10, 32, 32, 32), Coeffs(nu=0.01),
                     "3D+t unsteady incompressible NS (u,v,w,p) on a space-time grid 10 x 32^3, "
                     "t in [0,1], (x,y,z) on [0,2pi)^3, nu=0.01, central time differences"),
    "ns_3dt_large": Config("ns_3dt_large", NS_3DT, (20, 128, 128, 128), Coeffs(nu=0.01),
                           "3D+t unsteady incompressible NS (u,v,w,p) on a space-time grid "
                           "20 x 128^3 (41.9M points), t in [0,1], (x,y,z) on [0,2pi)^3, "
                           "nu=0.01, central time differences"),
}

CONFIG_ORDER = ("burgers_1dt", "helmholtz_2d", "heat_3d", "ns_2d", "ns_3d_tgv")
ADJACENT_CONFIGS = ("ns_3d_steady", "poisson_2d", "poisson_3d", "ns_2dt", "ns_3dt",
                    "ns_3dt_large")


def spacing(cfg_name: str, shape: Sequence[int]) -> Tuple[float, ...]:
    """Grid spacing per array axis for a config at a given shape.

    Burgers: axis 0 is t on [0,1], axis 1 is x on [-1,1], endpoint-inclusive.
    Helmholtz, heat, 2D NS, 3D steady NS, Poisson: endpoint-inclusive nodes on
    [0,1] per axis.
    3D TGV: periodic sampling x_i = 2*pi*i/n on [0,2pi).
    2D+t and 3D+t NS: axis 0 is t on [0,1] endpoint-inclusive; the spatial
    axes periodic on [0,2pi).
    """
    if cfg_name == "burgers_1dt":
        return (1.0 / (shape[0] - 1), 2.0 / (shape[1] - 1))
    if cfg_name in ("helmholtz_2d", "heat_3d", "ns_2d", "ns_3d_steady", "poisson_2d",
                    "poisson_3d"):
        return tuple(1.0 / (s - 1) for s in shape)
    if cfg_name == "ns_3d_tgv":
        return tuple(2.0 * math.pi / s for s in shape)
    if cfg_name in ("ns_2dt", "ns_3dt", "ns_3dt_large"):
        return (1.0 / (shape[0] - 1),) + tuple(2.0 * math.pi / s for s in shape[1:])
    raise KeyError(cfg_name)


def _axes(cfg_name: str, shape: Sequence[int]) -> List[np.ndarray]:
    """1-D node coordinates per axis (float64)."""
    h = spacing(cfg_name, shape)
    if cfg_name == "burgers_1dt":
        return [np.arange(shape[0]) * h[0], -1.0 + np.arange(shape[1]) * h[1]]
    return [np.arange(s) * hh for s, hh in zip(shape, h)]


def _mesh(coords: List[np.ndarray]) -> List[np.ndarray]:
    return np.meshgrid(*coords, indexing="ij", sparse=True)


def _fourier_sum(rng, X, n_modes, kmax, trig_choice=False):
    """sum over modes of (a/|kappa|) * trig(2 pi kappa.x + phi), kappa in {1..kmax}^d."""
    d = len(X)
    out = np.zeros(np.broadcast_shapes(*[x.shape for x in X]), dtype=np.float64)
    for _ in range(n_modes):
        kap = rng.integers(1, kmax + 1, size=d)
        a = rng.standard_normal()
        phi = rng.uniform(0.0, 2.0 * math.pi)
        use_cos = bool(rng.integers(0, 2)) if trig_choice else False
        arg = sum(2.0 * math.pi * float(kap[i]) * X[i] for i in range(d)) + phi
        out += (a / float(np.linalg.norm(kap))) * (np.cos(arg) if use_cos else np.sin(arg))
    return out


def _f32(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def make(cfg_name: str, seed: int = 42, shape: Optional[Sequence[int]] = None) -> Workload:
    """Seeded synthetic inputs for one config (full size unless ``shape`` is given)."""
    cfg = CONFIGS[cfg_name]
    shape = tuple(int(s) for s in (shape if shape is not None else cfg.shape))
    if len(shape) != OPS[cfg.op].ndim:
        raise ValueError(f"{cfg_name}: shape {shape} has wrong rank")
    rng = np.random.default_rng(seed)
    X = _mesh(_axes(cfg_name, shape))
    h = spacing(cfg_name, shape)
    noise = lambda: 0.01 * rng.standard_normal(shape)  # N(0, 0.01^2): std 0.01

    if cfg_name == "burgers_1dt":
        t, x = X
        u = np.zeros(shape)
        for k in range(1, 9):
            a = rng.standard_normal()
            phi, psi = rng.uniform(0.0, 2.0 * math.pi, size=2)
            m = int(rng.integers(0, 4))
            u = u + (a / k) * np.sin(math.pi * k * x + phi) * np.cos(math.pi * m * t + psi)
        u = u + noise()
        fields, consts = [_f32(u)], []
    elif cfg_name == "helmholtz_2d":
        u = _fourier_sum(rng, X, 16, 8, trig_choice=True) + noise()
        f = _fourier_sum(rng, X, 16, 8, trig_choice=True) + noise()
        fields, consts = [_f32(u)], [_f32(f)]
    elif cfg_name == "heat_3d":
        u0 = _fourier_sum(rng, X, 8, 4)
        u = u0 + noise()
        fields, consts = [_f32(u)], [_f32(u0)]
    elif cfg_name == "ns_2d":
        # streamfunction psi = sum (a/|kappa|) sin(2 pi kappa.x + phi);
        # u = d psi / d y (array axis 1), v = -d psi / d x (array axis 0), analytically.
        x, y = X
        u = np.zeros(shape)
        v = np.zeros(shape)
        for _ in range(16):
            kap = rng.integers(1, 9, size=2)
            a = rng.standard_normal()
            phi = rng.uniform(0.0, 2.0 * math.pi)
            amp = a / float(np.linalg.norm(kap))
            c = np.cos(2.0 * math.pi * (kap[0] * x + kap[1] * y) + phi)
            u = u + amp * 2.0 * math.pi * kap[1] * c
            v = v - amp * 2.0 * math.pi * kap[0] * c
        p = np.zeros(shape)
        for _ in range(8):
            kap = rng.integers(1, 9, size=2)
            b = rng.standard_normal()
            phi = rng.uniform(0.0, 2.0 * math.pi)
            p = p + b * np.sin(2.0 * math.pi * (kap[0] * x + kap[1] * y) + phi)
        fields, consts = [_f32(u), _f32(v), _f32(p)], []
    elif cfg_name == "ns_3d_tgv":
        x, y, z = X
        u_ic = np.sin(x) * np.cos(y) * np.cos(z)
        v_ic = -np.cos(x) * np.sin(y) * np.cos(z)
        w_ic = np.zeros(shape)
        p_ic = (np.cos(2.0 * x) + np.cos(2.0 * y)) * (np.cos(2.0 * z) + 2.0) / 16.0
        u_ic = np.broadcast_to(u_ic, shape)
        v_ic = np.broadcast_to(v_ic, shape)
        p_ic = np.broadcast_to(p_ic, shape)
        fields = [_f32(u_ic + noise()), _f32(v_ic + noise()), _f32(w_ic + noise()),
                  _f32(p_ic + noise())]
        consts = [_f32(u_ic), _f32(v_ic), _f32(w_ic)]
    elif cfg_name == "ns_3d_steady":
        # velocity = curl of a vector potential A (three sums of 6 modes of
        # amplitude a / (2 pi |kappa|)), so it is divergence-free analytically;
        # p = 8 modes; + N(0, 0.01^2) on every field
        def modes(n):
            out = []
            for _ in range(n):
                kap = rng.integers(1, 5, size=3)
                out.append((kap, rng.standard_normal() / float(np.linalg.norm(kap)),
                            rng.uniform(0.0, 2.0 * math.pi)))
            return out
        dA = [[np.zeros(shape) for _ in range(3)] for _ in range(3)]  # dA[i][j] = dA_i/dx_j
        for i in range(3):
            for kap, amp, phi in modes(6):
                c = np.cos(2.0 * math.pi * sum(float(kap[j]) * X[j] for j in range(3)) + phi)
                for j in range(3):
                    dA[i][j] = dA[i][j] + amp * float(kap[j]) * c
        u = dA[2][1] - dA[1][2]
        v = dA[0][2] - dA[2][0]
        w = dA[1][0] - dA[0][1]
        p = np.zeros(shape)
        for kap, amp, phi in modes(8):
            p = p + amp * np.sin(2.0 * math.pi * sum(float(kap[j]) * X[j] for j in range(3)) + phi)
        fields = [_f32(np.broadcast_to(q, shape) + noise()) for q in (u, v, w, p)]
        consts = []
    elif cfg_name in ("poisson_2d", "poisson_3d"):
        nm, km = (16, 8) if len(shape) == 2 else (8, 4)
        u = _fourier_sum(rng, X, nm, km, trig_choice=True) + noise()
        f = _fourier_sum(rng, X, nm, km, trig_choice=True) + noise()
        fields, consts = [_f32(u)], [_f32(f)]
    elif cfg_name == "ns_2dt":
        # decaying 2D Taylor-Green vortex (an exact NS solution) + N(0, 0.01^2)
        t, x, y = X
        nu = cfg.coeffs.nu
        e1, e2 = np.exp(-2.0 * nu * t), np.exp(-4.0 * nu * t)
        u = np.sin(x) * np.cos(y) * e1
        v = -np.cos(x) * np.sin(y) * e1
        p = 0.25 * (np.cos(2.0 * x) + np.cos(2.0 * y)) * e2
        fields = [_f32(np.broadcast_to(q, shape) + noise()) for q in (u, v, p)]
        consts = []
    elif cfg_name in ("ns_3dt", "ns_3dt_large"):
        # the 3D Taylor-Green vortex (the initial condition of the TGV workload)
        # decaying in time at the viscous rates of its velocity (3 nu) and
        # pressure (6 nu) modes, + N(0, 0.01^2) on every field
        t, x, y, z = X
        nu = cfg.coeffs.nu
        e1, e2 = np.exp(-3.0 * nu * t), np.exp(-6.0 * nu * t)
        u = np.sin(x) * np.cos(y) * np.cos(z) * e1
        v = -np.cos(x) * np.sin(y) * np.cos(z) * e1
        w = np.zeros(shape)
        p = (np.cos(2.0 * x) + np.cos(2.0 * y)) * (np.cos(2.0 * z) + 2.0) / 16.0 * e2
        fields = []
        for q in (u, v, w, p):  # (one at a time: the large grid is 168 MB per array)
            fields.append(_f32(np.broadcast_to(q, shape) + noise()))
        consts = []
    else:  # pragma: no cover
        raise KeyError(cfg_name)

    return Workload(cfg_name, cfg.op, shape, h, cfg.coeffs, fields, consts)


def normal_fields(op: int, shape: Sequence[int], seed: int,
                  h: Optional[Sequence[float]] = None,
                  coeffs: Optional[Coeffs] = None) -> Workload:
    """Standard-normal fields for every input (the paper's verification inputs,
    App. A.7: N(0,1) samples, seeds 42-46)."""
    spec = OPS[op]
    shape = tuple(int(s) for s in shape)
    rng = np.random.default_rng(seed)
    fields = [_f32(rng.standard_normal(shape)) for _ in spec.fields]
    consts = [_f32(rng.standard_normal(shape)) for _ in spec.consts]
    if h is None:
        h = tuple(1.0 / (s - 1) for s in shape)
    if coeffs is None:
        coeffs = {BURGERS_1DT: Coeffs(nu=0.01 / math.pi), HELMHOLTZ_2D: Coeffs(k=4 * math.pi),
                  HEAT_3D_BE: Coeffs(dt=1e-3, alpha=0.1), NS_2D_STEADY: Coeffs(nu=0.01),
                  NS_3D_BE: Coeffs(nu=0.01, dt=1e-2), NS_3D_STEADY: Coeffs(nu=0.01),
                  POISSON_2D: Coeffs(), POISSON_3D: Coeffs(), NS_2DT: Coeffs(nu=0.01),
                  NS_3DT: Coeffs(nu=0.01)}[op]
    return Workload(f"normal_{OP_NAMES[op]}", op, shape, tuple(float(x) for x in h), coeffs,
                    fields, consts)


def normal_fields_f32(op: int, shape: Sequence[int], seed: int,
                      h: Optional[Sequence[float]] = None,
                      coeffs: Optional[Coeffs] = None) -> Workload:
    """Standard-normal inputs drawn directly in float32 (a seeded stream of its
    own, distinct from normal_fields): for grids of billions of nodes, where
    drawing in float64 first would double the host memory and time."""
    wl = normal_fields(op, (3,) * OPS[op].ndim, seed, None, coeffs)  # coefficients only
    shape = tuple(int(s) for s in shape)
    rng = np.random.default_rng(seed)
    spec = OPS[op]
    fields = [rng.standard_normal(shape, dtype=np.float32) for _ in spec.fields]
    consts = [rng.standard_normal(shape, dtype=np.float32) for _ in spec.consts]
    if h is None:
        h = tuple(1.0 / (s - 1) for s in shape)
    return Workload(f"normal32_{OP_NAMES[op]}", op, shape, tuple(float(x) for x in h),
                    wl.coeffs if coeffs is None else coeffs, fields, consts)


@dataclasses.dataclass
class TiledWorkload:
    """A workload too large to draw value by value (billions of nodes): each
    array (fields, then consts) repeats one seeded draw of `period` standard
    normal float32 values in memory order.  The period is a prime, so no row,
    plane or time level holds its neighbour's values.  `window` rebuilds any
    sub-box of the arrays on the host from the draws; the arrays themselves
    are never built on the host."""

    name: str
    op: int
    shape: Tuple[int, ...]
    h: Tuple[float, ...]
    coeffs: Coeffs
    vectors: List[np.ndarray]  # float32, one draw per array

    @property
    def spec(self) -> OpSpec:
        return OPS[self.op]

    @property
    def n_points(self) -> int:
        return int(np.prod(self.shape))

    @property
    def n_residual_points(self) -> int:
        return int(np.prod([s - 2 for s in self.shape]))

    def window(self, box) -> Tuple[List[np.ndarray], List[np.ndarray]]:
        """(fields, consts) on the sub-box `box` (a tuple of slices)."""
        axes = [np.arange(*sl.indices(n)) for sl, n in zip(box, self.shape)]
        lin = np.ravel_multi_index(np.meshgrid(*axes, indexing="ij"), self.shape)
        arrays = [np.ascontiguousarray(v[lin % v.size]) for v in self.vectors]
        nf = len(self.spec.fields)
        return arrays[:nf], arrays[nf:]


def normal_tiled_f32(op: int, shape: Sequence[int], seed: int,
                     h: Optional[Sequence[float]] = None,
                     coeffs: Optional[Coeffs] = None, period: int = 1_000_003) -> TiledWorkload:
    """Standard-normal float32 inputs repeated with a prime period (TiledWorkload)."""
    wl = normal_fields(op, (3,) * OPS[op].ndim, seed, None, coeffs)  # coefficients only
    shape = tuple(int(s) for s in shape)
    rng = np.random.default_rng(seed)
    spec = OPS[op]
    vectors = [rng.standard_normal(period, dtype=np.float32) for _ in spec.fields + spec.consts]
    if h is None:
        h = tuple(1.0 / (s - 1) for s in shape)
    return TiledWorkload(f"tiled32_{OP_NAMES[op]}", op, shape, tuple(float(x) for x in h),
                         wl.coeffs if coeffs is None else coeffs, vectors)


def sensitivities(op: int, shape: Sequence[int], seed: int) -> List[np.ndarray]:
    """Upstream residual sensitivities G_b (one standard-normal float32 array
    per residual, full size) for the explicit-sensitivity backward."""
    rng = np.random.default_rng(seed)
    return [_f32(rng.standard_normal(tuple(int(s) for s in shape)))
            for _ in OPS[op].residuals]
