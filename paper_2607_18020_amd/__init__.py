"""MI355X (gfx950) differentiable finite-difference PDE residual operator.

Three C-ABI entry points (include/fpde.h), implemented as hand-written HIP
kernels in ``csrc/`` and exposed here through a thin ctypes binding:
``fpde_residual_fwd`` (fused stencil + mean-squared loss),
``fpde_residual_bwd`` (interior analytic adjoint, gather form) and
``fpde_bc_correct`` (boundary-gradient correction).  ``workloads`` holds the
seeded synthetic inputs of the five benchmark operators.
"""
from . import workloads  # noqa: F401

__all__ = ["workloads", "binding"]


def __getattr__(name):
    # the binding loads libfpde.so; import it lazily so that the workload
    # generators stay usable on machines without the built library
    if name == "binding":
        import importlib  # noqa: PLC0415
        return importlib.import_module(".binding", __name__)
    raise AttributeError(name)
