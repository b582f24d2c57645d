"""MI355X-native SLORR regularizer hot path.

SLORR-Hoyer (||W||_*^2 / ||W||_F^2) and SLORR-Nuc (||W||_*) forward and
backward over a whole weight set, computed SVD-free with Polar Express
(Sec. 3 of the paper) in hand-written HIP kernels for gfx950 behind the C ABI
of include/slorr.h. This package holds the ctypes binding (`Plan`,
`pe_coefficients`), the PyTorch integration (`Regularizer`, `SlorrFunction`,
`DecoupledSlorr`: Listing 1, App. E.2 and E.3) and the build script; the
library is libslorr.so next to this file.
"""
from .slorr import HOYER, NUCLEAR, Plan, SlorrError, pe_coefficients

__all__ = ["Plan", "pe_coefficients", "SlorrError", "HOYER", "NUCLEAR",
           "Regularizer", "SlorrFunction", "DecoupledSlorr"]


def __getattr__(name):
    # the torch integration is imported on first use (the binding itself
    # needs torch only when a plan is given a workspace)
    if name in ("Regularizer", "SlorrFunction", "DecoupledSlorr"):
        from . import integration
        return getattr(integration, name)
    raise AttributeError(name)
