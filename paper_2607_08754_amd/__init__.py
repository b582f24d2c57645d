"""MI355X-native SLORR regularizer hot path.

SLORR-Hoyer (||W||_*^2 / ||W||_F^2) and SLORR-Nuc (||W||_*) forward and
backward over a whole weight set, computed SVD-free with Polar Express
(Sec. 3 of the paper) in hand-written HIP kernels for gfx950 behind the C ABI
of include/slorr.h. This package holds the ctypes binding (`Plan`,
`pe_coefficients`) and the build script; the library is libslorr.so next to
this file.
"""
from .slorr import HOYER, NUCLEAR, Plan, SlorrError, pe_coefficients

__all__ = ["Plan", "pe_coefficients", "SlorrError", "HOYER", "NUCLEAR"]
