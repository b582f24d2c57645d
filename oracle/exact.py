"""Exact (SVD-based) SLORR quantities, used only to pin the oracle.

  * nuclear norm n = sum(sigma), Frobenius norm f, polar factor U V^T over the
    nonzero singular values (Sec. 3, footnote on the generalised polar factor)
  * exact gradients of Eq. SLORR_grads (derived in App. A as the minimum-norm
    Clarke gradients)
  * Prop. 1: delta = |1 - l^2|^((q+1)^T) for degree d = 2q + 1, and the value
    and gradient bounds it implies
  * Prop. 2: the exact one-step singular value update (App. B)

LAPACK SVD through NumPy (gesdd) is the reference for these; they never serve
as a parity target for the GPU path.

This module is test infrastructure (see the package docstring).
"""
from __future__ import annotations

import numpy as np

__all__ = ["svd_parts", "exact_values", "exact_grad", "prop1_delta", "prop1_bounds"]


def svd_parts(W, rtol: float = 1e-13):
    """Thin SVD restricted to the nonzero singular values."""
    W = np.asarray(W, dtype=np.float64)
    U, s, Vt = np.linalg.svd(W, full_matrices=False)
    keep = s > rtol * (s[0] if s.size else 0.0)
    return U[:, keep], s[keep], Vt[keep, :]


def exact_values(W):
    """(n, f, ||W||_2, U V^T) for W != 0."""
    U, s, Vt = svd_parts(W)
    return float(np.sum(s)), float(np.sqrt(np.sum(s * s))), float(s[0]), U @ Vt


def exact_grad(W, kind: str):
    """Eq. SLORR_grads: Hoyer 2 (n/f) (UV^T / f - n/f^3 W); nuclear U V^T."""
    W = np.asarray(W, dtype=np.float64)
    n, f, _, UV = exact_values(W)
    if kind == "nuclear":
        return UV
    return 2.0 * (n / f) * (UV / f - (n / f ** 3) * W)


def prop1_delta(ell: float, T: int, d: int = 5) -> float:
    """delta = |1 - l^2|^((q+1)^T), d = 2q + 1 (Prop. 1)."""
    q = (d - 1) // 2
    return float(abs(1.0 - ell * ell) ** ((q + 1) ** T))


def prop1_bounds(W, ell: float, T: int, d: int = 5):
    """Right-hand sides of Prop. 1 for matrix W:
    (polar spectral-norm error, relative nuclear error, relative Hoyer-value
     error, Hoyer-gradient spectral-norm error)."""
    n, f, s1, _ = exact_values(W)
    delta = prop1_delta(ell, T, d)
    return (delta, delta, delta * (2.0 + delta),
            2.0 * delta * (2.0 + delta) * (n / f ** 2 + n ** 2 / f ** 4 * s1))
