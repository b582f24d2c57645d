"""SLORR regularizer forward + backward, oracle side (float64, NumPy).

Follows Sec. 3 of the paper step by step, for one weight matrix W (M x N,
widened exactly from its storage type to float64):

  O1  f = ||W||_F = sqrt(sum W_ij^2),  f_eps = f + eps
          (Sec. 3 "Computing the nuclear and Frobenius norms"; Listing 1 adds
           eps to the norm)
  O2  Y = W^T if M > N else W: the Gram products are formed on the short side,
          which is the orientation behind the cost 4 P^2 Q + 2 P^3 with
          P = min(M, N), Q = max(M, N) (Sec. 3 "Computational cost")
  O3  X_0 = Y / f_eps           (Sec. 3 "Computing the polar factor": divide
                                 by the Frobenius norm plus eps)
  O4  for t = 1..T:             (Polar Express, odd polynomial of degree 5,
        A = X X^T                App. E.1)
        B = b_t A + c_t A A
        X = a_t X + B X         i.e. X <- p_t(X) = a_t X + b_t (XX^T)X
                                                 + c_t (XX^T)^2 X
  O5  P = X_T, transposed back when M > N: the approximate polar factor U V^T
  O6  n = sum(W * P)            (Sec. 3: sum(W . UV^T) = tr(Sigma) = ||W||_*)
  O7  Hoyer:   L = (n / f_eps)^2; Eq. SLORR_grads, d(||W||_*^2 / ||W||_F^2)/dW
               = (2 n / f^2) U V^T - (2 n^2 / f^4) W, with U V^T -> P and
               f -> f_eps (the substitution Listing 1 makes):
                 grad = g * (s1 * P - s2 * W),  s1 = 2 n / f_eps^2,
                                                s2 = 2 n^2 / f_eps^4
               (no differentiation through O4, Sec. 3)
      Nuclear: L = n,  grad = g * P      (Eq. SLORR_grads, right part)
  O8  set value = sum_i L_i     (Sec. 3, definition of L_hoyer and L_nuc)

g is the upstream scale (the loss weight lambda times the upstream gradient;
App. E.3 accumulates lambda * G into W.grad).

Reading (paper silent): a matrix with f_eps == 0 (only possible when W = 0 and
eps = 0) gives L = 0 and grad = 0, the limit along eps -> 0+.

This module is test infrastructure (see the package docstring).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

__all__ = ["OracleResult", "fwd_bwd", "fwd_bwd_set", "polar_iterate", "HOYER", "NUCLEAR"]

HOYER = "hoyer"
NUCLEAR = "nuclear"


@dataclass
class OracleResult:
    value: float        # L (squared Hoyer ratio, or nuclear-norm estimate)
    n_hat: float        # trace estimate of ||W||_*
    f: float            # ||W||_F
    f_eps: float        # ||W||_F + eps
    ratio: float        # n_hat / f_eps (Hoyer); n_hat (nuclear)
    polar: np.ndarray   # P, same shape as W
    grad: np.ndarray    # dL/dW times g, same shape as W


def polar_iterate(X0: np.ndarray, table: np.ndarray) -> np.ndarray:
    """O4: T steps X <- a X + (b A + c A A) X with A = X X^T."""
    X = np.array(X0, dtype=np.float64, copy=True)
    for a, b, c in np.asarray(table, dtype=np.float64):
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X


def fwd_bwd(W, kind: str, table, eps: float = 0.0, g: float = 1.0) -> OracleResult:
    """Approximate value and gradient of one matrix (steps O1-O7)."""
    W = np.asarray(W, dtype=np.float64)
    if W.ndim != 2:
        raise ValueError("W must be 2-D (reshape conv kernels to (C_out, -1))")
    if kind not in (HOYER, NUCLEAR):
        raise ValueError(f"unknown kind {kind!r}")
    M, N = W.shape
    f = float(np.sqrt(np.sum(W * W)))                     # O1
    f_eps = f + float(eps)
    if M == 0 or N == 0 or f_eps == 0.0:
        z = np.zeros_like(W)
        return OracleResult(0.0, 0.0, f, f_eps, 0.0, z, z.copy())
    tall = M > N                                          # O2
    Y = W.T if tall else W
    X = polar_iterate(Y / f_eps, table)                   # O3, O4
    P = X.T if tall else X                                # O5
    n_hat = float(np.sum(W * P))                          # O6
    if kind == HOYER:                                     # O7
        r = n_hat / f_eps
        value = r * r
        s1 = 2.0 * n_hat / f_eps ** 2
        s2 = 2.0 * n_hat ** 2 / f_eps ** 4
        grad = g * (s1 * P - s2 * W)
    else:
        r = n_hat
        value = n_hat
        grad = g * P
    return OracleResult(value, n_hat, f, f_eps, r, P, grad)


def fwd_bwd_set(Ws, kind: str, table, eps: float = 0.0, g: float = 1.0):
    """O8: per-matrix results and the set total (sum in index order)."""
    res = [fwd_bwd(W, kind, table, eps, g) for W in Ws]
    total = 0.0
    for r in res:
        total += r.value
    return res, total
