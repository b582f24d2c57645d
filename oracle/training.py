"""Training-loop uses of the SLORR gradient, oracle side (float64, NumPy).

  autograd_grads   Listing 1 used as a loss term: for loss = sum_i c_i L_i the
                   gradient of W_i is c_i G_i, with G_i the approximate
                   gradient of Eq. SLORR_grads (steps O1-O7 of oracle.slorr)
  alg2_accumulate  App. E.3, the memory-efficient loop: for every regularized
                   W, W.grad <- W.grad + lambda G(W), or lambda G(W) when W has
                   no gradient yet
  adamw_step       AdamW, Adam with decoupled weight decay (Loshchilov and
                   Hutter), without amsgrad:
                     W <- W (1 - eta wd)
                     m <- beta1 m + (1 - beta1) g,  v <- beta2 v + (1 - beta2) g^2
                     W <- W - eta (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
  decoupled_step   App. E.2, Alg. 1 (SLORR-Hoyer-D): G_pre from the weights
                   before the update, the AdamW step with the task gradient
                   (skipped when there is none), then W <- W - eta lambda G_pre

Reading (Alg. 1 names one learning rate): eta in the decoupled term is the
learning rate of the same optimizer step.

This module is test infrastructure (see the package docstring).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from .slorr import fwd_bwd

__all__ = ["autograd_grads", "alg2_accumulate", "AdamWState", "adamw_step", "decoupled_step"]


def autograd_grads(Ws: Sequence[np.ndarray], upstream: Sequence[float], kind: str, table,
                   eps: float = 0.0) -> List[np.ndarray]:
    """Gradients of sum_i upstream[i] L_i (Listing 1's backward: the
    incoming gradient times the rule of Eq. SLORR_grads)."""
    return [fwd_bwd(W, kind, table, eps, g=float(c)).grad for W, c in zip(Ws, upstream)]


def alg2_accumulate(Ws: Sequence[np.ndarray], grads: Sequence[Optional[np.ndarray]], lam: float,
                    kind: str, table, eps: float = 0.0) -> List[np.ndarray]:
    """App. E.3: the new gradient of each W after the regularizer's pass."""
    out = []
    for W, g in zip(Ws, grads):
        G = fwd_bwd(W, kind, table, eps, g=1.0).grad
        out.append(lam * G if g is None else np.asarray(g, dtype=np.float64) + lam * G)
    return out


@dataclass
class AdamWState:
    m: np.ndarray
    v: np.ndarray
    t: int = 0

    @staticmethod
    def zeros_like(W):
        W = np.asarray(W, dtype=np.float64)
        return AdamWState(np.zeros_like(W), np.zeros_like(W), 0)


def adamw_step(W, g, state: AdamWState, lr: float, betas=(0.9, 0.999), eps: float = 1e-8,
               weight_decay: float = 1e-2) -> np.ndarray:
    """One AdamW step; returns the new W and updates `state` in place."""
    W = np.asarray(W, dtype=np.float64)
    g = np.asarray(g, dtype=np.float64)
    b1, b2 = betas
    state.t += 1
    W = W * (1.0 - lr * weight_decay)
    state.m = b1 * state.m + (1.0 - b1) * g
    state.v = b2 * state.v + (1.0 - b2) * g * g
    m_hat = state.m / (1.0 - b1 ** state.t)
    v_hat = state.v / (1.0 - b2 ** state.t)
    return W - lr * m_hat / (np.sqrt(v_hat) + eps)


def decoupled_step(Ws: Sequence[np.ndarray], task_grads: Sequence[Optional[np.ndarray]],
                   states: Sequence[AdamWState], lr: float, lam: float, kind: str, table,
                   reg_eps: float = 0.0, betas=(0.9, 0.999), adam_eps: float = 1e-8,
                   weight_decay: float = 1e-2):
    """Alg. 1 over a regularized set. Returns (new weights, G_pre per matrix)."""
    new_W, G_pre = [], []
    for W, g, st in zip(Ws, task_grads, states):
        W = np.asarray(W, dtype=np.float64)
        G = fwd_bwd(W, kind, table, reg_eps, g=1.0).grad        # from the pre-update W
        if g is not None:
            W = adamw_step(W, g, st, lr, betas, adam_eps, weight_decay)
        new_W.append(W - lr * lam * G)
        G_pre.append(G)
    return new_W, G_pre
