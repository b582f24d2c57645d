"""Pins for the oracle's training-loop integrations (float64, CPU).

AdamW is checked against torch.optim.AdamW (float64 on the CPU), a library
routine written independently. The regularizer terms are checked against
finite differences of the exact (SVD) regularizers on inputs where the
iteration has converged to rounding (spectrum inside [l, 1] with a table
built for that l), and against two facts of the decoupled step: it reduces to
AdamW at lambda = 0, and with eps = 0 the Hoyer gradient is orthogonal to W
(<W, G> = 0, Sec. 3.1), so a pure regularizer step lengthens W by exactly
(eta lambda)^2 ||G||^2 in squared norm.
"""
import numpy as np
import pytest
import torch

from oracle.exact import exact_grad, exact_values
from oracle.pe_schedule import pe_schedule
from oracle.slorr import HOYER, NUCLEAR, fwd_bwd
from oracle.training import AdamWState, adamw_step, alg2_accumulate, autograd_grads, decoupled_step

TAB = pe_schedule(6)
TAB_CONV = pe_schedule(6, ell=0.1)          # error ~1e-30 for normalised spectra in [0.1, 1]


def _converged_matrix(rng, M, N):
    """W whose normalised singular values lie in [0.1, 1]: W / ||W||_F has
    sigma_max <= 1 and sigma_min / ||W||_F >= 0.1 for these spectra."""
    P = min(M, N)
    U, _ = np.linalg.qr(rng.standard_normal((M, P)))
    V, _ = np.linalg.qr(rng.standard_normal((N, P)))
    s = np.linspace(1.0, 0.6, P)
    W = (U * s[None, :]) @ V.T
    assert (s.min() / np.linalg.norm(s)) >= 0.1
    return W


def _exact_L(W, kind):
    n, f, _, _ = exact_values(W)
    return n * n / (f * f) if kind == HOYER else n


def test_adamw_matches_torch_adamw():
    rng = np.random.default_rng(1)
    W0 = rng.standard_normal((7, 5))
    grads = [rng.standard_normal((7, 5)) for _ in range(4)]
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=3e-2, betas=(0.8, 0.95), eps=1e-6, weight_decay=0.1)
    st = AdamWState.zeros_like(W0)
    W = W0
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W = adamw_step(W, g, st, 3e-2, (0.8, 0.95), 1e-6, 0.1)
        assert np.allclose(W, p.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_decoupled_lambda_zero_is_adamw():
    rng = np.random.default_rng(2)
    Ws = [rng.standard_normal((6, 9)), rng.standard_normal((9, 4))]
    gs = [rng.standard_normal(W.shape) for W in Ws]
    st1 = [AdamWState.zeros_like(W) for W in Ws]
    st2 = [AdamWState.zeros_like(W) for W in Ws]
    new, _ = decoupled_step(Ws, gs, st1, 1e-2, 0.0, HOYER, TAB)
    for W, g, s, Wn in zip(Ws, gs, st2, new):
        assert np.array_equal(Wn, adamw_step(W, g, s, 1e-2))


def test_decoupled_pure_regularizer_step_is_orthogonal():
    rng = np.random.default_rng(3)
    Ws = [rng.standard_normal((12, 20)), rng.standard_normal((20, 12))]
    lr, lam = 0.05, 0.3
    st = [AdamWState.zeros_like(W) for W in Ws]
    new, G = decoupled_step(Ws, [None, None], st, lr, lam, HOYER, TAB)
    for W, Wn, g in zip(Ws, new, G):
        lhs = np.sum(Wn * Wn)
        rhs = np.sum(W * W) + (lr * lam) ** 2 * np.sum(g * g)
        assert lhs == pytest.approx(rhs, rel=1e-12)
        assert st[0].t == 0                                 # no AdamW step without a task gradient


@pytest.mark.parametrize("kind", [HOYER, NUCLEAR])
def test_decoupled_step_first_order_decrease(kind):
    """With no task gradient the step is W - h G_pre; on converged inputs
    G_pre is the exact gradient, so L(W) - L(W - h G) = h ||grad L||^2 + O(h^2)."""
    rng = np.random.default_rng(4)
    W = _converged_matrix(rng, 10, 16)
    h = 1e-6
    new, G = decoupled_step([W], [None], [AdamWState.zeros_like(W)], 1.0, h, kind, TAB_CONV)
    Ge = exact_grad(W, kind)
    drop = (_exact_L(W, kind) - _exact_L(new[0], kind)) / h
    assert drop > 0
    assert drop == pytest.approx(np.sum(Ge * Ge), rel=1e-4)


@pytest.mark.parametrize("kind", [HOYER, NUCLEAR])
def test_alg2_matches_finite_differences_of_task_plus_regularizer(kind):
    rng = np.random.default_rng(5)
    W = _converged_matrix(rng, 6, 9)
    C = rng.standard_normal(W.shape)
    lam = 0.7
    task_grad = W - C                                       # of 0.5 ||W - C||^2
    g = alg2_accumulate([W], [task_grad], lam, kind, TAB_CONV)[0]

    def total(X):
        return 0.5 * np.sum((X - C) ** 2) + lam * _exact_L(X, kind)

    fd = np.zeros_like(W)
    step = 1e-6
    for i in range(W.shape[0]):
        for j in range(W.shape[1]):
            E = np.zeros_like(W)
            E[i, j] = step
            fd[i, j] = (total(W + E) - total(W - E)) / (2 * step)
    assert np.linalg.norm(g - fd) <= 1e-7 * np.linalg.norm(fd)


def test_alg2_without_existing_gradient():
    rng = np.random.default_rng(6)
    W = rng.standard_normal((5, 8))
    lam = 0.25
    g = alg2_accumulate([W], [None], lam, HOYER, TAB)[0]
    ref = fwd_bwd(W, HOYER, TAB, g=lam).grad
    assert np.allclose(g, ref, rtol=1e-14, atol=1e-17)


def test_autograd_grads_weight_each_matrix():
    rng = np.random.default_rng(7)
    Ws = [_converged_matrix(rng, 6, 9), _converged_matrix(rng, 9, 6)]
    c = [0.5, -2.0]
    gs = autograd_grads(Ws, c, HOYER, TAB_CONV)
    for W, ci, g in zip(Ws, c, gs):
        assert np.linalg.norm(g - ci * exact_grad(W, HOYER)) <= 1e-12 * np.linalg.norm(g)
