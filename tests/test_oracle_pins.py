"""Pins for the oracle's forward + backward (float64).

Each test checks the oracle against something other than itself: the SVD
(LAPACK) with the scalar polynomial applied to the singular values, closed
forms for diagonal, orthonormal-row and rank-1 inputs, Prop. 1's bounds,
the textbook Newton-Schulz quintic, invariances stated in Sec. 3.1, and
finite differences of the exact regularizers.
"""
import numpy as np
import pytest

from oracle.exact import exact_grad, exact_values, prop1_bounds, prop1_delta, svd_parts
from oracle.pe_schedule import E_STOP, apply_scalar, greedy_step, pe_schedule
from oracle.slorr import HOYER, NUCLEAR, fwd_bwd, fwd_bwd_set, polar_iterate

TAB6 = pe_schedule(6)
NS5 = np.array([[1.875, -1.25, 0.375]])


def _spectral(W, table, eps):
    """P and n from the SVD: odd polynomials act on singular values alone."""
    U, s, Vt = np.linalg.svd(W, full_matrices=False)
    f = np.sqrt(np.sum(s * s))
    phi = apply_scalar(table, s / (f + eps))
    return (U * phi[None, :]) @ Vt, float(np.sum(s * phi))


def _mat_with_spectrum(rng, M, N, s):
    P = min(M, N)
    U, _ = np.linalg.qr(rng.standard_normal((M, P)))
    V, _ = np.linalg.qr(rng.standard_normal((N, P)))
    return (U * s[None, :]) @ V.T


@pytest.mark.parametrize("shape", [(8, 8), (12, 30), (30, 12), (64, 128), (128, 64), (1, 7), (7, 1)])
@pytest.mark.parametrize("eps", [0.0, 1e-3])
def test_P1_spectral_identity(shape, eps):
    rng = np.random.default_rng(hash(shape) % 2**32)
    W = rng.standard_normal(shape)
    for table in (TAB6, pe_schedule(3), pe_schedule(5, d=3), NS5):
        r = fwd_bwd(W, HOYER, table, eps)
        P, n = _spectral(W, table, eps)
        assert np.linalg.norm(r.polar - P) <= 1e-12 * max(1.0, np.linalg.norm(P))
        assert r.n_hat == pytest.approx(n, rel=1e-12, abs=1e-14)
        assert r.f == pytest.approx(np.linalg.norm(W), rel=1e-14)


@pytest.mark.parametrize("M,N", [(6, 6), (5, 9), (9, 5)])
def test_P2_diagonal(M, N):
    d = np.array([3.0, -1.5, 0.0, 0.25, -2.0, 1e-4, 0.7, 0.0, 5.0])[: min(M, N)]
    W = np.zeros((M, N))
    W[np.arange(len(d)), np.arange(len(d))] = d
    eps = 1e-2
    f = np.sqrt(np.sum(d * d))
    phi = apply_scalar(TAB6, np.abs(d) / (f + eps))
    r = fwd_bwd(W, HOYER, TAB6, eps)
    off = r.polar.copy()
    off[np.arange(len(d)), np.arange(len(d))] = 0.0
    assert np.all(off == 0.0)                                  # stays exactly diagonal
    assert np.allclose(np.diag(r.polar)[: len(d)], np.sign(d) * phi, rtol=1e-13, atol=0)
    n = float(np.sum(np.abs(d) * phi))
    assert r.n_hat == pytest.approx(n, rel=1e-14)
    assert r.value == pytest.approx((n / (f + eps)) ** 2, rel=1e-13)
    rn = fwd_bwd(W, NUCLEAR, TAB6, eps, g=0.5)
    assert rn.value == pytest.approx(n, rel=1e-14)
    assert np.allclose(rn.grad, 0.5 * r.polar, rtol=0, atol=0)


@pytest.mark.parametrize("P,Q", [(16, 16), (32, 80), (128, 256)])
def test_P3_orthonormal_rows(P, Q):
    rng = np.random.default_rng(P * Q)
    Qm, _ = np.linalg.qr(rng.standard_normal((Q, P)))
    W = Qm.T * 0.37                          # P x Q, W W^T = 0.37^2 I
    r = fwd_bwd(W, HOYER, TAB6)
    x = 1.0 / np.sqrt(P)                     # every normalised singular value
    phi = apply_scalar(TAB6, np.array([x]))[0]
    assert r.n_hat == pytest.approx(0.37 * P * phi, rel=1e-13)
    assert r.value == pytest.approx(P * phi ** 2, rel=1e-13)
    # Hoyer ratio of an orthogonal matrix is sqrt(rank) (up to the schedule error)
    E6 = greedy_step(*_last_interval(6))[1]
    assert abs(r.ratio - np.sqrt(P)) <= np.sqrt(P) * E6 * 1.0001
    # stationary point (maximum of the ratio): the gradient vanishes
    scale = 2 * r.n_hat / r.f ** 2 * np.linalg.norm(r.polar)
    assert np.linalg.norm(r.grad) <= 1e-12 * scale
    # nuclear: ||Q||_* = n estimate
    rn = fwd_bwd(Qm.T, NUCLEAR, TAB6)
    assert abs(rn.value - P) <= P * E6 * 1.0001


def _last_interval(T):
    lo, hi = 1e-3, 1.0
    for _ in range(T - 1):
        _, err, _ = greedy_step(lo, hi)
        lo, hi = 1 - err, 1 + err
    return lo, hi


@pytest.mark.parametrize("M,N", [(40, 40), (20, 70), (70, 20)])
def test_P4_rank_one(M, N):
    rng = np.random.default_rng(M + 7 * N)
    u, v = rng.standard_normal(M), rng.standard_normal(N)
    W = np.outer(u, v)
    phi1 = apply_scalar(TAB6, np.array([1.0]))[0]
    r = fwd_bwd(W, HOYER, TAB6)
    # rounding noise in the null space is amplified by phi'(0) = prod a_t ~ 2e3,
    # hence 1e-10 rather than 1e-12 here
    assert r.value == pytest.approx(phi1 ** 2, rel=1e-10)
    assert abs(r.value - 1.0) <= 2.1 * 9.2e-4          # Hoyer of rank 1 is 1
    scale = 2 * r.n_hat / r.f ** 2 * np.linalg.norm(r.polar)
    assert np.linalg.norm(r.grad) <= 1e-9 * scale       # global minimum
    rn = fwd_bwd(W, NUCLEAR, TAB6)
    uv = np.outer(u / np.linalg.norm(u), v / np.linalg.norm(v))
    assert np.allclose(rn.grad, phi1 * uv, atol=1e-10)


def _schedule_error(T, ell):
    """E_T of the greedy schedule, with the schedule's own stop rule."""
    lo, hi, err = ell, 1.0, None
    for _ in range(T):
        if err is not None and err < E_STOP:
            break
        _, err, _ = greedy_step(lo, hi)
        lo, hi = 1 - err, 1 + err
    return err


def test_P5_prop1_bounds_meaningful():
    """Normalised spectrum inside [l, 1], schedule built for that l: all four
    bounds of Prop. 1 hold, and so does the tighter per-schedule bound E_T."""
    rng = np.random.default_rng(5)
    checked = 0
    for M, N in [(24, 24), (20, 50), (50, 20), (8, 30)]:
        P = min(M, N)
        s = rng.uniform(0.5, 1.0, P)
        W = _mat_with_spectrum(rng, M, N, s)
        sig = np.linalg.svd(W, compute_uv=False)
        ell = 0.95 * sig.min() / np.linalg.norm(W)
        assert ell > 0.05
        for T in range(1, 7):
            tab = pe_schedule(T, ell)
            r = fwd_bwd(W, HOYER, tab)
            n, f, s1, UV = exact_values(W)
            # Prop. 1 is exact arithmetic; FL adds a float64 rounding floor once
            # delta drops below what float64 can resolve
            FL = 1e-10
            b_pol, b_nuc, b_val, b_grad = prop1_bounds(W, ell, T)
            assert np.linalg.norm(r.polar - UV, 2) <= b_pol + FL
            assert abs(r.n_hat - n) / n <= b_nuc + FL
            assert abs(r.value - (n / f) ** 2) / (n / f) ** 2 <= b_val + FL
            assert np.linalg.norm(r.grad - exact_grad(W, HOYER), 2) <= b_grad + FL
            err = _schedule_error(T, ell)
            assert np.linalg.norm(r.polar - UV, 2) <= err * (1 + 1e-9) + FL
            checked += b_pol < 0.5          # bounds that actually bite
    assert checked >= 4


def test_P5_prop1_with_newton_schulz_every_ell():
    """Classical NS5 satisfies 1 - p(x)^2 <= (1 - x^2)^3 on [0, 1], so the
    Prop. 1 bound with q = 2 holds for any l <= smallest normalised sigma."""
    x = np.linspace(0, 1, 200001)
    p = apply_scalar(NS5, x)
    assert np.max((1 - p ** 2) - (1 - x ** 2) ** 3) <= 1e-15
    rng = np.random.default_rng(11)
    for T in (1, 2, 3, 4, 6):
        W = rng.standard_normal((30, 45))
        sig = np.linalg.svd(W, compute_uv=False)
        ell = sig.min() / np.linalg.norm(W)
        table = np.repeat(NS5, T, axis=0)
        r = fwd_bwd(W, HOYER, table)
        n, f, s1, UV = exact_values(W)
        b_pol, b_nuc, b_val, b_grad = prop1_bounds(W, ell, T)
        assert prop1_delta(ell, T) == b_pol
        assert np.linalg.norm(r.polar - UV, 2) <= b_pol
        assert abs(r.n_hat - n) / n <= b_nuc
        assert abs(r.value - (n / f) ** 2) / (n / f) ** 2 <= b_val
        assert np.linalg.norm(r.grad - exact_grad(W, HOYER), 2) <= b_grad


def test_P5_paper_setting_is_vacuous_but_holds():
    """At the paper's l = 1e-3, T = 6 the bound is ~1 and trivially met."""
    assert prop1_delta(1e-3, 6) == pytest.approx((1 - 1e-6) ** 729, rel=1e-15)
    rng = np.random.default_rng(2)
    W = rng.standard_normal((40, 90))
    r = fwd_bwd(W, HOYER, TAB6)
    n, f, s1, UV = exact_values(W)
    b = prop1_bounds(W, 1e-3, 6)
    assert np.linalg.norm(r.polar - UV, 2) <= b[0]
    assert abs(r.n_hat - n) / n <= b[1]


@pytest.mark.parametrize("shape", [(33, 33), (17, 50), (50, 17)])
def test_P6_gradient_orthogonal_to_W(shape):
    """<W, grad> = 2 r (n/f^2 - n/f^4 * f^2) = 0 with eps = 0 (Sec. 3.1)."""
    rng = np.random.default_rng(6)
    W = rng.standard_normal(shape)
    r = fwd_bwd(W, HOYER, TAB6, eps=0.0)
    assert abs(np.sum(W * r.grad)) <= 1e-13 * np.linalg.norm(W) * np.linalg.norm(r.grad)


def test_P7_scale_invariance():
    rng = np.random.default_rng(7)
    W = rng.standard_normal((24, 40))
    r = fwd_bwd(W, HOYER, TAB6)
    for alpha in (2.0 ** -20, 0.125, 4.0, 2.0 ** 30):
        ra = fwd_bwd(alpha * W, HOYER, TAB6)
        assert ra.value == r.value                      # bitwise for 2^k
        assert np.array_equal(ra.grad * alpha, r.grad)
    ra = fwd_bwd(3.7 * W, HOYER, TAB6)
    assert ra.value == pytest.approx(r.value, rel=1e-14)
    assert np.allclose(ra.grad * 3.7, r.grad, rtol=1e-12, atol=1e-15)


def test_P8_transpose_invariance():
    rng = np.random.default_rng(8)
    for shape in [(20, 36), (36, 20), (25, 25)]:
        W = rng.standard_normal(shape)
        r, rt = fwd_bwd(W, HOYER, TAB6), fwd_bwd(W.T, HOYER, TAB6)
        assert rt.value == pytest.approx(r.value, rel=1e-13)
        assert np.allclose(rt.grad, r.grad.T, rtol=1e-11, atol=1e-14)
        if shape[0] != shape[1]:                      # same canonical operand
            assert np.array_equal(rt.polar, r.polar.T)


@pytest.mark.parametrize("kind", [HOYER, NUCLEAR])
def test_P9_exact_gradient_finite_differences(kind):
    """Eq. SLORR_grads against central differences of the SVD-based value."""
    rng = np.random.default_rng(9)
    W = rng.standard_normal((5, 8))

    def val(X):
        s = np.linalg.svd(X, compute_uv=False)
        n = np.sum(s)
        return n * n / np.sum(s * s) if kind == HOYER else n

    G = exact_grad(W, kind)
    h = 1e-6
    fd = np.zeros_like(W)
    for i in range(W.shape[0]):
        for j in range(W.shape[1]):
            E = np.zeros_like(W)
            E[i, j] = h
            fd[i, j] = (val(W + E) - val(W - E)) / (2 * h)
    assert np.allclose(G, fd, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("kind", [HOYER, NUCLEAR])
def test_converged_oracle_matches_exact_gradient(kind):
    """With every normalised sigma >= l and many steps the approximate value
    and gradient reach the exact ones: pins the whole O1-O7 chain, including
    the gradient formula's signs and powers of f."""
    rng = np.random.default_rng(10)
    W = rng.standard_normal((12, 20)) + 0.1
    sig = np.linalg.svd(W, compute_uv=False)
    ell = 0.9 * sig.min() / np.linalg.norm(W)
    tab = pe_schedule(10, ell)
    r = fwd_bwd(W, kind, tab, g=1.7)
    n, f, _, UV = exact_values(W)
    ref = 1.7 * exact_grad(W, kind)
    assert np.allclose(r.grad, ref, rtol=1e-12, atol=1e-13)
    assert r.value == pytest.approx((n / f) ** 2 if kind == HOYER else n, rel=1e-13)


def test_P10_prop2_one_exact_step():
    """After W+ = W - eta * grad (exact), sigma+_i = sigma_i + c (sigma_i - tau)
    with tau = f^2 / n and c = 2 eta n^2 / f^4 (App. B); the singular vectors
    do not move, so this is exact."""
    rng = np.random.default_rng(12)
    W = rng.standard_normal((9, 14))
    U, s, Vt = svd_parts(W)
    n, f = np.sum(s), np.sqrt(np.sum(s * s))
    eta = 1e-3
    Wp = W - eta * exact_grad(W, HOYER)
    sp = np.linalg.svd(Wp, compute_uv=False)
    tau, c = f * f / n, 2 * eta * n * n / f ** 4
    assert np.allclose(sp, s + c * (s - tau), rtol=1e-12)
    grew = sp > s
    assert np.array_equal(grew, s > tau)                  # Prop. 2


def test_zero_and_degenerate_inputs():
    Z = np.zeros((6, 9))
    for eps in (0.0, 1e-7):
        for kind in (HOYER, NUCLEAR):
            r = fwd_bwd(Z, kind, TAB6, eps)
            assert r.value == 0.0 and np.all(r.grad == 0.0)
    r = fwd_bwd(np.zeros((0, 4)), HOYER, TAB6)
    assert r.value == 0.0 and r.grad.shape == (0, 4)
    # 1 x N: a single singular value -> rank one
    v = np.arange(1.0, 6.0)[None, :]
    r = fwd_bwd(v, HOYER, TAB6)
    phi1 = apply_scalar(TAB6, np.array([1.0]))[0]
    assert r.value == pytest.approx(phi1 ** 2, rel=1e-13)    # P = 1: no null space


def test_rank_deficient_no_null_space_leak():
    """p(0) = 0: exact zero singular values stay zero (App. D remark)."""
    rng = np.random.default_rng(13)
    W = rng.standard_normal((10, 3)) @ rng.standard_normal((3, 16))
    r = fwd_bwd(W, NUCLEAR, TAB6)
    U, s, Vt = np.linalg.svd(W, full_matrices=True)
    null_l = U[:, 3:]
    assert np.linalg.norm(null_l.T @ r.polar) <= 1e-10


def test_eps_enters_both_sides():
    """f -> f + eps in the normalisation and in the value/gradient formula
    (Listing 1 adds eps to the norm once and reuses it)."""
    W = np.diag([2.0, 1.0])
    eps = 0.5
    f = np.sqrt(5.0)
    phi = apply_scalar(TAB6, np.array([2.0, 1.0]) / (f + eps))
    n = 2 * phi[0] + phi[1]
    r = fwd_bwd(W, HOYER, TAB6, eps)
    assert r.value == pytest.approx((n / (f + eps)) ** 2, rel=1e-14)
    rr = n / (f + eps)
    want = 2 * rr * (np.diag(phi) / (f + eps) - n / (f + eps) ** 3 * W)
    assert np.allclose(r.grad, want, rtol=1e-12, atol=0)


def test_set_total_in_index_order():
    rng = np.random.default_rng(14)
    Ws = [rng.standard_normal(s) for s in [(4, 9), (9, 4), (7, 7)]]
    res, tot = fwd_bwd_set(Ws, HOYER, TAB6)
    assert tot == (res[0].value + res[1].value) + res[2].value


def test_polar_iterate_is_the_quintic():
    """One step equals a X + b X^3 + c X^5 in the odd-power sense
    (X X^T)^k X, written out independently."""
    rng = np.random.default_rng(15)
    X = rng.standard_normal((6, 11)) * 0.1
    a, b, c = TAB6[0]
    X3 = X @ X.T @ X
    X5 = X @ X.T @ X @ X.T @ X
    assert np.allclose(polar_iterate(X, TAB6[:1]), a * X + b * X3 + c * X5, rtol=1e-13, atol=1e-16)
