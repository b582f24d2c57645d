"""Polar Express polynomial schedule, oracle side (float64).

The paper uses Polar Express (Sec. 3, "Computing the polar factor") with the
settings of its App. E.1: lower bound l = 1e-3 on the smallest normalised
singular value, polynomial degree d = 5, T = 6 steps, and the input first
divided by its Frobenius norm so that every singular value lies in [0, 1].
The coefficients themselves are not printed, so they are rebuilt here from
the definition Polar Express gives of its schedule:

  * step t holds an interval [l_t, u_t] that contains every (normalised)
    singular value; [l_1, u_1] = [l, 1];
  * p_t is the odd polynomial of degree d that minimises
        max_{x in [l_t, u_t]} |1 - p_t(x)|            (greedy minimax),
    with optimal error E_t;
  * the image of [l_t, u_t] under p_t is [1 - E_t, 1 + E_t], which is the next
    interval: l_{t+1} = 1 - E_t, u_{t+1} = 1 + E_t.

Because the recursion never looks ahead, the T-step schedule is the first T
rows of any longer one.

The minimax problem is solved by the Remez exchange. For d = 5 the best odd
quintic equioscillates at 4 points (l_t, two interior extrema, u_t) with error
signs +, -, +, - (p is below 1 at l_t, above 1 at u_t); for d = 3 at 3 points.
The polynomial is parametrised in the odd basis
    g1 = x,  g2 = x (x^2 - 1),  g3 = x (x^2 - 1)^2
which spans the same space as {x, x^3, x^5} but stays well conditioned when
the interval shrinks around 1 (late steps); the returned coefficients are the
monomial ones (a_t, b_t, c_t) of p_t(x) = a_t x + b_t x^3 + c_t x^5.

Reading (paper silent on the details): of the Polar Express stabilisations
the paper mentions, the safety factor is applied to the default table: every
step but the last evaluates p_t(x / 1.01) (stabilize, default_table). The
greedy schedule maps [l, 1] onto [1 - E_1, 1 + E_1] with 1 + E_1 close to 2,
and near the top of each interval the next polynomials are steep: without the
factor, the rounding of a 16-bit iterate can push a singular value past the
next interval, after which the later polynomials send it far off (a random
7 x 13 bf16 matrix reached 27 instead of 1). The cushioned lower bound is not
applied. pe_schedule returns the greedy rows themselves. Once the
error E_t falls below E_STOP = 1e-4, the minimax problem on the next interval
[1 - E_t, 1 + E_t] is no longer resolvable in float64 (its own optimal error
is ~0.6 E_t^3 for d = 5, ~E_t^2 for d = 3, at or below the rounding of 1). From
then on every step uses the limit of the greedy polynomial as the interval
shrinks to {1}: the odd polynomial with p(1) = 1 and as many vanishing
derivatives at 1 as the degree allows, i.e. the Newton-Schulz polynomial
(15 x - 10 x^3 + 3 x^5) / 8 for d = 5 and (3 x - x^3) / 2 for d = 3. With
l = 1e-3, d = 5, steps 1-7 are minimax solutions and steps 8+ Newton-Schulz.

This module is test infrastructure (see the package docstring).
"""
from __future__ import annotations

import numpy as np

__all__ = ["greedy_step", "pe_schedule", "apply_scalar", "E_STOP", "NEWTON_SCHULZ"]

E_STOP = 1e-4
NEWTON_SCHULZ = {5: (1.875, -1.25, 0.375), 3: (1.5, -0.5, 0.0)}


def _basis(x: np.ndarray, d: int) -> np.ndarray:
    z = (x - 1.0) * (x + 1.0)            # x^2 - 1, accurate near x = 1
    cols = [x, x * z]
    if d == 5:
        cols.append(x * z * z)
    return np.stack(cols, axis=-1)


def _to_monomial(w: np.ndarray, d: int) -> np.ndarray:
    # alpha x + beta (x^3 - x) + gamma (x^5 - 2 x^3 + x)
    if d == 3:
        alpha, beta = w
        return np.array([alpha - beta, beta, 0.0])
    alpha, beta, gamma = w
    return np.array([alpha - beta + gamma, beta - 2.0 * gamma, gamma])


def _interior_extrema(w: np.ndarray, d: int) -> np.ndarray:
    """Roots z = x^2 - 1 of p'(x) = 0, written in the basis weights."""
    if d == 3:
        alpha, beta = w
        # p' = alpha + beta (3 x^2 - 1) = (alpha + 2 beta) + 3 beta z
        return np.array([-(alpha + 2.0 * beta) / (3.0 * beta)])
    alpha, beta, gamma = w
    # p' = alpha + beta (3z + 2) + gamma (5 z^2 + 4 z)
    qa, qb, qc = 5.0 * gamma, 3.0 * beta + 4.0 * gamma, alpha + 2.0 * beta
    disc = qb * qb - 4.0 * qa * qc
    if disc < 0.0 or qa == 0.0:
        raise FloatingPointError("no real interior extrema")
    s = np.sqrt(disc)
    q = -0.5 * (qb + (s if qb >= 0.0 else -s))
    return np.sort(np.array([q / qa, qc / q]))


def greedy_step(lo: float, hi: float, d: int = 5, iters: int = 200):
    """Minimax odd polynomial of degree d approximating 1 on [lo, hi].

    Returns (coeffs[3] monomial (a, b, c), E, alternation points).
    """
    if d not in (3, 5):
        raise ValueError("degree must be 3 or 5")
    if not (0.0 < lo < hi):
        raise ValueError("need 0 < lo < hi")
    n_int = (d - 1) // 2                   # interior alternation points
    k = np.arange(1, n_int + 1)
    mid, rad = 0.5 * (lo + hi), 0.5 * (hi - lo)
    inner = mid - rad * np.cos(np.pi * k / (n_int + 1))   # Chebyshev start
    for _ in range(iters):
        pts = np.concatenate([[lo], inner, [hi]])
        signs = (-1.0) ** np.arange(pts.size)          # e(x_i) = +E, -E, ...
        # p(x_i) + s_i E = 1   for i = 0..n_int+1
        mat = np.concatenate([_basis(pts, d), signs[:, None]], axis=1)
        sol = np.linalg.solve(mat, np.ones(pts.size))
        w, err = sol[:-1], sol[-1]
        z = _interior_extrema(w, d)
        lo2, hi2 = (lo - 1.0) * (lo + 1.0), (hi - 1.0) * (hi + 1.0)
        if np.any(z <= lo2) or np.any(z >= hi2):
            raise FloatingPointError("extrema left the interval")
        new_inner = np.sqrt(1.0 + z)
        if np.max(np.abs(new_inner - inner)) <= 4e-16 * hi:
            inner = new_inner
            break
        inner = new_inner
    pts = np.concatenate([[lo], inner, [hi]])
    return _to_monomial(w, d), float(abs(err)), pts


def pe_schedule(T: int, ell: float = 1e-3, d: int = 5) -> np.ndarray:
    """First T rows (a_t, b_t, c_t) of the greedy Polar Express schedule."""
    if T < 1:
        raise ValueError("T >= 1")
    rows = []
    lo, hi = float(ell), 1.0
    err = None
    for _ in range(T):
        if err is not None and err < E_STOP:
            rows.append(np.array(NEWTON_SCHULZ[d]))
            continue
        coeffs, err, _ = greedy_step(lo, hi, d)
        rows.append(coeffs)
        lo, hi = 1.0 - err, 1.0 + err
    return np.array(rows, dtype=np.float64)


DEFAULT_SAFETY = 0.01


def stabilize(table, delta: float = DEFAULT_SAFETY) -> np.ndarray:
    """The schedule with the numerical stabilisation applied (the reading taken
    of the paper's unspecified stabilisations of Polar Express): every step but
    the last evaluates its polynomial at x / (1 + delta),
        p_t(x / s) = (a_t / s) x + (b_t / s^3) x^3 + (c_t / s^5) x^5,  s = 1 + delta,
    so that a singular value pushed slightly above the step's interval by the
    rounding of a low-precision iterate is mapped back inside the next one
    instead of off the polynomial's controlled range."""
    t = np.array(table, dtype=np.float64, copy=True)
    s = 1.0 + float(delta)
    t[:-1, 0] /= s
    t[:-1, 1] /= s ** 3
    t[:-1, 2] /= s ** 5
    return t


def default_table(T: int, ell: float = 1e-3, d: int = 5, delta: float = DEFAULT_SAFETY) -> np.ndarray:
    """The default coefficient table: the first T greedy rows, stabilised."""
    return stabilize(pe_schedule(T, ell, d), delta)


def apply_scalar(table: np.ndarray, x: np.ndarray) -> np.ndarray:
    """phi(x) = p_T(...p_1(x)): the scalar map the matrix iteration applies
    to every singular value (odd polynomials commute with the SVD)."""
    y = np.asarray(x, dtype=np.float64).copy()
    for a, b, c in table:
        y2 = y * y
        y = a * y + b * y * y2 + c * y * y2 * y2
    return y
