"""Pins for the oracle's Polar Express schedule (greedy minimax odd polynomials).

Checked against what the mathematics fixes, not against the generator's own
code: the Chebyshev alternation theorem on a dense grid, the interval
recursion, the prefix property of a greedy schedule, the textbook
Newton-Schulz limits, and the per-step error guarantee on [l, 1].
"""
import json
import os

import numpy as np
import pytest

from oracle.pe_schedule import E_STOP, apply_scalar, default_table, greedy_step, pe_schedule, stabilize

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def _poly(c, x):
    return c[0] * x + c[1] * x ** 3 + c[2] * x ** 5


def _grid_extrema(c, lo, hi, n=400001):
    """Local extrema of e(x) = 1 - p(x) on a dense grid, endpoints included."""
    x = np.linspace(lo, hi, n)
    e = 1.0 - _poly(c, x)
    idx = [0]
    d = np.diff(e)
    for i in range(1, len(d)):
        if d[i - 1] * d[i] < 0:
            idx.append(i)
    idx.append(n - 1)
    return x[idx], e[idx], np.max(np.abs(e))


def _intervals(T, ell=1e-3, d=5):
    lo, hi, out = ell, 1.0, []
    for _ in range(T):
        c, err, _ = greedy_step(lo, hi, d)
        out.append((lo, hi, c, err))
        if err < E_STOP:
            break
        lo, hi = 1.0 - err, 1.0 + err
    return out


@pytest.mark.parametrize("d", [3, 5])
def test_alternation_theorem_on_dense_grid(d):
    """Best approximation <=> equioscillation at d//2 + 2 points with alternating
    signs and equal magnitude (Chebyshev alternation theorem)."""
    for lo, hi, c, err in _intervals(6, d=d):
        if hi - lo < 1e-6:
            continue          # grid too coarse for the last, tiny intervals
        xs, es, emax = _grid_extrema(c, lo, hi)
        assert len(xs) == d // 2 + 2, (lo, hi, xs)
        assert np.allclose(np.abs(es), emax, rtol=1e-6, atol=0)
        assert np.all(np.sign(es) == (-1.0) ** np.arange(len(es)))   # +, -, +, -
        assert es[0] > 0                                           # p(l_t) < 1
        assert emax == pytest.approx(err, rel=1e-6)


def test_interval_recursion():
    """Image of [l_t, u_t] is [1 - E_t, 1 + E_t] = [l_{t+1}, u_{t+1}]."""
    steps = _intervals(7)
    for (lo, hi, c, err), nxt in zip(steps[:-1], steps[1:]):
        assert _poly(c, lo) == pytest.approx(1.0 - err, abs=1e-13)
        assert _poly(c, hi) == pytest.approx(1.0 + err, abs=1e-13)
        assert nxt[0] == pytest.approx(1.0 - err, abs=1e-15)
        assert nxt[1] == pytest.approx(1.0 + err, abs=1e-15)
    errs = [s[3] for s in steps]
    assert all(e2 < e1 for e1, e2 in zip(errs, errs[1:]))            # monotone
    assert steps[0][0] == GOLDEN["polar_express"]["ell"]


def test_prefix_property():
    """A greedy schedule never looks ahead: T rows = first T rows of 12."""
    full = pe_schedule(12)
    for T in range(1, 12):
        assert np.array_equal(pe_schedule(T), full[:T])


@pytest.mark.parametrize("d,key", [(5, "newton_schulz_quintic"), (3, "newton_schulz_cubic")])
def test_newton_schulz_limit(d, key):
    """As the interval shrinks to {1}, the minimax polynomial tends to the
    Newton-Schulz polynomial with p(1) = 1 and as many vanishing derivatives."""
    ns = np.array(GOLDEN[key]["coeffs"])
    tab = pe_schedule(12, d=d)
    assert np.allclose(tab[-1], ns, atol=1e-5)
    if d == 5:
        assert np.allclose(tab[6], ns, atol=2e-6)    # step 7 already (E_6 ~ 9e-4)


def test_guarantee_on_unit_interval():
    """phi = p_T o ... o p_1 maps [l, 1] into [1 - E_T, 1 + E_T]."""
    ell = GOLDEN["polar_express"]["ell"]
    for T in range(1, 8):
        tab = pe_schedule(T, ell)
        err = _intervals(T, ell)[T - 1][3]
        x = np.concatenate([np.geomspace(ell, 1.0, 200001), np.linspace(ell, 1.0, 200001)])
        phi = apply_scalar(tab, x)
        assert np.max(np.abs(1.0 - phi)) <= err * (1 + 1e-9) + 1e-15


def test_first_step_values():
    """Spot values of the recursion for l = 1e-3, d = 5: the interval after
    step t (l_{t+1}) and E_6, recomputed by brute-force grid minimisation of
    the step-1 error over (a, b, c) around the Remez solution."""
    steps = _intervals(7)
    l_next = [1.0 - s[3] for s in steps[:6]]
    assert l_next[0] == pytest.approx(0.00847, rel=2e-3)
    assert l_next[5] == pytest.approx(0.99908, rel=1e-5)
    # no nearby (a, b, c) does better on [l, 1] than the Remez answer
    lo, hi, c, err = steps[0]
    x = np.linspace(lo, hi, 20001)
    rng = np.random.default_rng(0)
    for _ in range(200):
        cc = c + rng.normal(scale=1e-3, size=3) * np.abs(c)
        assert np.max(np.abs(1.0 - _poly(cc, x))) >= err * (1 - 1e-9)


def test_scalar_map_is_odd_and_zero_at_zero():
    tab = pe_schedule(6)
    x = np.linspace(-1, 1, 1001)
    assert np.allclose(apply_scalar(tab, -x), -apply_scalar(tab, x), rtol=0, atol=0)
    assert apply_scalar(tab, np.array([0.0]))[0] == 0.0
    # slope at 0 is prod a_t (the small-singular-value gain)
    assert apply_scalar(tab, np.array([1e-12]))[0] / 1e-12 == pytest.approx(np.prod(tab[:, 0]), rel=1e-9)


def _perturbed_map(tab, x, push):
    """The scalar map with every intermediate value pushed up by the factor
    (1 + push) before each step: the worst direction of an iterate's rounding
    near the top of an interval."""
    y = np.asarray(x, dtype=np.float64).copy()
    for a, b, c in tab:
        y = y * (1.0 + push)
        y = a * y + b * y ** 3 + c * y ** 5
    return y


def test_stabilised_table():
    """default_table = the greedy rows with every step but the last evaluated
    at x / (1 + delta): the rows are the argument-scaled polynomials (checked
    as values of p_t at sample points), delta = 0 leaves the table unchanged,
    and the property the scaling is for holds: with every intermediate value
    pushed up by 0.5 % (a rounding-sized perturbation at the steep top end of
    an interval) the stabilised map stays within 2 % of 1 on [l, 1], while the
    plain greedy map leaves the polynomials' controlled range."""
    raw = pe_schedule(6)
    assert np.array_equal(stabilize(raw, 0.0), raw)
    tab = default_table(6)
    assert np.array_equal(tab[-1], raw[-1])
    xs = np.linspace(-1.5, 1.5, 301)
    for t in range(5):
        want = _poly(raw[t], xs / 1.01)
        assert np.allclose(_poly(tab[t], xs), want, rtol=1e-13, atol=1e-13)
    x = np.linspace(1e-3, 1.0, 100001)
    assert np.max(np.abs(1.0 - _perturbed_map(tab, x, 0.005))) <= 0.02
    assert np.max(np.abs(_perturbed_map(raw, x, 0.005))) > 10.0
    # the unperturbed stabilised map still converges on [l, 1]
    assert np.max(np.abs(1.0 - apply_scalar(tab, x))) <= 4e-3
