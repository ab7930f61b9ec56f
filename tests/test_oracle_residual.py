"""Pins of the oracle's residual sampler (Prop. 1, Alg. 5, Alg. 7) (no GPU).

* Psi_alpha equals the trapezoid-normalised CDF of max(0, alpha N(u) - N(u - v))
  (the paper's own numerical method for its residual plots, App. D);
* sampled U follows that CDF (KS), down to alpha = e^-500;
* the paper-mode sampler (3 doublings, 4 bisections, tolerance 1e-6) equals the
  dyadic midpoint that the exact inverse of Psi fixes, including a binding
  doubling cap and early stops after 0..3 bisections;
* the Decomposition residual has density ∝ max(0, alpha q - p) in y-space (d = 1),
  and in d = 2, 8 its e-component follows psi_alpha while the orthogonal part is
  an independent N(0, I - e e^T).
"""
import math

import numpy as np
import pytest
from scipy import stats

from oracle.residual import (USAMPLE_EXACT, USAMPLE_PAPER, decomposition,
                             log_cdf, upper_end, usample)


def _trapezoid_cdf(log_alpha, v, npts=400001):
    """CDF of psi_alpha on a grid ending at the support's right end, by trapezoid."""
    us = log_alpha / v + v / 2
    lo = min(-12.0, us - 40.0 / max(1.0, abs(us)))
    u = np.linspace(lo, us, npts)
    # alpha N(u) - N(u - v) = alpha N(u) (1 - exp(u v - v^2/2 - log alpha))
    expo = np.minimum(u * v - 0.5 * v * v - log_alpha, 0.0)
    logf = log_alpha + stats.norm.logpdf(u) + np.log(-np.expm1(expo) + 1e-300)
    f = np.exp(logf - logf.max())
    c = np.concatenate([[0.0], np.cumsum(0.5 * (f[1:] + f[:-1]) * np.diff(u))])
    return u, c / c[-1]


CASES = [(0.0, 0.05), (0.0, 1.0), (0.0, 30.0), (math.log(0.5), 1.0), (math.log(1e-3), 1.0),
         (math.log(0.5), 0.05), (-500.0, 0.05), (-500.0, 30.0), (math.log(1e-3), 30.0)]


@pytest.mark.parametrize("log_alpha,v", CASES)
def test_cdf_matches_trapezoid(log_alpha, v):
    u, c = _trapezoid_cdf(log_alpha, v)
    for q in (0.01, 0.2, 0.5, 0.8, 0.99):
        x = float(np.interp(q, c, u))
        assert math.exp(log_cdf(x, log_alpha, v)) == pytest.approx(q, abs=2e-5)
    assert log_cdf(upper_end(log_alpha, v) + 1e-9, log_alpha, v) == 0.0


@pytest.mark.parametrize("log_alpha,v", CASES)
def test_usample_follows_psi(log_alpha, v):
    rng = np.random.default_rng(abs(hash((log_alpha, v))) % 2 ** 32)
    us = upper_end(log_alpha, v)
    draws = np.array([usample(rng.uniform(), log_alpha, v, USAMPLE_EXACT) for _ in range(1500)])
    assert np.all(draws <= us)
    u, c = _trapezoid_cdf(log_alpha, v)
    assert stats.kstest(draws, lambda t: np.interp(t, u, c)).pvalue > 1e-3


@pytest.mark.parametrize("log_alpha,v", [(0.0, 1.0), (math.log(0.5), 1.0), (-500.0, 30.0)])
def test_usample_paper_mode_close_to_exact(log_alpha, v):
    rng = np.random.default_rng(5)
    us = upper_end(log_alpha, v)
    for _ in range(200):
        u = rng.uniform()
        ue = usample(u, log_alpha, v, USAMPLE_EXACT)
        up = usample(u, log_alpha, v, USAMPLE_PAPER)
        assert up <= us
        # 4 bisection steps on a bracket of width <= 2^3 leave at most 2^-2 (plus
        # the case where 3 doublings do not reach the quantile)
        if math.exp(log_cdf(us - 8.0, log_alpha, v)) <= u:
            assert abs(up - ue) <= 0.25 + 1e-12


@pytest.mark.parametrize("alpha", [1.0, 0.3])
def test_decomposition_density_in_y_space(alpha):
    rng = np.random.default_rng(7)
    mq, mp, sigma = 0.2, 0.9, 0.5
    delta = np.array([(mp - mq) / sigma])
    v = abs(delta[0])
    ys = np.array([decomposition(delta, [mq], sigma,
                                 usample(rng.uniform(), math.log(alpha), v), [0.0])[0]
                   for _ in range(4000)])
    # density max(0, alpha N(y; m^q, s^2) - N(y; m^p, s^2)) on a grid, written in y
    grid = np.linspace(-6, 6, 200001)
    f = np.maximum(0.0, alpha * stats.norm.pdf(grid, mq, sigma) - stats.norm.pdf(grid, mp, sigma))
    c = np.concatenate([[0.0], np.cumsum(0.5 * (f[1:] + f[:-1]) * np.diff(grid))])
    c /= c[-1]
    assert stats.kstest(ys, lambda t: np.interp(t, grid, c)).pvalue > 1e-3


@pytest.mark.parametrize("d", [2, 8])
def test_decomposition_orthogonal_structure(d):
    rng = np.random.default_rng(8 + d)
    mq = rng.standard_normal(d)
    mp = mq + 0.4 * rng.standard_normal(d)
    sigma, log_alpha = 0.7, math.log(0.6)
    delta = (mp - mq) / sigma
    v = np.linalg.norm(delta)
    e = delta / v
    n = 4000
    ys = np.array([decomposition(delta, mq, sigma, usample(rng.uniform(), log_alpha, v),
                                 rng.standard_normal(d)) for _ in range(n)])
    z = (ys - mq) / sigma
    proj = z @ e
    u, c = _trapezoid_cdf(log_alpha, v)
    assert stats.kstest(proj, lambda t: np.interp(t, u, c)).pvalue > 1e-3
    # orthonormal basis of e-perp
    basis = np.linalg.svd(np.eye(d) - np.outer(e, e))[0][:, : d - 1]
    perp = z @ basis
    for i in range(d - 1):
        assert stats.kstest(perp[:, i], "norm").pvalue > 1e-4
        assert abs(np.corrcoef(perp[:, i], proj)[0, 1]) < 4.5 / np.sqrt(n)


PAPER_TOL = 1e-6   # the reading of the paper-mode tolerance (its value is not given)


def _paper_mode_from_exact(u, log_alpha, v):
    """The paper-mode draw (<= 3 doublings, <= 4 bisections, |Psi(mid) - u| <= tol)
    derived from the exact inverse of Psi alone.

    Psi is increasing on its support, so Psi(x) > u <=> x > Psi^-1(u) and
    |Psi(x) - u| <= tol <=> Psi^-1(u - tol) <= x <= Psi^-1(u + tol).  Doubling
    from [u* - 1, u*] stops at the first n in 0..3 with u* - 2^n <= Psi^-1(u),
    so the bracket is [u* - 2^n, u*] of width W = 2^n; after i bisections the
    midpoint is the centre of the dyadic cell holding t = (Psi^-1(u) - lo)/W
    (t clamped to [0, 1]: when the cap binds every midpoint lies above the
    quantile), lo + W (floor(2^i t) + 1/2) / 2^i.  The draw is the first of
    these midpoints (i = 0..3) inside the tolerance window, else the one after
    the fourth bisection.  Returns (draw, doublings, bisections)."""
    us = upper_end(log_alpha, v)

    def inv(q):
        return usample(q, log_alpha, v, USAMPLE_EXACT)

    ue = inv(u)
    n = next((n for n in range(4) if us - 2.0 ** n <= ue), 3)
    lo, width = us - 2.0 ** n, 2.0 ** n
    t = min(max((ue - lo) / width, 0.0), 1.0)
    wl = inv(u - PAPER_TOL) if u - PAPER_TOL > 0.0 else -math.inf
    wh = inv(u + PAPER_TOL) if u + PAPER_TOL < 1.0 else math.inf
    for i in range(5):
        j = min(math.floor(2 ** i * t), 2 ** i - 1)
        mid = lo + width * (j + 0.5) / 2 ** i
        if i == 4 or wl <= mid <= wh:
            return mid, n, i


def _u_with_exact_inverse_at(x, log_alpha, v):
    """The u in (0, 1) whose exact inverse is x (bisection on u; Psi^-1 is increasing)."""
    a, b = 0.0, 1.0
    for _ in range(80):
        m = 0.5 * (a + b)
        if usample(m, log_alpha, v, USAMPLE_EXACT) < x:
            a = m
        else:
            b = m
    return 0.5 * (a + b)


@pytest.mark.parametrize("log_alpha,v", [(0.0, 1.0), (math.log(0.5), 1.0), (math.log(1e-3), 0.3),
                                         (-500.0, 30.0), (0.0, 0.05)])
def test_usample_paper_mode_equals_dyadic_closed_form(log_alpha, v):
    # App. "Experimental details" / Alg. 7: the capped doubling and bisection.
    # Random u (no early stop in practice), a u so small that the three
    # doublings do not reach the quantile (the cap binds), and u placed just
    # inside (and, as a control, just outside) the tolerance window of the
    # midpoint after i bisections (i = 0..3).
    us = upper_end(log_alpha, v)
    tol = 1e-12 * max(1.0, abs(us))   # the candidates are >= 1/32 apart
    rng = np.random.default_rng(17)
    cases = [(float(q), None) for q in rng.uniform(size=60)] + [(1e-300, "cap")]
    lo0 = us - 1.0
    for i in range(4):
        # the midpoint after i bisections of [u* - 1, u*] when the quantile is
        # in its lowest dyadic cell: u* - 1 + 2^-(i+1)
        target = lo0 + 2.0 ** -(i + 1)
        q = _u_with_exact_inverse_at(target, log_alpha, v)
        if 10 * PAPER_TOL < q < 1.0 - 10 * PAPER_TOL:
            cases.append((q + 0.4 * PAPER_TOL, i))
            cases.append((q + 3.0 * PAPER_TOL, -1 - i))
    stops = set()
    for u, kind in cases:
        want, n, i = _paper_mode_from_exact(u, log_alpha, v)
        got = usample(u, log_alpha, v, USAMPLE_PAPER)
        assert abs(got - want) <= tol, (u, kind, got, want, n, i)
        if kind == "cap":
            assert n == 3 and usample(u, log_alpha, v, USAMPLE_EXACT) < us - 8.0
        elif kind is not None and kind >= 0:
            assert i <= kind, (u, kind, i)
            stops.add(i)
        elif kind is not None:
            # just outside the window: the draw is not that midpoint
            assert abs(got - (lo0 + 2.0 ** kind)) > tol, (u, kind, got)
    assert stops, "no early stop was constructed"
