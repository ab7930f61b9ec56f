"""Pins of the oracle's residual sampler (Prop. 1, Alg. 5, Alg. 7) (no GPU).

* Psi_alpha equals the trapezoid-normalised CDF of max(0, alpha N(u) - N(u - v))
  (the paper's own numerical method for its residual plots, App. D);
* sampled U follows that CDF (KS), down to alpha = e^-500;
* the paper-mode sampler (3 doublings, 4 bisections) stays inside the bracket and
  close to the exact inverse;
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
