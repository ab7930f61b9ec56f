"""Pins of the oracle's VP schedule and Gaussian-mixture target (no GPU).

* abar(s) equals exp(-int_0^s beta) by quadrature;
* a one-component mixture reduces to the textbook Gaussian score;
* the mixture score is the gradient of the mixture log-density (finite differences);
* the marginal q_s matches samples of the forward process (KS, d = 1);
* the Euler-Maruyama chain m^q_n(y) + sigma_n xi, started from N(0, I), ends at
  the data law for two churn values (this pins sigma_n, c1_n, c2_n together);
* above d = 64 the squared distances by the norm expansion equal the direct
  differences, and so do the scores built on them.
"""
import numpy as np
import pytest
from scipy import integrate, stats
from scipy.special import logsumexp

from oracle.gmm import GMM, target_mean
from oracle.schedule import Schedule


def test_abar_matches_quadrature():
    sch = Schedule(100)
    for s in (0.0, 0.01, 0.3, 0.77, 1.0):
        integral, _ = integrate.quad(lambda t: float(sch.beta(t)), 0.0, s)
        assert sch.abar(s) == pytest.approx(np.exp(-integral), rel=1e-12, abs=1e-300)


def test_schedule_step_times():
    sch = Schedule(200, churn=0.5)
    assert sch.fwd_time(0) == 1.0
    assert sch.fwd_time(199) == pytest.approx(1.0 / 200)
    # sigma^2 is the EM increment variance eps^2 g^2 delta
    assert sch.sigma(10) ** 2 == pytest.approx(0.25 * float(sch.beta(1 - 10 / 200)) / 200)


def test_single_component_score_is_gaussian_score():
    rng = np.random.default_rng(0)
    d = 5
    mu = rng.standard_normal((1, d))
    g = GMM(mu, [0.3], [0.0])
    x = rng.standard_normal((7, d))
    a = 0.6
    s2 = a * a * 0.3 + 1 - a * a
    assert np.allclose(g.score(x, a), (a * mu - x) / s2, rtol=1e-12, atol=1e-12)


def test_score_is_gradient_of_log_density():
    rng = np.random.default_rng(1)
    d, M = 3, 5
    g = GMM(rng.standard_normal((M, d)) * 1.5, rng.uniform(0.05, 0.5, M),
            np.log(rng.dirichlet(np.ones(M))))
    x = rng.standard_normal((6, d))
    for a in (0.05, 0.5, 0.95):
        sc = g.score(x, a)
        h = 1e-5
        fd = np.empty_like(x)
        for i in range(d):
            e = np.zeros(d)
            e[i] = h
            fd[:, i] = (g.log_density(x + e, a) - g.log_density(x - e, a)) / (2 * h)
        assert np.allclose(sc, fd, rtol=1e-6, atol=1e-6)


def _mixture_logpdf_1d(y, mu, var, w, a):
    comps = [np.log(w[m]) + stats.norm.logpdf(y, a * mu[m], np.sqrt(a * a * var[m] + 1 - a * a))
             for m in range(len(w))]
    return logsumexp(np.stack(comps), axis=0)


def test_log_density_matches_forward_process_samples():
    rng = np.random.default_rng(2)
    mu = np.array([[-2.0], [0.5], [3.0]])
    var = np.array([0.1, 0.4, 0.2])
    w = np.array([0.5, 0.2, 0.3])
    g = GMM(mu, var, np.log(w))
    a = 0.7
    # oracle density equals an independent scipy mixture density
    ys = np.linspace(-5, 6, 41)
    assert np.allclose(g.log_density(ys[:, None], a), _mixture_logpdf_1d(ys, mu[:, 0], var, w, a),
                       rtol=1e-12, atol=1e-12)
    # and samples of X_s = a X_0 + sqrt(1 - a^2) eps follow it
    n = 40000
    comp = rng.choice(3, size=n, p=w)
    x0 = mu[comp, 0] + np.sqrt(var[comp]) * rng.standard_normal(n)
    xs = a * x0 + np.sqrt(1 - a * a) * rng.standard_normal(n)
    grid = np.linspace(-8, 9, 20001)
    pdf = np.exp(g.log_density(grid[:, None], a))
    cdf = np.concatenate([[0.0], np.cumsum(0.5 * (pdf[1:] + pdf[:-1]) * np.diff(grid))])
    assert cdf[-1] == pytest.approx(1.0, abs=1e-6)
    assert stats.kstest(xs, lambda t: np.interp(t, grid, cdf)).pvalue > 1e-3


@pytest.mark.parametrize("churn", [1.0, 0.5])
def test_em_chain_reaches_data_law(churn):
    # Gaussian data N(mu0, v0): the generative SDE maps N(0, I) at t = 0 to the data
    # law at t = 1; Euler-Maruyama with N = 1000 steps is within O(delta) of it.
    mu0, v0 = 1.5, 0.3
    g = GMM(np.array([[mu0]]), [v0], [0.0])
    sch = Schedule(1000, churn=churn)
    rng = np.random.default_rng(3)
    y = rng.standard_normal((20000, 1))
    for n in range(sch.n_steps):
        mq, _ = target_mean(g, sch, y, n)
        y = mq + sch.sigma(n) * rng.standard_normal(y.shape)
    assert y.mean() == pytest.approx(mu0, abs=0.03)
    assert y.var() == pytest.approx(v0, rel=0.05)


@pytest.mark.parametrize("d,M,a", [(3072, 64, 0.02), (3072, 64, 0.9), (16384, 24, 0.5), (65, 7, 0.99)])
def test_expanded_distances_match_direct(d, M, a):
    # above d = 64 the oracle forms ||x - a mu||^2 by the float64 norm
    # expansion (one matrix product); the direct differences on a subset of
    # rows fix it: rows near a component, far from all of them, and at the
    # data end (a close to 1, small s2) where the logits are sharpest
    rng = np.random.default_rng(d + M)
    mu = rng.standard_normal((M, d))
    var = rng.uniform(0.01, 0.2, M)
    g = GMM(mu, var, np.log(rng.dirichlet(np.ones(M))))
    x = np.concatenate([a * mu[:3] + 0.1 * rng.standard_normal((3, d)),
                        rng.standard_normal((2, d)) * 3.0])
    av = np.full(len(x), a)
    direct = g.sq_dist(x, av, direct=True)
    expd = g.sq_dist(x, av, direct=False)
    assert np.allclose(expd, direct, rtol=1e-12, atol=0.0)
    sd = g.score(x, a, direct=True)
    se = g.score(x, a, direct=False)
    err = np.linalg.norm(se - sd, axis=1) / np.linalg.norm(sd, axis=1)
    assert err.max() <= 1e-9, err
