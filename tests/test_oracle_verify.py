"""Pins of the oracle's verification (Alg. 2, Alg. 6) (no GPU).

* ell_j equals the difference of two Gaussian log-densities (scipy);
* token acceptance probability equals 2 Phi(-||m^p - m^q|| / (2 sigma))
  (the Mahalanobis form quoted in App. G) by Monte Carlo;
* the closed-form acceptance lemma (App. C, omega = 1) by Monte Carlo;
* the numerator v_j of h_j equals int max(0, alpha q - p) by brute-force 2-D quadrature;
* one round of block or token verification followed by the residual keeps
  the target chain's law exactly (KS on every produced step);
* block verification accepts at least as many steps as token verification;
* with a constant offset token verification's tau is geometric.
"""
import math

import numpy as np
import pytest
from scipy import stats
from scipy.special import ndtr

from oracle.residual import USAMPLE_EXACT, decomposition, usample
from oracle.verify import (block_log_h, block_verify, log_ratio_terms, log_v,
                           token_verify)


def test_log_ratio_is_log_density_difference():
    rng = np.random.default_rng(0)
    K, d = 4, 7
    mp = rng.standard_normal((K, d))
    mq = mp + 0.3 * rng.standard_normal((K, d))
    sigma = rng.uniform(0.2, 1.0, K)
    y = mp + sigma[:, None] * rng.standard_normal((K, d))
    nrm2, dot, ell = log_ratio_terms(y, mp, mq, sigma)
    for j in range(K):
        lq = stats.norm.logpdf(y[j], mq[j], sigma[j]).sum()
        lp = stats.norm.logpdf(y[j], mp[j], sigma[j]).sum()
        assert ell[j] == pytest.approx(lq - lp, rel=1e-10, abs=1e-10)
        assert nrm2[j] == pytest.approx(np.sum((mp[j] - mq[j]) ** 2) / sigma[j] ** 2, rel=1e-12)


@pytest.mark.parametrize("v", [0.3, 0.8, 2.0])
def test_token_acceptance_matches_mahalanobis_form(v):
    rng = np.random.default_rng(1)
    d, n = 3, 200000
    direction = rng.standard_normal(d)
    delta = v * direction / np.linalg.norm(direction)
    sigma = 0.5
    mq = np.zeros(d)
    mp = mq + sigma * delta
    y = mp + sigma * rng.standard_normal((n, d))
    _, _, ell = log_ratio_terms(y[:, None, :], np.broadcast_to(mp, (n, 1, d)),
                                np.broadcast_to(mq, (n, 1, d)), np.full((n, 1), sigma))
    p_acc = np.mean(np.minimum(1.0, np.exp(ell[:, 0])))
    expect = 2.0 * ndtr(-0.5 * np.linalg.norm(mp - mq) / sigma)
    assert p_acc == pytest.approx(expect, abs=4 * np.sqrt(expect * (1 - expect) / n))


@pytest.mark.parametrize("alpha,v", [(0.5, 1.0), (0.05, 2.0), (0.9, 0.3)])
def test_acceptance_lemma_closed_form(alpha, v):
    rng = np.random.default_rng(2)
    n = 200000
    z = rng.standard_normal((n, 2))
    delta = np.array([v, 0.0])
    ell = -(z @ delta) - 0.5 * v * v
    mc = np.mean(np.minimum(1.0, alpha * np.exp(ell)))
    A = math.log(alpha) / v - v / 2
    closed = ndtr(A) + alpha * (1 - ndtr(A + v))
    assert mc == pytest.approx(closed, abs=4.0 / np.sqrt(n))


@pytest.mark.parametrize("alpha,v", [(1.0, 0.3), (0.5, 1.0), (0.05, 2.0), (0.999, 0.01)])
def test_v_numerator_is_residual_mass(alpha, v):
    # int max(0, alpha N(y; m^q) - N(y; m^p)) dy in d = 2 on a grid, no reduction
    theta = 0.7
    mp = v * np.array([math.cos(theta), math.sin(theta)])
    h = 0.006
    g = np.arange(-9.0, 9.0 + h, h)
    X, Y = np.meshgrid(g, g, indexing="ij")
    q = np.exp(-0.5 * (X ** 2 + Y ** 2)) / (2 * np.pi)
    p = np.exp(-0.5 * ((X - mp[0]) ** 2 + (Y - mp[1]) ** 2)) / (2 * np.pi)
    mass = np.trapezoid(np.trapezoid(np.maximum(0.0, alpha * q - p), g, axis=1), g)
    assert math.exp(log_v(math.log(alpha), v)) == pytest.approx(mass, rel=2e-4, abs=1e-7)


def test_h_edge_readings():
    assert block_log_h(0.0, 1.3) == 0.0             # alpha_j = 1 -> h_j = 1
    assert block_log_h(-0.2, 0.0) == -math.inf      # ||Delta_{j+1}|| = 0, alpha < 1 -> h = 0
    # extreme log alpha stays finite and in (0, 1)
    lh = block_log_h(-1.0e4, 100.0)
    assert -math.inf < lh < 0.0


class _ToyChain:
    """A small 1-D non-Markov drafter and Markov target used to test exactness."""

    def __init__(self, K, offset=0.0):
        self.K = K
        self.offset = offset
        self.sig = np.array([0.6, 0.5, 0.45, 0.4, 0.35][: K + 1])

    def f(self, j, y):           # target mean of step j given the state
        return 0.9 * y + 0.3 * np.sin(y) + 0.1 * j

    def drafter(self, j, hist):  # draft mean of step j given the draft history
        return 0.85 * hist[-1] + 0.05 * hist[0] + 0.1 * j + 0.2 + self.offset * self.sig[j]


def _round(toy, y0, rng, mode):
    K = toy.K
    yh = [y0]
    mp = []
    for j in range(K):
        mp.append(toy.drafter(j, yh))
        yh.append(mp[-1] + toy.sig[j] * rng.standard_normal())
    mq = [toy.f(j, yh[j]) for j in range(K)]
    arr = lambda a: np.array(a)[:, None]
    nrm2, _, ell = log_ratio_terms(arr(yh[1:]), arr(mp), arr(mq), toy.sig[:K])
    eta = rng.uniform(size=K)
    res = block_verify(ell, nrm2, K, eta) if mode == "block" else token_verify(ell, K, eta)
    tau = res["tau"]
    out = list(yh[1:tau])
    if tau <= K:
        delta = np.array([(mp[tau - 1] - mq[tau - 1]) / toy.sig[tau - 1]])
        U = usample(rng.uniform(), res["log_alpha_res"], abs(delta[0]), USAMPLE_EXACT)
        out.append(decomposition(delta, [mq[tau - 1]], toy.sig[tau - 1], U, [0.0])[0])
    # finish the remaining steps with exact target draws
    while len(out) < K:
        j = len(out)
        out.append(toy.f(j, out[-1]) + toy.sig[j] * rng.standard_normal())
    return out, tau


# the last case has a large draft/target mismatch: there the block residual's
# weight alpha_{tau-1} is far from 1 often enough that drawing the residual
# with alpha = 1 instead is detected
@pytest.mark.parametrize("mode,K,offset,n", [("block", 2, 0.0, 12000), ("block", 3, 0.5, 12000),
                                             ("token", 3, 0.0, 12000), ("block", 2, 1.8, 30000)])
def test_one_round_is_exact(mode, K, offset, n):
    toy = _ToyChain(K, offset)
    rng = np.random.default_rng(10 + K)
    y0 = 0.4
    outs = np.array([_round(toy, y0, rng, mode)[0] for _ in range(n)])
    prev = np.full(n, y0)
    for j in range(K):
        z = (outs[:, j] - toy.f(j, prev)) / toy.sig[j]
        assert stats.kstest(z, "norm").pvalue > 1e-3, (mode, j)
        prev = outs[:, j]


def test_block_accepts_at_least_token():
    toy = _ToyChain(4)
    rng_b = np.random.default_rng(20)
    rng_t = np.random.default_rng(20)
    n = 6000
    tb = np.mean([_round(toy, 0.4, rng_b, "block")[1] for _ in range(n)])
    tt = np.mean([_round(toy, 0.4, rng_t, "token")[1] for _ in range(n)])
    assert tb >= tt - 0.02
    assert tb > tt  # strictly better on this toy


def test_token_tau_geometric_for_constant_offset():
    rng = np.random.default_rng(30)
    K, v, n = 5, 0.9, 40000
    taus = []
    for _ in range(n):
        z = rng.standard_normal(K)
        ell = -z * v - 0.5 * v * v
        taus.append(token_verify(ell, K, rng.uniform(size=K))["tau"])
    a = 2 * ndtr(-v / 2)
    expect = sum(a ** j for j in range(K + 1))
    assert np.mean(taus) == pytest.approx(expect, abs=4 * np.std(taus) / np.sqrt(n))


def test_degenerate_zero_offset_accepts_everything():
    rng = np.random.default_rng(40)
    K = 6
    ell = np.zeros(K)
    nrm2 = np.zeros(K)
    for _ in range(100):
        eta = rng.uniform(size=K)
        assert block_verify(ell, nrm2, K, eta)["tau"] == K + 1
        assert token_verify(ell, K, eta)["tau"] == K + 1
