"""Pins of the oracle's variants: the reflection residual (Alg. 4), the Frozen
Drafter (Sec. 3.3) and temperature (App. "Temperature") (no GPU).

Reflection:
* (I - 2 e e^T) is an isometry that negates the e-component, keeps the
  orthogonal part and is its own inverse;
* one round of sample verification with the reflection residual outputs
  exactly q = N(m^q, sigma^2 I) (KS per coordinate and along e, d = 2);
* the full sampler with token verification and the reflection residual
  follows the plain Euler-Maruyama law.
Temperature:
* the tempered sample-verification acceptance matches its closed form
  P_acc(omega) = Phi(-v/2) + exp(v^2 c (c - 1)/2) Phi(v/2 - c v), c = omega^-2
  (the expectation of min(1, e^{c ell}) over ell ~ N(-v^2/2, v^2));
* the output mean shift of one tempered round with the untempered
  decomposition residual matches m^q + sigma e g(v, omega) with g computed by
  quadrature, zero at omega = 1, positive above and negative below (the
  temperature proposition);
* block verification with K_b = 1 takes the same coins as sample
  verification at any omega, and omega = 1 changes nothing;
* block efficiency grows with omega.
Frozen Drafter:
* Delta_1 = 0 in every round (the first draft mean is the target mean at the
  state), so every round accepts the first draft;
* with K = 1 the sampler is, path by path, the plain EM chain whose odd steps
  take the DRAFT noise and even steps the TARGET noise of the round;
* the sampler follows the plain EM law.
"""
import math

import numpy as np
import pytest
from scipy import integrate, stats

from oracle import philox
from oracle import sampler as S
from oracle.gmm import GMM, target_mean
from oracle.residual import USAMPLE_EXACT, decomposition, reflection, usample
from oracle.schedule import Schedule
from oracle.verify import block_verify, log_ratio_terms, token_verify


def _gmm(d, seed):
    rng = np.random.default_rng(seed)
    M = 3
    return GMM(rng.standard_normal((M, d)) * 2.0, rng.uniform(0.05, 0.5, M),
               np.log(rng.dirichlet(np.ones(M))))


# ------------------------------------------------------------- reflection --
def test_reflection_is_householder():
    rng = np.random.default_rng(1)
    d = 7
    delta = rng.standard_normal(d)
    z = rng.standard_normal(d)
    mq = rng.standard_normal(d)
    s = 0.3
    e = delta / np.linalg.norm(delta)
    zr = (reflection(delta, z, mq, s) - mq) / s
    assert np.linalg.norm(zr) == pytest.approx(np.linalg.norm(z), rel=1e-14)
    assert zr @ e == pytest.approx(-(z @ e), rel=1e-13)
    perp = lambda v: v - e * (e @ v)
    np.testing.assert_allclose(perp(zr), perp(z), rtol=0, atol=1e-14)
    back = (reflection(delta, zr, mq, s) - mq) / s
    np.testing.assert_allclose(back, z, rtol=0, atol=1e-14)
    # the scale of Delta does not matter, only its direction
    np.testing.assert_allclose(reflection(5.0 * delta, z, mq, s), reflection(delta, z, mq, s),
                               rtol=0, atol=1e-14)


@pytest.mark.parametrize("shift", [0.4, 1.5])
def test_reflection_round_outputs_target(shift):
    rng = np.random.default_rng(2)
    d, n, s = 2, 6000, 0.8
    mq = np.array([0.3, -0.2])
    mp = mq + shift * np.array([0.6, 0.8]) * s
    delta = (mp - mq) / s
    e = delta / np.linalg.norm(delta)
    ys = np.empty((n, d))
    acc = 0
    for i in range(n):
        z = rng.standard_normal(d)
        yhat = mp + s * z
        _, _, ell = log_ratio_terms(yhat[None], mp[None], mq[None], [s])
        res = token_verify(ell, 1, [rng.uniform()])
        if res["tau"] == 2:
            ys[i] = yhat
            acc += 1
        else:
            ys[i] = reflection(delta, z, mq, s)
    zq = (ys - mq) / s
    for c in range(d):
        assert stats.kstest(zq[:, c], "norm").pvalue > 1e-3
    assert stats.kstest(zq @ e, "norm").pvalue > 1e-3
    # the acceptance of sample verification, 2 Phi(-||Delta||/2)
    p = 2.0 * stats.norm.cdf(-np.linalg.norm(delta) / 2)
    assert abs(acc / n - p) < 4.5 * math.sqrt(p * (1 - p) / n)


@pytest.mark.parametrize("d,K,N", [(1, 3, 12), (2, 4, 10)])
def test_reflection_sampler_law_matches_plain_em(d, K, N):
    g = _gmm(d, 1)
    sch = Schedule(N)
    B = 900
    spec = S.run_sampler(g, sch, B, K, seed=21, mode=S.TOKEN, residual=S.REFLECTION)["y"]
    em = S.run_plain_em(g, sch, B, seed=22)
    for i in range(d):
        assert stats.ks_2samp(spec[:, i], em[:, i]).pvalue > 1e-3


def test_reflection_rejected_with_block_verification():
    g = _gmm(1, 1)
    with pytest.raises(ValueError):
        S.run_sampler(g, Schedule(4), 2, 2, seed=1, mode=S.BLOCK, residual=S.REFLECTION)


# ------------------------------------------------------------ temperature --
def p_accept_closed_form(v, omega):
    c = 1.0 / (omega * omega)
    return stats.norm.cdf(-v / 2) + math.exp(0.5 * v * v * c * (c - 1.0)) * stats.norm.cdf(v / 2 - c * v)


@pytest.mark.parametrize("v,omega", [(0.5, 0.5), (0.5, 2.0), (2.0, 0.5), (2.0, 2.0), (1.0, 1.0)])
def test_tempered_acceptance_closed_form(v, omega):
    rng = np.random.default_rng(3)
    d, n = 3, 20000
    delta = np.zeros(d)
    delta[1] = v
    z = rng.standard_normal((n, d))
    ell = -(z @ delta) - 0.5 * v * v
    eta = rng.uniform(size=n)
    acc = np.array([token_verify([ell[i]], 1, [eta[i]], omega)["tau"] == 2 for i in range(n)])
    p = p_accept_closed_form(v, omega)
    assert abs(acc.mean() - p) < 4.5 * math.sqrt(p * (1 - p) / n)
    if omega == 1.0:
        assert p == pytest.approx(2 * stats.norm.cdf(-v / 2), rel=1e-15)


def mean_shift_quadrature(v, omega):
    """g(v, omega): the mean of e.z over one tempered round (y = m^q + sigma z).

    Drafts have e.z = u ~ N(v, 1) and are kept with probability
    min(1, exp((v^2 - 2 u v) / (2 omega^2))); a rejection draws u from
    psi_1 ∝ max(0, N(u) - N(u - v)), whose mean is -v Phi(-v/2) / (1 - 2 Phi(-v/2)).
    """
    c = 1.0 / (omega * omega)
    f = lambda u: u * stats.norm.pdf(u - v) * min(1.0, math.exp(c * (0.5 * v * v - u * v)))
    acc_mean = integrate.quad(f, v - 12, v + 12, points=[v / 2], limit=200, epsabs=1e-12)[0]
    pa = integrate.quad(lambda u: stats.norm.pdf(u - v) * min(1.0, math.exp(c * (0.5 * v * v - u * v))),
                        v - 12, v + 12, points=[v / 2], limit=200, epsabs=1e-13)[0]
    q = stats.norm.cdf(-v / 2)
    mu_res = -v * q / (1.0 - 2.0 * q)
    return acc_mean + (1.0 - pa) * mu_res, pa


@pytest.mark.parametrize("omega", [0.5, 1.0, 2.0])
def test_tempered_mean_shift(omega):
    v = 1.0
    g, pa = mean_shift_quadrature(v, omega)
    assert pa == pytest.approx(p_accept_closed_form(v, omega), abs=1e-9)
    if omega == 1.0:
        assert abs(g) < 1e-9
    elif omega > 1.0:
        assert g > 0.02
    else:
        assert g < -0.02
    rng = np.random.default_rng(4)
    d, n, s = 2, 5000, 0.6
    mq = np.array([0.1, 0.4])
    e = np.array([0.8, -0.6])
    mp = mq + s * v * e
    delta = (mp - mq) / s
    u = np.empty(n)
    for i in range(n):
        z = rng.standard_normal(d)
        yhat = mp + s * z
        _, _, ell = log_ratio_terms(yhat[None], mp[None], mq[None], [s])
        res = token_verify(ell, 1, [rng.uniform()], omega)
        if res["tau"] == 2:
            y = yhat
        else:
            U = usample(rng.uniform(), res["log_alpha_res"], v, USAMPLE_EXACT)
            y = decomposition(delta, mq, s, U, rng.standard_normal(d))
        u[i] = ((y - mq) / s) @ e
    se = u.std() / math.sqrt(n)
    assert abs(u.mean() - g) < 4.5 * se


def test_block_with_one_step_takes_sample_coins():
    rng = np.random.default_rng(5)
    for omega in (0.5, 1.0, 2.0):
        for _ in range(300):
            ell = [rng.normal(-0.5, 1.0)]
            eta = [rng.uniform()]
            rb = block_verify(ell, [rng.uniform(0.1, 2.0)], 1, eta, omega)
            rt = token_verify(ell, 1, eta, omega)
            assert rb["tau"] == rt["tau"]


def test_omega_one_changes_nothing():
    g = _gmm(2, 7)
    sch = Schedule(9)
    for mode in (S.BLOCK, S.TOKEN):
        a = S.run_sampler(g, sch, 12, 3, seed=4, mode=mode)
        b = S.run_sampler(g, sch, 12, 3, seed=4, mode=mode, omega=1.0)
        assert np.array_equal(a["y"], b["y"])
        # (most rounds here reject the first draft, where omega has no effect)
        c = S.run_sampler(g, sch, 12, 3, seed=4, mode=mode, omega=0.3)
        assert not np.array_equal(a["y"], c["y"])


def test_block_efficiency_grows_with_omega():
    g = _gmm(1, 2)
    sch = Schedule(20)
    be = [S.block_efficiency(S.run_sampler(g, sch, 150, 4, seed=3, mode=S.BLOCK, omega=w)["trace"])
          for w in (0.5, 1.0, 2.0)]
    assert be[0] < be[1] < be[2]


# ---------------------------------------------------------- frozen drafter --
@pytest.mark.parametrize("mode", [S.BLOCK, S.TOKEN])
def test_frozen_first_draft_is_target_mean(mode):
    g = _gmm(2, 4)
    sch = Schedule(15)
    res = S.run_sampler(g, sch, 30, 4, seed=5, mode=mode, drafter=S.FROZEN, keep_trace=True)
    for rec in res["trace"]:
        assert sum(info["steps"] for info in rec) == sch.n_steps
        for info in rec:
            assert info["nrm2"][0] == 0.0
            assert info["tau"] >= 2


@pytest.mark.parametrize("N", [7, 8])
def test_frozen_k1_is_plain_em_path(N):
    g = _gmm(3, 8)
    sch = Schedule(N)
    seed, B = 13, 5
    res = S.run_sampler(g, sch, B, 1, seed=seed, drafter=S.FROZEN)
    for b in range(B):
        y = philox.normal_vector(seed, b, 0, philox.TAG_INIT, 0, g.d)
        k, r = 0, 0
        while k < N:
            mq, _ = target_mean(g, sch, y, k)
            y = mq[0] + sch.sigma(k) * philox.normal_vector(seed, b, r, philox.TAG_DRAFT, 1, g.d)
            k += 1
            if k < N:
                mq, _ = target_mean(g, sch, y, k)
                y = mq[0] + sch.sigma(k) * philox.normal_vector(seed, b, r, philox.TAG_TARGET, 0, g.d)
                k += 1
            r += 1
        np.testing.assert_allclose(res["y"][b], y, rtol=1e-12, atol=1e-12)
        assert res["rounds"][b] == (N + 1) // 2


@pytest.mark.parametrize("mode,d,K,N", [(S.BLOCK, 1, 3, 12), (S.TOKEN, 2, 4, 10)])
def test_frozen_sampler_law_matches_plain_em(mode, d, K, N):
    g = _gmm(d, 1)
    sch = Schedule(N)
    B = 900
    spec = S.run_sampler(g, sch, B, K, seed=31, mode=mode, drafter=S.FROZEN)["y"]
    em = S.run_plain_em(g, sch, B, seed=32)
    for i in range(d):
        assert stats.ks_2samp(spec[:, i], em[:, i]).pvalue > 1e-3
