"""Draft verification: token (Alg. 2) and block (Alg. 6) verification.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Per draft step j = 1..K_b (paper Alg. 2 / Alg. 6):
    Delta_j = (m^p_{k+j-1} - m^q_{k+j-1}) / sigma_{k+j-1}
    Z_j     = (yhat_{k+j} - m^p_{k+j-1}) / sigma_{k+j-1}
and, in log space (App. A.2),
    log N(Z_j + Delta_j) / N(Z_j) = -Z_j^T Delta_j - ||Delta_j||^2 / 2 =: ell_j.

Token verification (Alg. 2): alpha_j = min(1, e^{ell_j}), independent coins
c_j = [eta_j < alpha_j], tau = first j with c_j = 0 (K_b + 1 if none),
alpha_res = 1.

Block verification (Alg. 6): log alpha_0 = 0,
    log alpha_j = min(0, log alpha_{j-1} + ell_j)                 (App. A.2)
    h_j = v_j / (v_j + 1 - alpha_j)  for j < K_b,  h_{K_b} = alpha_{K_b},
    v_j = alpha_j Phi(log alpha_j/||Delta_{j+1}|| + ||Delta_{j+1}||/2)
          - Phi(log alpha_j/||Delta_{j+1}|| - ||Delta_{j+1}||/2),
coins c_j = [eta_j < h_j], c_0 = 1, tau = 1 + max{j : c_j = 1},
alpha_res = alpha_{tau-1}.  v_j is evaluated with log-CDF primitives and a
stable log(1 - e^x) as App. A.2 recommends.

Temperature (App. "Temperature", the tempered sample and block verification
algorithms): with p, q given the covariance omega^2 I the log ratio becomes
ell_j / omega^2, so both recursions above take ell_j / omega^2 in place of
ell_j; h_j keeps the untempered ||Delta_{j+1}||, and alpha_res (block) is the
tempered alpha_{tau-1}.  omega = 1 is the exact method; omega != 1 is lossy.

Readings where the paper is silent (listed in the design notes):
  * alpha_j = 1 gives h_j = 1 (the 0/0 limit v/(v + 0) with v > 0, and the
    value the block acceptance takes when nothing has been lost yet);
  * ||Delta_{j+1}|| = 0 with alpha_j < 1 gives v_j = 0, hence h_j = 0;
  * the coin is strict, eta < h, and compared in log space, log eta < log h,
    in float64;
  * eta_j is uniform number j-1 of the (chain, round, COIN) Philox stream.

Parity: pinned by the token-acceptance closed form 2 Phi(-||Delta||/2),
the closed-form acceptance lemma, quadrature of int max(0, alpha q - p) for
h_j, and the exactness of one verification round (tests/test_oracle_verify.py).
"""
import math

import numpy as np
from scipy.special import erfcx, log_ndtr

from . import philox

LN2 = math.log(2.0)


def log1mexp(x):
    """log(1 - e^x) for x <= 0 (Maechler 2012: expm1 branch above -ln 2, log1p below)."""
    if x >= 0.0:
        return -math.inf
    if x > -LN2:
        return math.log(-math.expm1(x))
    return math.log1p(-math.exp(x))


def logaddexp(a, b):
    if a == -math.inf:
        return b
    if b == -math.inf:
        return a
    m = max(a, b)
    return m + math.log(math.exp(a - m) + math.exp(b - m))


def log_ratio_terms(y_draft, mp, mq, sigma):
    """||Delta_j||^2, Z_j^T Delta_j and ell_j for arrays [..., K, d] and sigma [..., K]."""
    y_draft = np.asarray(y_draft, dtype=np.float64)
    mp = np.asarray(mp, dtype=np.float64)
    mq = np.asarray(mq, dtype=np.float64)
    sigma = np.asarray(sigma, dtype=np.float64)[..., None]
    delta = (mp - mq) / sigma
    z = (y_draft - mp) / sigma
    nrm2 = np.sum(delta * delta, axis=-1)
    dot = np.sum(z * delta, axis=-1)
    return nrm2, dot, -dot - 0.5 * nrm2


SQRT1_2 = math.sqrt(0.5)


def log_ratio_below(x, log_alpha, v):
    """log(Phi(x - v) / (alpha Phi(x))) for v > 0.

    For x < 0 both log-CDFs are about -x^2/2 and their difference cancels
    catastrophically far in the tail; with Phi(y) = erfcx(-y/sqrt 2) e^{-y^2/2} / 2
    the quadratic terms cancel exactly and the ratio is
        log erfcx(-(x - v)/sqrt 2) - log erfcx(-x/sqrt 2) + v (x - u*),
    u* = log(alpha)/v + v/2.  Elsewhere the log-CDFs are subtracted directly.
    """
    if x < 0.0:
        us = log_alpha / v + 0.5 * v
        return (math.log(float(erfcx(-(x - v) * SQRT1_2))) - math.log(float(erfcx(-x * SQRT1_2)))
                + v * (x - us))
    return float(log_ndtr(x - v)) - float(log_ndtr(x)) - log_alpha


def log_excess(x, log_alpha, v):
    """log(alpha Phi(x) - Phi(x - v)) for x <= u* = log(alpha)/v + v/2, v > 0."""
    return log_alpha + float(log_ndtr(x)) + log1mexp(min(0.0, log_ratio_below(x, log_alpha, v)))


def log_v(log_alpha, vnorm):
    """log of alpha Phi(log alpha/v + v/2) - Phi(log alpha/v - v/2), v = ||Delta|| > 0."""
    return log_excess(log_alpha / vnorm + 0.5 * vnorm, log_alpha, vnorm)


def block_log_h(log_alpha, vnorm_next):
    """log h_j of Alg. 6 for j < K_b, from log alpha_j and ||Delta_{j+1}||."""
    if log_alpha >= 0.0:
        return 0.0
    if vnorm_next <= 0.0:
        return -math.inf
    lv = log_v(log_alpha, vnorm_next)
    return lv - logaddexp(lv, log1mexp(log_alpha))


def coin_uniforms(seed, chain, rnd, K):
    """eta_1..eta_K: uniform j-1 of the (chain, round, COIN) stream."""
    return np.array([philox.uniform_at(seed, chain, rnd, philox.TAG_COIN, 0, j) for j in range(K)])


def block_verify(ell, nrm2, kb, eta, omega=1.0):
    """Alg. 6 for one chain (with temperature omega: the tempered block verification).

    ell, nrm2: [>= kb] per-step ell_j and ||Delta_j||^2 (index j-1); eta: [>= kb].
    Returns dict(tau, log_alpha_res, log_alpha[kb], log_h[kb], coins[kb]).
    """
    w2 = float(omega) * float(omega)
    log_alpha = np.empty(kb)
    acc = 0.0
    for j in range(kb):
        acc = min(0.0, acc + float(ell[j]) / w2)
        log_alpha[j] = acc
    log_h = np.empty(kb)
    for j in range(kb):
        if j + 1 < kb:
            log_h[j] = block_log_h(log_alpha[j], math.sqrt(float(nrm2[j + 1])))
        else:
            log_h[j] = log_alpha[j]
    coins = np.array([math.log(float(eta[j])) < log_h[j] for j in range(kb)])
    accepted = [j + 1 for j in range(kb) if coins[j]]
    last = max(accepted) if accepted else 0
    tau = 1 + last
    log_alpha_res = 0.0 if tau == 1 else float(log_alpha[tau - 2])
    return dict(tau=tau, log_alpha_res=log_alpha_res, log_alpha=log_alpha,
                log_h=log_h, coins=coins)


def token_verify(ell, kb, eta, omega=1.0):
    """Alg. 2 for one chain: independent coins against min(1, ratio) (the
    ratio of the omega^2-covariance densities with temperature omega)."""
    w2 = float(omega) * float(omega)
    log_a = np.array([min(0.0, float(ell[j]) / w2) for j in range(kb)])
    coins = np.array([math.log(float(eta[j])) < log_a[j] for j in range(kb)])
    tau = kb + 1
    for j in range(kb):
        if not coins[j]:
            tau = j + 1
            break
    return dict(tau=tau, log_alpha_res=0.0, log_alpha=log_a, log_h=log_a, coins=coins)


def ties(res, eta, window=1e-6):
    """Steps j whose coin lies within `window` of its threshold (|eta_j - h_j|)."""
    h = np.exp(res["log_h"])
    return [j + 1 for j in range(len(h)) if abs(float(eta[j]) - h[j]) <= window]
