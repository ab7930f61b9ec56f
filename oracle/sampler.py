"""Speculative diffusion sampling with block (or token) verification.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Follows the full algorithm of App. B (Alg. 8) chain by chain, with the
Free Drafter of Sec. 3.3 as the drafter:

  Y_0 ~ N(0, I) (INIT stream); the target is called once explicitly at Y_0 to
  seed the cached score S_c (the only explicit call, Sec. 3.3).
  Each round, with K_b = min(K, N - k):
    draft   yhat_0 = Y_k; for i = 1..K_b, n = k + i - 1:
              m^p_{i-1} = c1_n yhat_{i-1} + c2_n S_c          (eq. frozen-draft-drift
              yhat_i    = m^p_{i-1} + sigma_n xi_i               with the cached score)
    target  m^q_{j} = m^q_{k+j}(yhat_j) for j = 0..min(K_b + 1, N - k) - 1
    verify  tau, alpha_res from Alg. 6 (block) or Alg. 2 (token)
    resid   k + tau <= N:  tau = K_b + 1 -> Y = m^q_{K_b} + sigma_{k+K_b} xi'   (TARGET stream)
                           else -> Decomposition with alpha = alpha_res          (Alg. 5 + 7)
            k + tau > N:   Y_N = yhat_{K_b}
    cache   the Free Drafter keeps the target score of the rejected draft
            yhat_tau (tau <= K_b) or of yhat_{K_b} after a full accept
            (the score that produced the extra sample)
    commit  k <- min(k + tau, N), round <- round + 1.

Variants (the paper's alternatives to the defaults above):
  * residual REFLECTION (Alg. 4, sample verification only): a rejection at
    tau gives Y = m^q_{tau-1} + sigma (I - 2 e e^T) Z_tau, Z_tau the draft
    noise of the rejected step, e = Delta_tau/||Delta_tau||;
  * drafter FROZEN (Sec. 3.3, eq. frozen-draft-drift): each round first calls
    the target at (Y_k, k) and drafts with that score, S_c = s(Y_k, k);
  * temperature omega (App. "Temperature"): the verification takes
    ell_j / omega^2 (see verify.py); the residual keeps the untempered Delta
    and, for block verification, the tempered alpha_res.  Lossy for omega != 1.

Also the plain Euler-Maruyama chain Y_{n+1} = m^q_n(Y_n) + sigma_n xi_n,
whose law the speculative sampler must reproduce exactly (Sec. 2/3.2).

Parity: the exact numeric trajectories are fixed only by this oracle and the
shared Philox contract ("parity unpinned" for single trajectories); their law
is pinned by the distribution tests against the plain EM chain and the
degenerate drafter = target case, and the Free Drafter's cache row by finite
differences of log q at the rejected (or last) draft and its time.  The variants are pinned the same way
(tests/test_oracle_variants.py): the reflection and Frozen-Drafter samplers
against the plain EM law, the Frozen Drafter with K = 1 path by path against
an EM chain with the round's noises, temperature by the closed-form tempered
acceptance and the quadrature of the temperature proposition's mean shift.
"""
import math

import numpy as np

from . import philox
from .gmm import target_mean
from .residual import (USAMPLE_EXACT, decomposition, reflection, resid_noise,
                       usample, usample_uniform)
from .verify import (block_verify, coin_uniforms, log_ratio_terms, ties,
                     token_verify)

BLOCK = 0
TOKEN = 1
DECOMPOSITION = 0
REFLECTION = 1
FREE = 0
FROZEN = 1


def verify_chain(y_draft, mp, mq, sigma, kb, seed, chain, rnd, mode=BLOCK,
                 usample_mode=USAMPLE_EXACT, omega=1.0):
    """One chain's verification (Alg. 6 or Alg. 2, tempered by omega) plus its U draw (Alg. 7).

    y_draft, mp, mq: [>= kb, d] rows j-1 = yhat_{k+j}, m^p_{k+j-1}, m^q_{k+j-1};
    sigma: [>= kb] sigma_{k+j-1}.
    """
    nrm2, dot, ell = log_ratio_terms(y_draft[:kb], mp[:kb], mq[:kb], sigma[:kb])
    eta = coin_uniforms(seed, chain, rnd, kb)
    if mode == BLOCK:
        res = block_verify(ell, nrm2, kb, eta, omega)
    else:
        res = token_verify(ell, kb, eta, omega)
    tau = res["tau"]
    U = float("nan")
    if tau <= kb:
        u = usample_uniform(seed, chain, rnd)
        U = usample(u, res["log_alpha_res"], math.sqrt(float(nrm2[tau - 1])), usample_mode)
    res.update(nrm2=nrm2, dot=dot, ell=ell, eta=eta, U=U, ties=ties(res, eta))
    return res


def residual_chain(y_draft, mp, mq, sigma, kb, tau, U, steps_left, seed, chain, rnd,
                   residual=DECOMPOSITION):
    """The new state Y_{k+tau} of one chain (the residual part of Alg. 8).

    y_draft: [>= kb, d] drafts yhat_{k+1..}; mp: [>= kb, d]; mq: [>= kb+1, d]
    (row kb used only by the full-accept target draw); sigma: [>= kb+1].
    residual: DECOMPOSITION (Alg. 5 with U) or REFLECTION (Alg. 4, U unused).
    """
    d = np.asarray(mq).shape[-1]
    if tau <= kb:
        mp_t = np.asarray(mp[tau - 1], np.float64)
        delta = (mp_t - np.asarray(mq[tau - 1], np.float64)) / sigma[tau - 1]
        if residual == REFLECTION:
            z = (np.asarray(y_draft[tau - 1], np.float64) - mp_t) / sigma[tau - 1]
            return reflection(delta, z, mq[tau - 1], sigma[tau - 1])
        G = resid_noise(seed, chain, rnd, d)
        return decomposition(delta, mq[tau - 1], sigma[tau - 1], U, G)
    if kb + 1 <= steps_left:
        xi = philox.normal_vector(seed, chain, rnd, philox.TAG_TARGET, 0, d)
        return np.asarray(mq[kb], np.float64) + sigma[kb] * xi
    return np.asarray(y_draft[kb - 1], np.float64)


def draft_chain(y, score_c, k, kb, sched, seed, chain, rnd):
    """Free-Drafter block: drafts yhat_{k..k+kb} [kb+1, d] and means m^p [kb, d]."""
    d = y.shape[0]
    yh = np.empty((kb + 1, d))
    mp = np.empty((kb, d))
    yh[0] = y
    for i in range(1, kb + 1):
        n = k + i - 1
        mp[i - 1] = sched.c1(n) * yh[i - 1] + sched.c2(n) * score_c
        xi = philox.normal_vector(seed, chain, rnd, philox.TAG_DRAFT, i, d)
        yh[i] = mp[i - 1] + sched.sigma(n) * xi
    return yh, mp


def init_state(gmm, sched, seed, chain):
    """Y_0 ~ N(0, I) and the explicit first target call that seeds the cache."""
    y = philox.normal_vector(seed, chain, 0, philox.TAG_INIT, 0, gmm.d)
    _, sc = target_mean(gmm, sched, y, 0)
    return y, sc[0]


def check_options(mode, residual, drafter, omega):
    if mode not in (BLOCK, TOKEN) or residual not in (DECOMPOSITION, REFLECTION):
        raise ValueError("unknown verification mode or residual")
    if drafter not in (FREE, FROZEN):
        raise ValueError("unknown drafter")
    if residual == REFLECTION and mode != TOKEN:
        raise ValueError("the reflection residual is valid with sample (token) verification only")
    if not (omega > 0.0 and math.isfinite(omega)):
        raise ValueError("the temperature must be positive and finite")


def run_round(gmm, sched, K, y, score_c, k, rnd, seed, chain, mode=BLOCK,
              usample_mode=USAMPLE_EXACT, residual=DECOMPOSITION, drafter=FREE, omega=1.0):
    """One round of Alg. 8 for one chain; returns (y, score_c, k, info)."""
    N = sched.n_steps
    kb = min(K, N - k)
    if drafter == FROZEN:
        # the Frozen Drafter's one target call of the round, at the state itself
        _, s0 = target_mean(gmm, sched, y, k)
        score_c = s0[0]
    yh, mp = draft_chain(y, score_c, k, kb, sched, seed, chain, rnd)
    nrows = min(kb + 1, N - k)
    mq, sc = target_mean(gmm, sched, yh[:nrows], k + np.arange(nrows))
    sig = sched.sigma(k + np.arange(kb + 1))
    v = verify_chain(yh[1:], mp, mq, sig, kb, seed, chain, rnd, mode, usample_mode, omega)
    tau = v["tau"]
    y_new = residual_chain(yh[1:], mp, mq, sig, kb, tau, v["U"], N - k, seed, chain, rnd,
                           residual)
    k_new = min(k + tau, N)
    if k_new < N:
        score_c = sc[min(tau, kb)]
    info = dict(k=k, kb=kb, tau=tau, steps=k_new - k, U=v["U"],
                log_alpha_res=v["log_alpha_res"], log_h=v["log_h"], eta=v["eta"],
                ties=v["ties"], ell=v["ell"], nrm2=v["nrm2"], yh=yh, mp=mp, mq=mq)
    return y_new, score_c, k_new, info


def run_sampler(gmm, sched, B, K, seed, mode=BLOCK, usample_mode=USAMPLE_EXACT,
                chains=None, keep_trace=False, residual=DECOMPOSITION, drafter=FREE,
                omega=1.0):
    """Alg. 8 for chains `chains` (default 0..B-1). Returns final states and per-round records."""
    check_options(mode, residual, drafter, omega)
    chains = list(range(B)) if chains is None else list(chains)
    ys, rounds, trace = [], [], []
    for b in chains:
        y, sc = init_state(gmm, sched, seed, b)
        k, r, rec = 0, 0, []
        while k < sched.n_steps:
            y, sc, k, info = run_round(gmm, sched, K, y, sc, k, r, seed, b, mode, usample_mode,
                                       residual, drafter, omega)
            if not keep_trace:
                for key in ("yh", "mp", "mq"):
                    info.pop(key)
            rec.append(info)
            r += 1
        ys.append(y)
        rounds.append(r)
        trace.append(rec)
    return dict(y=np.array(ys), rounds=np.array(rounds), trace=trace, chains=chains)


def block_efficiency(trace):
    """Pooled steps advanced per round over all chains (the paper's BE)."""
    steps = sum(info["steps"] for rec in trace for info in rec)
    rounds = sum(len(rec) for rec in trace)
    return steps / rounds


def run_plain_em(gmm, sched, B, seed):
    """Plain Euler-Maruyama chain from Y_0 ~ N(0, I): the law to reproduce."""
    d = gmm.d
    y = np.stack([philox.normal_vector(seed, b, 0, philox.TAG_INIT, 0, d) for b in range(B)])
    for n in range(sched.n_steps):
        mq, _ = target_mean(gmm, sched, y, n)
        xi = np.stack([philox.normal_vector(seed, b, n, philox.TAG_TARGET, 1, d) for b in range(B)])
        y = mq + sched.sigma(n) * xi
    return y
