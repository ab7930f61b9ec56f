"""Residual distribution r(y; alpha) ∝ max(0, alpha q(y) - p(y)) and its sampler.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Prop. 1 (eq. decomp): with p = N(m^p, s^2 I), q = N(m^q, s^2 I),
Delta = (m^p - m^q)/s, e = Delta/||Delta||, the residual is sampled as
    U ~ psi_alpha,  Z_perp ~ N(0, I - e e^T),  Y = m^q + s (U e + Z_perp),
where psi_alpha(u) ∝ max(0, alpha N(u) - N(u - v)), v = ||Delta||, with CDF
(eq. u-cdf)
    Psi_alpha(u) = (alpha Phi(u) - Phi(u - v)) / (alpha Phi(u*) - Phi(u* - v)),  u < u*,
    Psi_alpha(u) = 1 otherwise,       u* = log(alpha)/v + v/2.
Alg. 5 draws Z_perp as G - e (e^T G) with G ~ N(0, I).

U is drawn by inverting Psi (Alg. 7, App. A.1): u ~ U(0,1); bracket
[u* - 1, u*]; while Psi(lower) > u the lower end is pushed down by doubling
the bracket width; then bisection on Psi(mid) < u.  Two stopping readings:
  * exact: no cap on the doubling beyond 64 steps; bisect until the midpoint
    equals an end of the bracket in float64 (the bracket has collapsed);
  * paper: at most 3 doublings and 4 bisection steps with tolerance
    |Psi(mid) - u| <= 1e-6 (the caps of the paper's experiments, App. I;
    the tolerance value is not given there and 1e-6 is this reading).
Psi is evaluated in log space: log(alpha Phi(x) - Phi(x - v))
= log alpha + log Phi(x) + log(1 - exp(log Phi(x - v) - log Phi(x) - log alpha)),
with the log-CDF difference taken through erfcx in the left tail (App. A.2 asks
for stable log-space primitives; the plain difference loses all digits there).

The reflection residual (Alg. 4) of sample verification is here too:
Y = m^q + sigma (I - 2 e e^T) Z with Z the rejected step's draft noise.

Parity: pinned by trapezoid integration of the unnormalised density (the
paper's own numerical method for its residual plots), KS tests of sampled
U against Psi, exactness of the sampled residual in d = 1, 2, 8, and, for the
paper mode, the dyadic midpoint that the exact inverse determines (the caps
and the tolerance stop included).
"""
import math

import numpy as np

from . import philox
from .verify import log_excess

USAMPLE_EXACT = 0
USAMPLE_PAPER = 1
PAPER_TOL = 1e-6


def upper_end(log_alpha, v):
    """u* = log(alpha)/v + v/2, the right end of the support of psi_alpha (Cor. non-zero-res)."""
    return log_alpha / v + 0.5 * v


def log_mass_below(x, log_alpha, v):
    """log(alpha Phi(x) - Phi(x - v)) for x <= u* (see verify.log_excess for the tail form)."""
    return log_excess(x, log_alpha, v)


def log_cdf(x, log_alpha, v):
    """log Psi_alpha(x) (eq. u-cdf)."""
    us = upper_end(log_alpha, v)
    if x >= us:
        return 0.0
    return log_mass_below(x, log_alpha, v) - log_mass_below(us, log_alpha, v)


def usample(u, log_alpha, v, mode=USAMPLE_EXACT):
    """Alg. 7: invert Psi_alpha at the uniform u by doubling + bisection."""
    logu = math.log(u)
    hi = upper_end(log_alpha, v)
    lo = hi - 1.0
    max_double = 64 if mode == USAMPLE_EXACT else 3
    n = 0
    while n < max_double and log_cdf(lo, log_alpha, v) > logu:
        lo = hi - 2.0 * (hi - lo)
        n += 1
    if mode == USAMPLE_EXACT:
        mid = 0.5 * (lo + hi)
        for _ in range(200):
            mid = 0.5 * (lo + hi)
            if mid == lo or mid == hi:
                break
            if log_cdf(mid, log_alpha, v) < logu:
                lo = mid
            else:
                hi = mid
        return mid
    mid = 0.5 * (lo + hi)
    n = 0
    while n < 4:
        lc = log_cdf(mid, log_alpha, v)
        if abs(math.exp(lc) - u) <= PAPER_TOL:
            break
        if lc < logu:
            lo = mid
        else:
            hi = mid
        mid = 0.5 * (lo + hi)
        n += 1
    return mid


def decomposition(delta, mq, sigma, U, G):
    """Alg. 5 given U and G: Y = m^q + sigma (U e + G - e (e^T G)), e = Delta/||Delta||."""
    delta = np.asarray(delta, dtype=np.float64)
    e = delta / np.linalg.norm(delta)
    G = np.asarray(G, dtype=np.float64)
    z_perp = G - e * np.dot(e, G)
    return np.asarray(mq, dtype=np.float64) + sigma * (U * e + z_perp)


def reflection(delta, z, mq, sigma):
    """Alg. 4 (the reflection residual of sample verification): e = Delta/||Delta||,
    Z_r = (I - 2 e e^T) Z, Y = m^q + sigma Z_r, with Z the draft noise of the
    rejected step.  It takes no alpha: it is exact with sample (token)
    verification only (Sec. 4's impossibility result rules it out for blocks)."""
    delta = np.asarray(delta, dtype=np.float64)
    e = delta / np.linalg.norm(delta)
    z = np.asarray(z, dtype=np.float64)
    z_r = z - 2.0 * e * np.dot(e, z)
    return np.asarray(mq, dtype=np.float64) + sigma * z_r


def usample_uniform(seed, chain, rnd):
    """The uniform u of Alg. 7: number 0 of the (chain, round, USAMPLE) stream."""
    return philox.uniform_at(seed, chain, rnd, philox.TAG_USAMPLE, 0, 0)


def resid_noise(seed, chain, rnd, d):
    """G of Alg. 5: the (chain, round, RESID) normal vector."""
    return philox.normal_vector(seed, chain, rnd, philox.TAG_RESID, 0, d)
