"""Closed-form Gaussian-mixture target: score and EM mean m^q.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Data law q_data = sum_m w_m N(mu_m, v_m I) in R^d.  Under the VP forward
process X_s = a X_0 + sqrt(1 - a^2) eps (a = a(s), see schedule.py) the
marginal is again a mixture,
    q_s(x) = sum_m w_m N(x; a mu_m, s2_m I),   s2_m = a^2 v_m + 1 - a^2,
so the Stein score s_s(x) = grad log q_s(x) of the paper's Sec. 2 is
    s_s(x) = sum_m r_m(x) (a mu_m - x) / s2_m,
    r_m(x) = softmax_m( log w_m - (d/2) log s2_m - ||x - a mu_m||^2 / (2 s2_m) ).
The target EM mean is m^q_n(x) = c1_n x + c2_n s_{1-t_n}(x)
(eq. target-distribution).

Squared distances ||x - a mu_m||^2: for d <= 64 formed from the differences,
one mixture component at a time; above that from the float64 expansion
||x||^2 - 2 a x.mu_m + a^2 ||mu_m||^2 (one matrix product over all components),
which is checked against the direct differences on a subset of rows.

Parity: pinned by the single-component reduction, a finite-difference
gradient of log q_s, Monte Carlo moments of the forward marginal, and the
expansion against direct distances.
"""
import numpy as np


DIRECT_MAX_D = 64   # above this dimension the squared distances use the expansion


class GMM:
    def __init__(self, mu, var, log_w):
        self.mu = np.asarray(mu, dtype=np.float64)          # [M, d]
        self.var = np.asarray(var, dtype=np.float64)        # [M]
        self.log_w = np.asarray(log_w, dtype=np.float64)    # [M]
        self.M, self.d = self.mu.shape
        self._mu2 = None

    def sq_dist(self, x, a, direct=None):
        """||x_r - a_r mu_m||^2 for rows x [R, d], signal levels a [R]: [R, M]."""
        if direct is None:
            direct = self.d <= DIRECT_MAX_D
        if direct:
            out = np.empty((x.shape[0], self.M))
            for m in range(self.M):
                diff = x - a[:, None] * self.mu[m][None, :]
                out[:, m] = np.sum(diff * diff, axis=1)
            return out
        if self._mu2 is None:
            self._mu2 = np.sum(self.mu * self.mu, axis=1)
        return (np.sum(x * x, axis=1)[:, None] - 2.0 * a[:, None] * (x @ self.mu.T)
                + (a * a)[:, None] * self._mu2[None, :])

    def log_density(self, x, a):
        """log q_s(x) for rows x [R, d] at signal level a (scalar or [R])."""
        x = np.atleast_2d(np.asarray(x, dtype=np.float64))
        a = np.broadcast_to(np.asarray(a, dtype=np.float64), (x.shape[0],))
        s2 = (a * a)[:, None] * self.var[None, :] + 1.0 - (a * a)[:, None]
        comp = (self.log_w[None, :] - 0.5 * self.d * np.log(2.0 * np.pi * s2)
                - self.sq_dist(x, a) / (2.0 * s2))
        mx = comp.max(axis=1, keepdims=True)
        return (mx + np.log(np.sum(np.exp(comp - mx), axis=1, keepdims=True)))[:, 0]

    def responsibilities(self, x, a, direct=None):
        x = np.atleast_2d(np.asarray(x, dtype=np.float64))
        a = np.broadcast_to(np.asarray(a, dtype=np.float64), (x.shape[0],))
        s2 = (a * a)[:, None] * self.var[None, :] + 1.0 - (a * a)[:, None]
        logit = (self.log_w[None, :] - 0.5 * self.d * np.log(s2)
                 - self.sq_dist(x, a, direct) / (2.0 * s2))
        logit -= logit.max(axis=1, keepdims=True)
        r = np.exp(logit)
        return r / r.sum(axis=1, keepdims=True)

    def score(self, x, a, direct=None):
        """s_s(x) for rows x [R, d] at signal level a (scalar or [R]).

        sum_m r_m (a mu_m - x) / s2_m: per component for d <= 64, else as the
        product (r a / s2) mu minus x sum_m r_m / s2_m.
        """
        x = np.atleast_2d(np.asarray(x, dtype=np.float64))
        a = np.broadcast_to(np.asarray(a, dtype=np.float64), (x.shape[0],))
        if direct is None:
            direct = self.d <= DIRECT_MAX_D
        r = self.responsibilities(x, a, direct)
        s2 = (a * a)[:, None] * self.var[None, :] + 1.0 - (a * a)[:, None]
        w = r / s2
        if not direct:
            return (w * a[:, None]) @ self.mu - np.sum(w, axis=1)[:, None] * x
        out = np.zeros_like(x)
        for m in range(self.M):
            out += w[:, m][:, None] * (a[:, None] * self.mu[m][None, :] - x)
        return out


def target_mean(gmm, sched, x, n):
    """m^q_n(x) and the score it uses, for rows x [R, d] at steps n (int or [R])."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    n = np.broadcast_to(np.asarray(n), (x.shape[0],))
    sc = gmm.score(x, sched.signal(n))
    mq = sched.c1(n)[:, None] * x + sched.c2(n)[:, None] * sc
    return mq, sc
