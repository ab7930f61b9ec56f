"""VP-SDE coefficients of the Euler-Maruyama chain.

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

Paper Sec. 2 (eqs. forward-process, backward-process, target-distribution):
  forward   dX_t = f_t X_t dt + g_t dB_t with q_1 ~ N(0, I);
  generative dY_t = b_t(Y_t) dt + eps g_{1-t} dW_t with
            b_t(x) = -f_{1-t} x + (1 + eps^2)/2 g_{1-t}^2 s_{1-t}(x),  eps > 0;
  grid      t_n = n delta, delta = 1/N;
  EM kernel q(y'|y) = N(m^q_n(y), sigma_n^2 I), m^q_n(y) = y + delta b_{t_n}(y),
            sigma_n = sqrt(delta) eps g_{1-t_n}.

The variance-preserving instance (the reading used throughout; the paper's own
experiments use a different schedule): beta(s) = beta_min + s (beta_max - beta_min),
f_s = -beta(s)/2, g_s^2 = beta(s), and the signal level of q_s is
a(s) = sqrt(abar(s)), abar(s) = exp(-int_0^s beta) = exp(-(beta_min s + (beta_max-beta_min) s^2 / 2)).

With s_n = 1 - t_n (the forward time seen at step n) the EM mean is affine in
(y, score):  m^q_n(y) = c1_n y + c2_n s_{s_n}(y),
  c1_n = 1 + delta beta(s_n)/2,   c2_n = delta (1 + eps^2) beta(s_n)/2.

Parity: pinned by quadrature of beta (abar) and by Gaussian-data sampling
(the EM chain started from N(0, I) must end at the data variance).
"""
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Schedule:
    n_steps: int          # N, number of EM steps
    beta_min: float = 0.1
    beta_max: float = 20.0
    churn: float = 1.0    # eps > 0

    def beta(self, s):
        return self.beta_min + np.asarray(s, dtype=np.float64) * (self.beta_max - self.beta_min)

    def abar(self, s):
        s = np.asarray(s, dtype=np.float64)
        return np.exp(-(self.beta_min * s + 0.5 * (self.beta_max - self.beta_min) * s * s))

    def fwd_time(self, n):
        """Forward time 1 - t_n seen by step n."""
        return 1.0 - np.asarray(n, dtype=np.float64) / self.n_steps

    def signal(self, n):
        """a_n = sqrt(abar(1 - t_n))."""
        return np.sqrt(self.abar(self.fwd_time(n)))

    def sigma(self, n):
        """sigma_n = sqrt(delta) * eps * g_{1 - t_n}."""
        return self.churn * np.sqrt(self.beta(self.fwd_time(n)) / self.n_steps)

    def c1(self, n):
        """Coefficient of y in m^q_n (from -f = beta/2)."""
        return 1.0 + 0.5 * self.beta(self.fwd_time(n)) / self.n_steps

    def c2(self, n):
        """Coefficient of the score in m^q_n."""
        return 0.5 * (1.0 + self.churn ** 2) * self.beta(self.fwd_time(n)) / self.n_steps
