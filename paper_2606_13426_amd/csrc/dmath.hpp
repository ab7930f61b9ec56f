// Float64 normal-CDF primitives for the acceptance scan and U-sampling,
// written in log space as App. A.2 of the paper recommends.
//
// Every function here takes one instruction path for every argument: the
// U-sampler evaluates them on all 64 lanes of a wavefront at points that
// span many orders of magnitude, and a branch on the argument would make the
// wavefront execute every side of it.  Case distinctions are selects between
// values computed on all lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

#include "erfcx_table.hpp"

namespace sd {

constexpr double kSqrt1_2 = 0.70710678118654752440;
constexpr double kInvSqrtPi = 0.56418958354775628695;

// erfcx(y) = e^{y^2} erfc(y) for y >= 0 by Weideman's rational approximation
// (SIAM J. Numer. Anal. 31 (1994)): with Z = (L - y)/(L + y),
//   erfcx(y) = 2 p(Z)/(L + y)^2 + 1/(sqrt(pi) (L + y)),
// p of degree N - 1 (N = 40, coefficients in erfcx_table.hpp; relative error
// below 1e-15 on y >= 0, and y -> infinity gives the 1/(sqrt(pi) y) tail).
__device__ inline double erfcx_pos(double y) {
  const double inv = 1.0 / (kWeidemanL + y);
  const double z = (kWeidemanL - y) * inv;
  double p = kWeidemanA[0];
#pragma unroll
  for (int n = 1; n < kWeidemanN; ++n) p = fma(p, z, kWeidemanA[n]);
  return fma(2.0 * p, inv, kInvSqrtPi) * inv;
}

// log(1 - e^r) for r < 0 as log(-expm1(r)): exact to rounding near 0, and an
// absolute error of about e^r (harmless in sums of logs) far below it.
__device__ inline double log1mexp(double r) { return log(-expm1(r)); }

__device__ inline double logaddexp(double a, double b) {
  const double m = fmax(a, b);
  if (m == -INFINITY) return -INFINITY;
  return m + log(exp(a - m) + exp(b - m));
}

// log(alpha Phi(x) - Phi(x - v)) for x <= u* = log(alpha)/v + v/2, v > 0
// (the mass below x of the unnormalised residual law, Alg. 7), from
// e1 = erfcx(|x|/sqrt 2) and e2 = erfcx((v - x)/sqrt 2) (v - x >= v/2 > 0):
//   log Phi(x)     = log(e1/2) - x^2/2             for x <= 0,
//                  = log1p(-(e1/2) e^{-x^2/2})     for x > 0,
//   log Phi(x - v) = log(e2/2) - (x - v)^2/2,
// and the log-ratio r = log Phi(x - v) - log Phi(x) - log alpha, which for
// x <= 0 is log(e2/e1) + v (x - u*): the quadratic terms cancel exactly, so r
// keeps its digits far into the left tail where both log-CDFs are ~ -x^2/2.
// The result is log alpha + log Phi(x) + log(1 - e^r).
__device__ inline double log_excess(double x, double la, double v) {
  const double us = la / v + 0.5 * v;
  const double e1 = erfcx_pos(fabs(x) * kSqrt1_2);
  const double e2 = erfcx_pos((v - x) * kSqrt1_2);
  const double l1 = log(0.5 * e1), l2 = log(0.5 * e2);
  const double hx2 = 0.5 * x * x;
  const double right = log1p(-0.5 * e1 * exp(-hx2));
  const bool left = x <= 0.0;
  const double lphi = left ? l1 - hx2 : right;
  const double xv = x - v;
  const double r = left ? (l2 - l1) + v * (x - us) : (l2 - 0.5 * xv * xv) - lphi - la;
  return la + lphi + log1mexp(fmin(r, -0.0));
}

// log h_j of block verification for j < K_b from log alpha_j and
// ||Delta_{j+1}||: h = v/(v + 1 - alpha), v = alpha Phi(u*) - Phi(u* - ||D||).
// alpha = 1 gives h = 1; ||Delta_{j+1}|| = 0 with alpha < 1 gives h = 0.
__device__ inline double block_log_h(double la, double vnext) {
  const bool pos = vnext > 0.0;
  const double vs = pos ? vnext : 1.0;
  const double lv = log_excess(la / vs + 0.5 * vs, la, vs);
  const double lh = lv - logaddexp(lv, log1mexp(fmin(la, -0.0)));
  return la >= 0.0 ? 0.0 : pos ? lh : -INFINITY;
}

}  // namespace sd
