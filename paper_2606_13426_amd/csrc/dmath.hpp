// Float64 normal-CDF primitives for the acceptance scan and U-sampling,
// written in log space as App. A.2 of the paper recommends.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>

namespace sd {

constexpr double kSqrt1_2 = 0.70710678118654752440;
constexpr double kLn2 = 0.69314718055994530942;

// log Phi(x).  For x < -1 uses Phi(x) = erfcx(t) e^{-t^2} / 2, t = -x/sqrt 2,
// which stays accurate far into the left tail; otherwise log1p of the
// complementary tail.
__device__ inline double log_ndtr(double x) {
  if (x < -1.0) {
    const double t = -x * kSqrt1_2;
    return log(0.5 * erfcx(t)) - t * t;
  }
  return log1p(-0.5 * erfc(x * kSqrt1_2));
}

// log(1 - e^x), x <= 0 (Maechler 2012).
__device__ inline double log1mexp(double x) {
  if (x >= 0.0) return -INFINITY;
  return x > -kLn2 ? log(-expm1(x)) : log1p(-exp(x));
}

__device__ inline double logaddexp(double a, double b) {
  if (a == -INFINITY) return b;
  if (b == -INFINITY) return a;
  const double m = fmax(a, b);
  return m + log(exp(a - m) + exp(b - m));
}

// log(Phi(x - v) / (alpha Phi(x))), v > 0.  For x < 0 the two log-CDFs are
// ~ -x^2/2 and cancel; through erfcx the quadratic terms cancel exactly:
//   log erfcx(-(x - v)/sqrt 2) - log erfcx(-x/sqrt 2) + v (x - u*),
// u* = log(alpha)/v + v/2.
__device__ inline double log_ratio_below(double x, double la, double v) {
  if (x < 0.0) {
    const double us = la / v + 0.5 * v;
    return log(erfcx(-(x - v) * kSqrt1_2)) - log(erfcx(-x * kSqrt1_2)) + v * (x - us);
  }
  return log_ndtr(x - v) - log_ndtr(x) - la;
}

// log(alpha Phi(x) - Phi(x - v)) for x <= u*.  Below -1 both CDFs come from
// one erfcx pair: log Phi(x) = log(erfcx(t1)/2) - t1^2 and the ratio above.
__device__ inline double log_excess(double x, double la, double v) {
  if (x < -1.0) {
    const double t1 = -x * kSqrt1_2, t2 = -(x - v) * kSqrt1_2;
    const double e1 = erfcx(t1), e2 = erfcx(t2);
    const double us = la / v + 0.5 * v;
    const double r = log(e2 / e1) + v * (x - us);
    return la + log(0.5 * e1) - t1 * t1 + log1mexp(fmin(0.0, r));
  }
  return la + log_ndtr(x) + log1mexp(fmin(0.0, log_ratio_below(x, la, v)));
}

// log h_j of block verification for j < K_b from log alpha_j and
// ||Delta_{j+1}||: h = v/(v + 1 - alpha), v = alpha Phi(u*) - Phi(u* - ||D||).
// alpha = 1 gives h = 1; ||Delta_{j+1}|| = 0 with alpha < 1 gives h = 0.
__device__ inline double block_log_h(double la, double vnext) {
  if (la >= 0.0) return 0.0;
  if (!(vnext > 0.0)) return -INFINITY;
  const double lv = log_excess(la / vnext + 0.5 * vnext, la, vnext);
  return lv - logaddexp(lv, log1mexp(la));
}

}  // namespace sd
