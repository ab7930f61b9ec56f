// Verification of drafted blocks: log density ratios (App. A.2) reduced over
// d, then the block (Alg. 6) or token (Alg. 2) acceptance scan and the U draw
// of Alg. 7.
//
// logratio_kernel: one workgroup per (chain, draft row).  The three float32
// rows (draft, draft mean, target mean) are streamed once with 16-byte
// non-temporal loads; differences and products are formed in float64 and
// accumulated in float64, then reduced across the wavefront with shuffles and
// across the four wavefronts through LDS.  Pure HBM streaming: 12 B per element.
//
// scan_kernel: one wavefront per chain, lane j-1 owns draft step j (K <= 64).
// Every lane replays the prefix recursion log alpha_j = min(0, log alpha_{j-1}
// + ell_j) in the same order as the definition, evaluates its h_j, draws its
// coin, and a ballot gives tau.  U is found by inverting Psi_alpha: the
// doubling of Alg. 7 is done for all 64 candidate lower ends at once (lane i
// tests u* - 2^i), and the bisection becomes a 64-way multisection that
// shrinks the bracket 65-fold per step until it is 1e-8 (relative) wide, then
// a linear interpolation of log Psi inside it (see usample_exact).
//
// Both scans take the temperature as w2 = omega^2 (the tempered
// verifications of the appendix divide every ell_j by omega^2), and the
// sampler's scan can hand the reflection residual (Alg. 4) to the next kernel
// instead of the Decomposition residual, skipping the U draw.
#include "common.hpp"
#include "dmath.hpp"
#include "philox.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;
typedef float f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__global__ __launch_bounds__(kThreads) void logratio_kernel(
    int K, int d, const float* __restrict__ yd, int64_t yc, int64_t yr,
    const float* __restrict__ mp, int64_t pc, int64_t pr, const float* __restrict__ mq,
    int64_t qc, int64_t qr, const double* __restrict__ sigma, const int32_t* __restrict__ kb,
    double* __restrict__ dn, double* __restrict__ lr, bool vec, const int* gate) {
  if (gate && *gate == 0) return;
  const int row = blockIdx.x;
  const int b = row / K, j = row - b * K;
  if (j >= kb[b]) {
    if (threadIdx.x == 0) {
      dn[row] = 0.0;
      lr[row] = 0.0;
    }
    return;
  }
  const float* py = yd + (int64_t)b * yc + (int64_t)j * yr;
  const float* pp = mp + (int64_t)b * pc + (int64_t)j * pr;
  const float* pq = mq + (int64_t)b * qc + (int64_t)j * qr;
  double s2 = 0.0, sz = 0.0;
  if (vec) {
    const f4v* vy = reinterpret_cast<const f4v*>(py);
    const f4v* vp = reinterpret_cast<const f4v*>(pp);
    const f4v* vq = reinterpret_cast<const f4v*>(pq);
    const int n4 = d >> 2;
#pragma unroll 4
    for (int i = threadIdx.x; i < n4; i += kThreads) {
      const f4v a = __builtin_nontemporal_load(vy + i);
      const f4v p = __builtin_nontemporal_load(vp + i);
      const f4v q = __builtin_nontemporal_load(vq + i);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const double dd = (double)p[c] - (double)q[c];
        const double zz = (double)a[c] - (double)p[c];
        s2 = fma(dd, dd, s2);
        sz = fma(zz, dd, sz);
      }
    }
  } else {
    for (int i = threadIdx.x; i < d; i += kThreads) {
      const double dd = (double)pp[i] - (double)pq[i];
      const double zz = (double)py[i] - (double)pp[i];
      s2 = fma(dd, dd, s2);
      sz = fma(zz, dd, sz);
    }
  }
  s2 = wave_sum(s2);
  sz = wave_sum(sz);
  __shared__ double red[2][kThreads / 64];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) {
    red[0][w] = s2;
    red[1][w] = sz;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double t2 = 0.0, tz = 0.0;
    for (int i = 0; i < kThreads / 64; ++i) {
      t2 += red[0][i];
      tz += red[1][i];
    }
    const double s = sigma[(int64_t)b * (K + 1) + j];
    const double inv = 1.0 / (s * s);
    dn[row] = sqrt(t2 * inv);
    lr[row] = -tz * inv - 0.5 * t2 * inv;
  }
}

// log Psi_alpha(x) given the log normaliser Lstar = log(alpha Phi(u*) - Phi(u* - v)).
__device__ __forceinline__ double log_cdf(double x, double la, double v, double us,
                                          double Lstar) {
  if (x >= us) return 0.0;
  return log_excess(x, la, v) - Lstar;
}

// Inverse of Psi_alpha at u, with all 64 lanes of the wavefront: the doubling
// of Alg. 7 for 63 candidate lower ends at once (lane i tests u* - 2^i), then
// a 64-way multisection (lane i evaluates log Psi at the i+1-th of 65
// points).  After the second and later multisection passes the four points
// around the crossing (the pass's points and the bracket's ends) give the
// cubic inverse interpolant of log Psi at log u; it is taken when it lies in
// the new bracket and agrees with both quadratic interpolants to 1e-13
// (relative), i.e. where log Psi is smooth on the scale of the points --
// typically after the second or third pass.  Otherwise the multisection goes
// on until the bracket is 1e-8 (relative) wide and a linear interpolation of
// log Psi between its ends, whose values the lanes already hold, closes it:
// its error is far below the bracket width except next to u*, where the
// density vanishes (there it is at most the width).
__device__ double usample_exact(double u, double la, double v, int lane) {
  const double us = la / v + 0.5 * v;
  const double logu = log(u);
  // one pass: lanes 0..62 the doubling candidates u* - 2^i, lane 63 the
  // normaliser log(alpha Phi(u*) - Phi(u* - v))
  const double le = log_excess(lane < 63 ? us - ldexp(1.0, lane) : us, la, v);
  const double Lstar = __shfl(le, 63);
  const double fc = le - Lstar;
  const uint64_t above = __ballot(lane < 63 && fc > logu) | (1ull << 63);
  const int p = (~above == 0ull) ? 63 : (__ffsll((unsigned long long)~above) - 1);
  double lo = us - ldexp(1.0, p), flo = p < 63 ? __shfl(fc, p < 63 ? p : 0) : -INFINITY;
  double hi = p == 0 ? us : us - ldexp(1.0, p - 1), fhi = p == 0 ? 0.0 : __shfl(fc, p > 0 ? p - 1 : 0);
  for (int it = 0; it < 64; ++it) {
    const double mid = 0.5 * (lo + hi);
    if (!(mid > lo && mid < hi) || hi - lo <= 1e-8 * fmax(1.0, fabs(lo))) break;
    const double x = lo + (hi - lo) * ((double)(lane + 1) / 65.0);
    const double fx = log_cdf(x, la, v, us, Lstar);
    const uint64_t below = __ballot(fx < logu);
    const int cnt = __popcll(below);
    const double nlo = __shfl(x, cnt > 0 ? cnt - 1 : 0), nflo = __shfl(fx, cnt > 0 ? cnt - 1 : 0);
    const double nhi = __shfl(x, cnt < 64 ? cnt : 63), nfhi = __shfl(fx, cnt < 64 ? cnt : 63);
    // the points in order: e = 0 the bracket's low end, e = i + 1 lane i's
    // point, e = 65 its high end; the crossing lies between e = cnt and cnt + 1
    const int e0 = min(max(cnt - 1, 0), 62);
    double px[4], pf[4];  // points and their log Psi, increasing
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = e0 + q;
      const int src = min(max(e - 1, 0), 63);
      const double sx = __shfl(x, src), sf = __shfl(fx, src);
      px[q] = e == 0 ? lo : e == 65 ? hi : sx;
      pf[q] = e == 0 ? flo : e == 65 ? fhi : sf;
    }
    // (after the first pass the points are still too far apart to pass the test)
    if (it > 0 && isfinite(pf[0]) && isfinite(pf[3]) && pf[0] < pf[1] && pf[1] < pf[2] &&
        pf[2] < pf[3]) {
      // Lagrange weights in log Psi at log u, from the six reciprocal differences
      const double r01 = 1.0 / (pf[0] - pf[1]), r02 = 1.0 / (pf[0] - pf[2]), r03 = 1.0 / (pf[0] - pf[3]);
      const double r12 = 1.0 / (pf[1] - pf[2]), r13 = 1.0 / (pf[1] - pf[3]), r23 = 1.0 / (pf[2] - pf[3]);
      const double d0 = logu - pf[0], d1 = logu - pf[1], d2 = logu - pf[2], d3 = logu - pf[3];
      const double x3 = px[0] * (d1 * d2 * d3) * (r01 * r02 * r03) - px[1] * (d0 * d2 * d3) * (r01 * r12 * r13) +
                        px[2] * (d0 * d1 * d3) * (r02 * r12 * r23) - px[3] * (d0 * d1 * d2) * (r03 * r13 * r23);
      const double q0 = px[0] * (d1 * d2) * (r01 * r02) - px[1] * (d0 * d2) * (r01 * r12) +
                        px[2] * (d0 * d1) * (r02 * r12);
      const double q1 = px[1] * (d2 * d3) * (r12 * r13) - px[2] * (d1 * d3) * (r12 * r23) +
                        px[3] * (d1 * d2) * (r13 * r23);
      const double blo = cnt > 0 ? nlo : lo, bhi = cnt < 64 ? nhi : hi;
      if (fmax(fabs(x3 - q0), fabs(x3 - q1)) <= 1e-13 * fmax(1.0, fabs(x3)) && x3 >= blo && x3 <= bhi)
        return x3;
    }
    if (cnt > 0) {
      lo = nlo;
      flo = nflo;
    }
    if (cnt < 64) {
      hi = nhi;
      fhi = nfhi;
    }
  }
  const double t = fhi > flo ? (logu - flo) / (fhi - flo) : 0.5;
  return lo + (hi - lo) * fmin(fmax(t, 0.0), 1.0);
}

// The capped doubling/bisection of the paper's experiments (3 + 4 steps).
__device__ double usample_paper(double u, double la, double v) {
  const double us = la / v + 0.5 * v;
  const double Lstar = log_excess(us, la, v);
  const double logu = log(u);
  double hi = us, lo = us - 1.0;
  for (int n = 0; n < 3 && log_cdf(lo, la, v, us, Lstar) > logu; ++n) lo = hi - 2.0 * (hi - lo);
  double mid = 0.5 * (lo + hi);
  for (int n = 0; n < 4; ++n) {
    const double lc = log_cdf(mid, la, v, us, Lstar);
    if (fabs(exp(lc) - u) <= 1e-6) break;
    if (lc < logu)
      lo = mid;
    else
      hi = mid;
    mid = 0.5 * (lo + hi);
  }
  return mid;
}

// The acceptance decision of one chain (one wavefront; lane j-1 holds ell_j
// and ||Delta_j|| of draft step j, kb valid steps): prefix recursion, h_j,
// coins, tau, alpha_res and, when tau <= kb and need_u, the U draw of Alg. 7.
// Temperature omega (w2 = omega^2): the tempered verifications of the
// appendix use ell_j / omega^2 wherever ell_j enters the acceptance, and the
// untempered ||Delta||; w2 = 1 is the exact method.
struct Decision {
  int tau;
  double la_res, U;
  uint64_t coins;
  uint64_t ties;  // steps whose coin lies within kTieWindow of its threshold
};

// A coin within this distance of its threshold (|eta_j - h_j|, or alpha_j for
// token verification) is a tie: rounding in another implementation may flip
// it, so such decisions are counted.
constexpr double kTieWindow = 1e-6;

__device__ Decision decide(int mode, int umode, int kb, double ell_raw, double vn, uint32_t b,
                           uint32_t r, uint64_t seed, int lane, double w2, bool need_u) {
  const bool valid = lane < kb;
  const double ell = ell_raw / w2;
  // prefix recursion, replayed per lane in the definition's order
  double acc = 0.0, la = 0.0;
  for (int i = 0; i < kb; ++i) {
    const double e = __shfl(ell, i);
    acc = fmin(0.0, acc + e);
    if (i == lane) la = acc;
  }
  const double vnext = __shfl_down(vn, 1);
  double lh;
  if (mode == SD_BLOCK)
    lh = (lane + 1 < kb) ? block_log_h(la, vnext) : la;
  else
    lh = fmin(0.0, ell);
  const uint4 w = philox((uint32_t)(lane >> 2), b, r, TAG_COIN << 24, seed);
  const double eta = uniform64(pick(w, lane & 3));
  const uint64_t cm = __ballot(valid && log(eta) < lh);
  const uint64_t tm = __ballot(valid && fabs(eta - exp(lh)) <= kTieWindow);
  const uint64_t vmask = kb >= 64 ? ~0ull : ((1ull << kb) - 1ull);
  int t;
  if (mode == SD_BLOCK) {
    t = cm ? (64 - __clzll((long long)cm)) + 1 : 1;
  } else {
    const uint64_t rej = ~cm & vmask;
    t = rej ? __ffsll((unsigned long long)rej) : kb + 1;
  }
  const double la_prev = __shfl(la, t >= 2 ? t - 2 : 0);
  const double la_res = (mode == SD_BLOCK && t >= 2) ? la_prev : 0.0;
  double U = NAN;
  if (t <= kb && need_u) {
    const double v = __shfl(vn, t - 1);  // > 0: a rejection never lands on a zero offset
    const uint4 wu = philox(0u, b, r, TAG_USAMPLE << 24, seed);
    const double u = uniform64(wu.x);
    if (umode == SD_USAMPLE_PAPER) {
      double up = 0.0;
      if (lane == 0) up = usample_paper(u, la_res, v);
      U = __shfl(up, 0);
    } else {
      U = usample_exact(u, la_res, v, lane);
    }
  }
  return Decision{t, la_res, U, cm, tm};
}

__global__ __launch_bounds__(kThreads) void scan_kernel(
    int B, int K, int mode, int umode, const double* __restrict__ dn,
    const double* __restrict__ lr, const int32_t* __restrict__ kbv,
    const uint32_t* __restrict__ rnd, uint64_t seed, double w2, int32_t* __restrict__ tau,
    double* __restrict__ lar, double* __restrict__ ures, uint64_t* __restrict__ coins,
    int* nanflag, const int* gate) {
  if (gate && *gate == 0) return;
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (b >= B) return;  // whole wavefront
  const int kb = min(kbv[b], K);
  if (kb <= 0) {
    if (lane == 0) {
      tau[b] = 0;
      lar[b] = 0.0;
      ures[b] = NAN;
      if (coins) coins[b] = 0ull;
    }
    return;
  }
  const bool valid = lane < kb;
  const double ell = valid ? lr[(int64_t)b * K + lane] : 0.0;
  const double vn = valid ? dn[(int64_t)b * K + lane] : 0.0;
  if (nanflag && __ballot(valid && !(isfinite(ell) && isfinite(vn))) != 0ull && lane == 0)
    atomicOr(nanflag, 1);
  const Decision D = decide(mode, umode, kb, ell, vn, (uint32_t)b, rnd[b], seed, lane, w2, true);
  if (lane == 0) {
    tau[b] = D.tau;
    lar[b] = D.la_res;
    ures[b] = D.U;
    if (coins) coins[b] = D.coins;
  }
}

// The sampler's verification: sums the partials of the fused target call
// (fixed tile order) into ||Delta_j||, ell_j and, for the residual,
// e.G = sum_i (m^p - m^q)_i G_i / (sigma ||Delta||) of every row, decides, and
// hands the next kernel what it needs to form the residual elementwise:
//   rmode 1: y = m^q + sigma G + rcoef (m^p - m^q),  rcoef = (U - e.G)/||Delta||
//   rmode 2: y = m^q_{K_b} + sigma xi'  (full accept, target draw)
//   rmode 3: y = yhat_{K_b}             (full accept that reaches step N)
//   rmode 4: y = yhat_tau - rcoef (m^p - m^q),  rcoef = 1 + 2 D.W / D.D
//            (reflection residual, Alg. 4: m^q + sigma (I - 2 e e^T) Z with
//            D = m^p - m^q = sigma Delta and W = yhat_tau - m^p = sigma Z,
//            whose two sums are the log-ratio partials of row tau - 1)
// The round's decision record (tau, coins, log alpha_res, U) is kept per chain,
// and the coins within kTieWindow of their thresholds are added to ties[b].
// It also clears the next round's active flag before looking at its gate,
// and stores the gate (whether any chain was still active after the previous
// round) tagged with that round's index, (pub_round << 1) | flag, into
// host_prev, a word of mapped host memory that the host polls, so that
// neither a device-to-host copy nor an event is queued per round.
__global__ __launch_bounds__(kThreads) void scan_fused_kernel(
    int B, int K, int d, int N, int mode, int umode, const double* __restrict__ lrp, int nct,
    const double* __restrict__ sigma, const int32_t* __restrict__ kcur,
    const uint32_t* __restrict__ rcur, uint64_t seed, double w2, bool reflect,
    int32_t* __restrict__ tau, int32_t* __restrict__ rmode,
    float* __restrict__ rcoef, float* __restrict__ rsig, uint64_t* __restrict__ coins,
    double* __restrict__ lar, double* __restrict__ ures, int32_t* __restrict__ ties,
    int* nanflag, int* act_next, int* host_prev, int pub_round, const int* gate, int chain0) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    *act_next = 0;
    if (host_prev) {
      __atomic_store_n(host_prev, (pub_round << 1) | (gate ? *gate : 1), __ATOMIC_RELAXED);
      __threadfence_system();
    }
  }
  if (gate && *gate == 0) return;
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (b >= B) return;
  const int K1 = K + 1;
  const int k = kcur[b];
  const int kb = k < N ? min(K, N - k) : 0;
  if (kb <= 0) {
    if (lane == 0) {
      tau[b] = 0;
      rmode[b] = 0;
    }
    return;
  }
  const bool valid = lane < kb;
  // Sum the column-tile partials of each draft row: row j is spread over lpr
  // lanes (64 / K rounded up to a power of two), each lane takes every lpr-th
  // tile with four independent accumulators (loads in flight together), and
  // the lanes of a row combine in a fixed xor tree; then lane j fetches row
  // j's totals.  Fixed order throughout, so the sums are deterministic.
  int kp = 1;
  while (kp < K) kp <<= 1;
  const int lpr = 64 / kp, j = lane / lpr, sub = lane % lpr;
  double a2[4] = {0.0, 0.0, 0.0, 0.0}, az[4] = {0.0, 0.0, 0.0, 0.0}, ag[4] = {0.0, 0.0, 0.0, 0.0};
  if (j < kb) {
    const double* pl = lrp + ((int64_t)b * K1 + j) * nct * 3;
    int ct = sub;
    for (; ct + 3 * lpr < nct; ct += 4 * lpr) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const double* q = pl + 3 * (ct + u * lpr);
        a2[u] += q[0];
        az[u] += q[1];
        ag[u] += q[2];
      }
    }
    for (; ct < nct; ct += lpr) {
      a2[0] += pl[3 * ct];
      az[0] += pl[3 * ct + 1];
      ag[0] += pl[3 * ct + 2];
    }
  }
  double s2 = (a2[0] + a2[1]) + (a2[2] + a2[3]);
  double sz = (az[0] + az[1]) + (az[2] + az[3]);
  double sgd = (ag[0] + ag[1]) + (ag[2] + ag[3]);
  for (int o = 1; o < lpr; o <<= 1) {
    s2 += __shfl_xor(s2, o);
    sz += __shfl_xor(sz, o);
    sgd += __shfl_xor(sgd, o);
  }
  const int src = min(lane * lpr, 63);
  s2 = __shfl(s2, src);
  sz = __shfl(sz, src);
  sgd = __shfl(sgd, src);
  // sigma of rows 0..K_b (lane j holds row j); the residual's sigma is taken
  // from these lanes below instead of a second load
  const double sgl = lane <= kb ? sigma[(int64_t)b * K1 + lane] : 1.0;
  const double sg = valid ? sgl : 1.0;
  const double inv = 1.0 / (sg * sg);
  const double vn = valid ? sqrt(s2 * inv) : 0.0;
  const double ell = valid ? -sz * inv - 0.5 * s2 * inv : 0.0;
  if (__ballot(valid && !(isfinite(ell) && isfinite(vn))) != 0ull && lane == 0) atomicOr(nanflag, 1);
  const uint32_t r = rcur[b];
  const Decision D = decide(mode, umode, kb, ell, vn, (uint32_t)(chain0 + b), r, seed, lane, w2,
                            !reflect);
  const int t = D.tau;
  int rm;
  float cf = 0.f, sgo = 0.f;
  const double st = __shfl(sgl, t <= kb ? t - 1 : kb);
  const double s2t = __shfl(s2, t <= kb ? t - 1 : 0), szt = __shfl(sz, t <= kb ? t - 1 : 0);
  if (t <= kb && reflect) {
    // D.D > 0: a rejection never lands on a zero offset (kept as a guard)
    rm = 4;
    cf = s2t > 0.0 ? (float)(1.0 + 2.0 * szt / s2t) : 1.0f;
  } else if (t <= kb) {
    const double v = __shfl(vn, t - 1);
    const double eG = __shfl(sgd, t - 1) / (st * v);
    rm = 1;
    cf = (float)((D.U - eG) / v);
    sgo = (float)st;
  } else if (kb + 1 <= N - k) {
    rm = 2;
    sgo = (float)st;
  } else {
    rm = 3;
  }
  if (lane == 0) {
    tau[b] = t;
    rmode[b] = rm;
    rcoef[b] = cf;
    rsig[b] = sgo;
    coins[b] = D.coins;
    lar[b] = D.la_res;
    ures[b] = D.U;
    ties[b] += __popcll(D.ties);
  }
}

}  // namespace

hipError_t verify_launch(int B, int K, int d, int mode, const float* yd, sd_stride ys,
                         const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                         const double* sigma, const int32_t* kb, const uint32_t* rnd,
                         uint64_t seed, int umode, double w2, int32_t* tau, double* lar,
                         double* ures, double* dn, double* lr, uint64_t* coins, int* nanflag,
                         hipStream_t s, const int* gate) {
  const bool vec = (d % 4 == 0) && ys.chain % 4 == 0 && ys.row % 4 == 0 && mps.chain % 4 == 0 &&
                   mps.row % 4 == 0 && mqs.chain % 4 == 0 && mqs.row % 4 == 0 &&
                   aligned16(yd) && aligned16(mp) && aligned16(mq);
  const int64_t rows = (int64_t)B * K;
  hipError_t e = timed("logratio_reduce", s, [&] {
    logratio_kernel<<<(unsigned)rows, kThreads, 0, s>>>(K, d, yd, ys.chain, ys.row, mp,
                                                        mps.chain, mps.row, mq, mqs.chain,
                                                        mqs.row, sigma, kb, dn, lr, vec, gate);
  });
  if (e != hipSuccess) return e;
  const int per = kThreads / 64;
  return timed("block_scan", s, [&] {
    scan_kernel<<<(B + per - 1) / per, kThreads, 0, s>>>(B, K, mode, umode, dn, lr, kb, rnd, seed,
                                                        w2, tau, lar, ures, coins, nanflag, gate);
  });
}

hipError_t scan_fused_launch(int B, int K, int d, int N, int mode, int umode, const double* lrp,
                             int nct, const double* sigma, const int32_t* kcur,
                             const uint32_t* rcur, uint64_t seed, double w2, bool reflect,
                             int32_t* tau, int32_t* rmode, float* rcoef, float* rsig,
                             uint64_t* coins, double* lar, double* ures, int32_t* ties,
                             int* nanflag, int* act_next, int* host_prev, int pub_round,
                             hipStream_t s, const int* gate, int chain0) {
  const int per = kThreads / 64;
  return launch_timed("scan_fused", scan_fused_kernel, dim3((B + per - 1) / per), dim3(kThreads), s,
                      B, K, d, N, mode, umode, lrp, nct, sigma, kcur, rcur, seed, w2, reflect, tau,
                      rmode, rcoef, rsig, coins, lar, ures, ties, nanflag, act_next, host_prev,
                      pub_round, gate, chain0);
}

}  // namespace sd
