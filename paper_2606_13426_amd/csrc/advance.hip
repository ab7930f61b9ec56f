// The sampler's end of a round and start of the next, fused elementwise.
//
// After the fused verification has decided tau (and, for a rejection, the
// scalar rcoef = (U - e.G)/||Delta||), every remaining step of the round is
// elementwise in the coordinates:
//   residual  y_i = m^q_i + sigma G_i + rcoef (m^p_i - m^q_i)     (Alg. 5 with e.G known)
//             or y_i = yhat_tau,i - rcoef (m^p_i - m^q_i)          (Alg. 4, reflection)
//             or the full-accept target draw, or the last draft at step N (Alg. 8);
//   commit    k <- min(k + tau, N), round <- round + 1 (one thread per chain),
//             the new state into x row 0 (and into y once the chain is done);
//   draft     the next round's Free-Drafter block from y_i, whose cached score
//             is that of row min(tau, K_b) of this round (Sec. 3.3), recovered
//             from the same round's (x, m^q) rows.
// Each thread owns four coordinates of one chain: it reads every row it needs
// (x and m^q of the residual row, the cache rows, the last draft) before it
// overwrites that chain's x rows and cache row sv = c2_c S_c at the same
// coordinates, so one pass replaces the separate residual, commit and draft
// kernels and the state never leaves registers between them.  The draft means
// m^p are not stored: where the residual needs one it is recomputed from the
// draft state and the cache with draft_mean, bit for bit.
// With the Frozen Drafter the next draft needs a target call at the new state
// first, so the kernel stops after writing the state into x row 0 and points
// the next cache at that row and step.
#include "common.hpp"
#include "philox.hpp"
#include "rows.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void advance_kernel(
    Sched sc, const float4* __restrict__ coef, int B, int K, int d, uint64_t seed,
    const int32_t* __restrict__ kcur, const uint32_t* __restrict__ rcur,
    const int32_t* __restrict__ crow_cur, const int32_t* __restrict__ cstep_cur,
    int32_t* __restrict__ knext, uint32_t* __restrict__ rnext, int32_t* __restrict__ crow_next,
    int32_t* __restrict__ cstep_next, const int32_t* __restrict__ tauv,
    const int32_t* __restrict__ rmode, const float* __restrict__ rcoef,
    const float* __restrict__ rsig, float* __restrict__ X, float* __restrict__ SV,
    const float* __restrict__ MQ, float* __restrict__ y, int32_t* __restrict__ step,
    double* __restrict__ sigma, int32_t* __restrict__ hist, int64_t* __restrict__ steps,
    int* act_next, int32_t* __restrict__ trace, int r_round, int trace_rounds, bool vec_ok,
    bool frozen, bool stream, const int* gate, int chain0, int trace_ld) {
  if (gate && *gate == 0) return;
  const int N = sc.N, K1 = K + 1;
  const int b = blockIdx.y;
  const uint32_t chain = (uint32_t)(chain0 + b);  // the generator's chain index
  const int t = tauv[b];
  const int k = kcur[b];
  const uint32_t r = rcur[b];
  const bool active = t > 0;
  const int kb = active ? min(K, N - k) : 0;
  const int knew = active ? min(k + t, N) : k;
  const int cr = frozen ? 0 : min(t, kb);
  const int cs = frozen ? min(knew, N - 1) : min(k + cr, N - 1);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (active) {
      knext[b] = knew;
      rnext[b] = r + 1u;
      crow_next[b] = cr;
      cstep_next[b] = cs;
      hist[(int64_t)b * (SD_MAX_BLOCK + 2) + t] += 1;
      steps[b] += knew - k;
      if (knew < N) *act_next = 1;
    } else {
      knext[b] = k;
      rnext[b] = r;
      crow_next[b] = crow_cur[b];
      cstep_next[b] = cstep_cur[b];
    }
    if (trace && r_round < trace_rounds) trace[(int64_t)r_round * trace_ld + b] = active ? t : 0;
  }
  if (!active) return;
  // the next round's step index and sigma of every target row
  if (blockIdx.x == 0 && threadIdx.x <= K && knew < N) {
    const int j = threadIdx.x;
    step[(int64_t)b * K1 + j] = min(knew + j, N - 1);
    sigma[(int64_t)b * K1 + j] = sched_sigma(sc, min(knew + j, N));
  }
  const int g = blockIdx.x * kThreads + threadIdx.x;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const int cnt = min(4, d - e0);
  const bool vec = vec_ok && cnt == 4;
  float* xb = X + (int64_t)b * K1 * d + e0;
  float* sb = SV + (int64_t)b * d + e0;
  const float* qb = MQ + (int64_t)b * K1 * d + e0;
  float yv[4];
  const int rm = rmode[b];
  if (rm == 1) {
    // m^p of row t - 1 from its draft state and this round's cache
    float xv[4], qv[4], sv[4];
    load4(xb + (int64_t)(t - 1) * d, cnt, vec, xv);
    load4(qb + (int64_t)(t - 1) * d, cnt, vec, qv);
    load4(sb, cnt, vec, sv);
    const float4 cn = step_coef(sc, coef, k + t - 1);
    const float c2s = cn.y * step_coef(sc, coef, cstep_cur[b]).w;
    const float sg = rsig[b], cf = rcoef[b];
    const float4 z = normals4(philox((uint32_t)g, chain, r, TAG_RESID << 24, seed));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float pv = draft_mean(cn.x, xv[c], c2s, sv[c]);
      yv[c] = qv[c] + sg * get4(z, c) + cf * (pv - qv[c]);
    }
  } else if (rm == 4) {
    // reflection: yhat_tau - rcoef (m^p - m^q) of row t - 1
    float xv[4], xn[4], qv[4], sv[4];
    load4(xb + (int64_t)(t - 1) * d, cnt, vec, xv);
    load4(xb + (int64_t)t * d, cnt, vec, xn);
    load4(qb + (int64_t)(t - 1) * d, cnt, vec, qv);
    load4(sb, cnt, vec, sv);
    const float4 cn = step_coef(sc, coef, k + t - 1);
    const float c2s = cn.y * step_coef(sc, coef, cstep_cur[b]).w;
    const float cf = rcoef[b];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float pv = draft_mean(cn.x, xv[c], c2s, sv[c]);
      yv[c] = xn[c] - cf * (pv - qv[c]);
    }
  } else if (rm == 2) {
    float qv[4];
    load4(qb + (int64_t)kb * d, cnt, vec, qv);
    const float sg = rsig[b];
    const float4 z = normals4(philox((uint32_t)g, chain, r, TAG_TARGET << 24, seed));
#pragma unroll
    for (int c = 0; c < 4; ++c) yv[c] = qv[c] + sg * get4(z, c);
  } else {
    load4(xb + (int64_t)kb * d, cnt, vec, yv);
  }
  // y holds the state only where something reads it before the next round's
  // advance: the Frozen Drafter's draft (from y) and the run's output once the
  // chain has reached step N; otherwise x row 0 carries it
  if (frozen || knew >= N) store4(y + (int64_t)b * d + e0, cnt, vec, yv);
  if (knew >= N) return;
  if (frozen) {
    store4(xb, cnt, vec, yv, stream);
    return;
  }
  float xcv[4], qcv[4], sv[4];
  load4(xb + (int64_t)cr * d, cnt, vec, xcv);
  load4(qb + (int64_t)cr * d, cnt, vec, qcv);
  const float4 cc = step_coef(sc, coef, cs);
#pragma unroll
  for (int c = 0; c < 4; ++c) sv[c] = qcv[c] - cc.x * xcv[c];  // c2_c S_c
  store4(sb, cnt, vec, sv);
  store4(xb, cnt, vec, yv, stream);
  draft_rows(sc, coef, K, knew, min(K, N - knew), chain, r + 1u, seed, g, yv, sv, cc.w, xb,
             d, nullptr, d, cnt, vec, stream);
}

}  // namespace

hipError_t advance_launch(const Sched& sc, const float4* coef, int B, int K, int d,
                          uint64_t seed, const int32_t* kcur, const uint32_t* rcur,
                          const int32_t* crow_cur, const int32_t* cstep_cur, int32_t* knext,
                          uint32_t* rnext, int32_t* crow_next, int32_t* cstep_next,
                          const int32_t* tau, const int32_t* rmode, const float* rcoef,
                          const float* rsig, float* x, float* sv, const float* mq, float* y,
                          int32_t* step, double* sigma, int32_t* hist, int64_t* steps,
                          int* act_next, int32_t* trace, int r, int trace_rounds, bool frozen,
                          hipStream_t s, const int* gate, int chain0, int trace_ld,
                          int64_t stream_bytes) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  const bool vec = (d % 4 == 0) && aligned16(x) && aligned16(sv) && aligned16(mq) && aligned16(y);
  const bool stream = stream_rows(stream_bytes > 0 ? stream_bytes : (int64_t)B * (K + 1) * d * 4);
  return launch_timed("advance", advance_kernel, grid, dim3(kThreads), s, sc, coef, B, K, d, seed,
                      kcur, rcur, crow_cur, cstep_cur, knext, rnext, crow_next, cstep_next, tau, rmode,
                      rcoef, rsig, x, sv, mq, y, step, sigma, hist, steps, act_next, trace, r,
                      trace_rounds, vec, frozen, stream, gate, chain0, trace_ld > 0 ? trace_ld : B);
}

}  // namespace sd
