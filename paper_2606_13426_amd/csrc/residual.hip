// The new state of each chain after verification (Alg. 8, residual part) and
// the sampler's commit step.
//
// residual_kernel: one workgroup per chain.  For a rejection at tau the
// Decomposition residual (Prop. 1, Alg. 5) is
//     y = m^q + sigma (U e + G - e (e.G)),  e = (m^p - m^q) / (sigma ||Delta||),
// rewritten per coordinate as  y_i = mq_i + sigma G_i + c (mp_i - mq_i)  with
// c = (U - e.G)/||Delta||, so one float64 reduction (e.G) followed by one
// elementwise pass suffices; G is regenerated from Philox in both passes
// instead of being stored.
#include "common.hpp"
#include "philox.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double block_sum(double v, double* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < kThreads / 64; ++i) t += red[i];
  return t;
}

__global__ __launch_bounds__(kThreads) void residual_kernel(
    int K, int d, const float* __restrict__ yd, int64_t yc, int64_t yr,
    const float* __restrict__ mp, int64_t pc, int64_t pr, const float* __restrict__ mq,
    int64_t qc, int64_t qr, const double* __restrict__ sigma, const int32_t* __restrict__ kbv,
    const int32_t* __restrict__ left, const int32_t* __restrict__ tauv,
    const double* __restrict__ ures, const double* __restrict__ dn,
    const uint32_t* __restrict__ rnd, uint64_t seed, float* __restrict__ y, const int* gate) {
  if (gate && *gate == 0) return;
  const int b = blockIdx.x;
  const int t = tauv[b];
  const int kb = min(kbv[b], K);
  if (t <= 0 || kb <= 0 || t > kb + 1) return;
  const uint32_t r = rnd[b];
  float* out = y + (int64_t)b * d;
  const int ng = (d + 3) / 4;
  if (t <= kb) {
    const float* p = mp + (int64_t)b * pc + (int64_t)(t - 1) * pr;
    const float* q = mq + (int64_t)b * qc + (int64_t)(t - 1) * qr;
    const double s = sigma[(int64_t)b * (K + 1) + (t - 1)];
    const double v = dn[(int64_t)b * K + (t - 1)];
    const uint32_t c3 = TAG_RESID << 24;
    double acc = 0.0;
    for (int g = threadIdx.x; g < ng; g += kThreads) {
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
      const int e0 = 4 * g, cnt = min(4, d - e0);
      for (int c = 0; c < cnt; ++c)
        acc += ((double)p[e0 + c] - (double)q[e0 + c]) * (double)get4(z, c);
    }
    __shared__ double red[kThreads / 64];
    const double eG = block_sum(acc, red) / (s * v);
    const float coef = (float)((ures[b] - eG) / v);
    const float sf = (float)s;
    for (int g = threadIdx.x; g < ng; g += kThreads) {
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
      const int e0 = 4 * g, cnt = min(4, d - e0);
      for (int c = 0; c < cnt; ++c) {
        const float qi = q[e0 + c];
        out[e0 + c] = qi + sf * get4(z, c) + coef * (p[e0 + c] - qi);
      }
    }
  } else if (kb + 1 <= left[b]) {
    // full accept: draw Y_{k+K_b+1} from the target kernel at the last draft
    const float* q = mq + (int64_t)b * qc + (int64_t)kb * qr;
    const float sf = (float)sigma[(int64_t)b * (K + 1) + kb];
    for (int g = threadIdx.x; g < ng; g += kThreads) {
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, TAG_TARGET << 24, seed));
      const int e0 = 4 * g, cnt = min(4, d - e0);
      for (int c = 0; c < cnt; ++c) out[e0 + c] = q[e0 + c] + sf * get4(z, c);
    }
  } else {
    // the block reached step N: the last draft is Y_N
    const float* src = yd + (int64_t)b * yc + (int64_t)(kb - 1) * yr;
    for (int i = threadIdx.x; i < d; i += kThreads) out[i] = src[i];
  }
}

// Advance k, the round counter and the Free-Drafter cache (the target score
// of row min(tau, K_b) of this round), count the chains still active and
// record tau.
__global__ __launch_bounds__(kThreads) void commit_kernel(
    int B, int K, int d, int N, const int32_t* __restrict__ tauv, const int32_t* __restrict__ kbv,
    int32_t* kk, uint32_t* rnd, const float* __restrict__ score, int64_t sc, int64_t sr,
    float* __restrict__ cache, int* cnt, int64_t* hist, int64_t* steps, int32_t* trace, int r,
    int trace_rounds, const int* gate) {
  if (gate && *gate == 0) return;
  const int b = blockIdx.x;
  const int t = tauv[b];
  const int kb = min(kbv[b], K);
  if (t <= 0 || t > kb + 1) {
    if (threadIdx.x == 0 && trace && r < trace_rounds) trace[(int64_t)r * B + b] = 0;
    return;
  }
  const int k = kk[b];
  const int knew = min(k + t, N);
  if (knew < N) {
    const float* src = score + (int64_t)b * sc + (int64_t)min(t, kb) * sr;
    float* dst = cache + (int64_t)b * d;
    for (int i = threadIdx.x; i < d; i += kThreads) dst[i] = src[i];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    kk[b] = knew;
    rnd[b] = rnd[b] + 1u;
    if (knew < N) atomicAdd(cnt, 1);
    atomicAdd((unsigned long long*)&hist[t], 1ull);
    atomicAdd((unsigned long long*)steps, (unsigned long long)(knew - k));
    if (trace && r < trace_rounds) trace[(int64_t)r * B + b] = t;
  }
}

}  // namespace

hipError_t residual_launch(int B, int K, int d, const float* yd, sd_stride ys, const float* mp,
                           sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                           const int32_t* kb, const int32_t* left, const int32_t* tau,
                           const double* ures, const double* dn, const uint32_t* rnd,
                           uint64_t seed, float* y, hipStream_t s, const int* gate) {
  return timed("residual_draw", s, [&] {
    residual_kernel<<<B, kThreads, 0, s>>>(K, d, yd, ys.chain, ys.row, mp, mps.chain, mps.row, mq,
                                           mqs.chain, mqs.row, sigma, kb, left, tau, ures, dn,
                                           rnd, seed, y, gate);
  });
}

hipError_t commit_launch(int B, int K, int d, int N, const int32_t* tau, const int32_t* kb,
                         int32_t* k, uint32_t* rnd, const float* score, sd_stride ss,
                         float* cache, int* cnt, int64_t* hist, int64_t* steps, int32_t* trace,
                         int r, int trace_rounds, hipStream_t s, const int* gate) {
  return timed("commit", s, [&] {
    commit_kernel<<<B, kThreads, 0, s>>>(B, K, d, N, tau, kb, k, rnd, score, ss.chain, ss.row,
                                         cache, cnt, hist, steps, trace, r, trace_rounds, gate);
  });
}

}  // namespace sd
