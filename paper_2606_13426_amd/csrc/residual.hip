// The new state of each chain after verification (Alg. 8, residual part) and
// the sampler's commit step.
//
// residual_kernel: one workgroup per chain.  For a rejection at tau the
// Decomposition residual (Prop. 1, Alg. 5) is
//     y = m^q + sigma (U e + G - e (e.G)),  e = (m^p - m^q) / (sigma ||Delta||),
// rewritten per coordinate as  y_i = mq_i + sigma G_i + c (mp_i - mq_i)  with
// c = (U - e.G)/||Delta||, so one float64 reduction (e.G) followed by one
// elementwise pass suffices; G and the two rows stay in registers between the
// passes (up to 512 threads x 4 groups of 4 coordinates).
//
// The reflection residual of sample verification (Alg. 4),
//     y = m^q + sigma (I - 2 e e^T) Z,  Z = (yhat_tau - m^p) / sigma,
// is with D = m^p - m^q and W = yhat_tau - m^p
//     y_i = yhat_i - c D_i,  c = 1 + 2 (D.W) / (D.D),
// two float64 reductions and one elementwise pass (reflection_row).
#include "common.hpp"
#include "philox.hpp"

namespace sd {
namespace {

constexpr int kMaxThreads = 512;
constexpr int kKeep = 6;  // float4 groups per thread kept in registers (d <= 12288)

// Sum over the workgroup (blockDim.x a multiple of 64, at most 512).
__device__ __forceinline__ double block_sum(double v, double* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += red[i];
  return t;
}

__device__ __forceinline__ void ld4(const float* p, int cnt, float (&v)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = c < cnt ? p[c] : 0.0f;
}

// VEC: every row is 16-byte aligned and d % 4 == 0 (cnt is then always 4), so
// a group is one 16-byte access.
template <bool VEC>
__device__ __forceinline__ void ldg(const float* p, int cnt, float (&v)[4]) {
  if constexpr (VEC) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else {
    ld4(p, cnt, v);
  }
}
template <bool VEC>
__device__ __forceinline__ void stg(float* p, int cnt, const float (&v)[4]) {
  if constexpr (VEC) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (c < cnt) p[c] = v[c];
  }
}

// The rejection case: one pass reads m^q, m^p and draws G for this thread's
// groups (m^q and m^p - m^q kept in registers), reduces e.G, and the second
// pass writes y = m^q + sigma G + c (m^p - m^q), drawing G again (the same
// counter-based normals) rather than holding it: fewer registers, more
// workgroups in flight.  Groups beyond kKeep * blockDim.x (d > 12288) are
// re-read and redrawn in the second pass.
template <bool VEC>
__device__ __forceinline__ void decomposition_row(int b, int d, uint32_t r, uint64_t seed,
                                                  const float* p, const float* q, double s,
                                                  double v, double U, float* out, double* red) {
  const int ng = (d + 3) / 4;
  const int nt = blockDim.x;
  const uint32_t c3 = TAG_RESID << 24;
  float gq[kKeep][4], gd[kKeep][4];
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < kKeep; ++i) {
    const int g = threadIdx.x + i * nt;
    if (g < ng) {
      const int e0 = 4 * g, cnt = min(4, d - e0);
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
      float pv[4];
      ldg<VEC>(p + e0, cnt, pv);
      ldg<VEC>(q + e0, cnt, gq[i]);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        gd[i][c] = pv[c] - gq[i][c];
        if (c < cnt) acc += ((double)pv[c] - (double)gq[i][c]) * (double)get4(z, c);
      }
    }
  }
  for (int g = threadIdx.x + kKeep * nt; g < ng; g += nt) {
    const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
    const int e0 = 4 * g, cnt = min(4, d - e0);
    for (int c = 0; c < cnt; ++c) acc += ((double)p[e0 + c] - (double)q[e0 + c]) * (double)get4(z, c);
  }
  const double eG = block_sum(acc, red) / (s * v);
  const float coef = (float)((U - eG) / v);
  const float sf = (float)s;
#pragma unroll
  for (int i = 0; i < kKeep; ++i) {
    const int g = threadIdx.x + i * nt;
    if (g < ng) {
      const int e0 = 4 * g, cnt = min(4, d - e0);
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
      float o[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) o[c] = gq[i][c] + sf * get4(z, c) + coef * gd[i][c];
      stg<VEC>(out + e0, cnt, o);
    }
  }
  for (int g = threadIdx.x + kKeep * nt; g < ng; g += nt) {
    const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, c3, seed));
    const int e0 = 4 * g, cnt = min(4, d - e0);
    for (int c = 0; c < cnt; ++c) {
      const float qi = q[e0 + c];
      out[e0 + c] = qi + sf * get4(z, c) + coef * (p[e0 + c] - qi);
    }
  }
}

// The reflection residual of one rejected chain: sums D.D and D.W over the
// row in float64 (the thread's groups kept in registers up to kKeep), then
// y = yhat - c D.
__device__ __forceinline__ void reflection_row(int d, const float* yh, const float* p,
                                               const float* q, float* out, double* red) {
  const int ng = (d + 3) / 4;
  const int nt = blockDim.x;
  float gy[kKeep][4], gd[kKeep][4];
  double a2 = 0.0, az = 0.0;
#pragma unroll
  for (int i = 0; i < kKeep; ++i) {
    const int g = threadIdx.x + i * nt;
    if (g < ng) {
      const int e0 = 4 * g, cnt = min(4, d - e0);
      float pv[4], qv[4];
      ld4(yh + e0, cnt, gy[i]);
      ld4(p + e0, cnt, pv);
      ld4(q + e0, cnt, qv);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        gd[i][c] = pv[c] - qv[c];
        const double dd = (double)pv[c] - (double)qv[c];
        const double ww = (double)gy[i][c] - (double)pv[c];
        a2 = fma(dd, dd, a2);  // zero-padded lanes add zeros
        az = fma(ww, dd, az);
      }
    }
  }
  for (int g = threadIdx.x + kKeep * nt; g < ng; g += nt) {
    const int e0 = 4 * g, cnt = min(4, d - e0);
    for (int c = 0; c < cnt; ++c) {
      const double dd = (double)p[e0 + c] - (double)q[e0 + c];
      a2 = fma(dd, dd, a2);
      az = fma((double)yh[e0 + c] - (double)p[e0 + c], dd, az);
    }
  }
  const double t2 = block_sum(a2, red);
  __syncthreads();  // every thread has read red before it is reused
  const double tz = block_sum(az, red);
  // (no direction when D = 0: the draft noise is kept, y = yhat; a verification
  // never rejects such a step)
  const float cf = t2 > 0.0 ? (float)(1.0 + 2.0 * tz / t2) : 1.0f;
#pragma unroll
  for (int i = 0; i < kKeep; ++i) {
    const int g = threadIdx.x + i * nt;
    if (g < ng) {
      const int e0 = 4 * g, cnt = min(4, d - e0);
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (c < cnt) out[e0 + c] = gy[i][c] - cf * gd[i][c];
    }
  }
  for (int g = threadIdx.x + kKeep * nt; g < ng; g += nt) {
    const int e0 = 4 * g, cnt = min(4, d - e0);
    for (int c = 0; c < cnt; ++c) out[e0 + c] = yh[e0 + c] - cf * (p[e0 + c] - q[e0 + c]);
  }
}

// With COMMIT (the sampler) the same workgroup then advances the chain:
// k <- min(k + tau, N), round <- round + 1, and records where the Free Drafter
// finds its cached score next round (row min(tau, K_b) of this round's target
// means, at step k + min(tau, K_b)) and how many steps the chain advanced.
// Four wavefronts per SIMD (two 512-thread workgroups per compute unit): the
// register budget of 128 keeps a second chain's loads in flight while one
// workgroup reduces.
template <bool COMMIT, bool VEC>
__global__ __launch_bounds__(kMaxThreads, 4) void residual_kernel(
    int B, int K, int d, int N, const float* __restrict__ yd, int64_t yc, int64_t yr,
    const float* __restrict__ mp, int64_t pc, int64_t pr, const float* __restrict__ mq,
    int64_t qc, int64_t qr, const double* __restrict__ sigma, const int32_t* __restrict__ kbv,
    const int32_t* __restrict__ left, const int32_t* __restrict__ tauv,
    const double* __restrict__ ures, const double* __restrict__ dn, uint32_t* rnd, uint64_t seed,
    float* __restrict__ y, int32_t* kk, int32_t* crow, int32_t* cstep, int32_t* adv,
    int32_t* trace, int r_round, int trace_rounds, bool reflect, const int* gate) {
  __shared__ double red[kMaxThreads / 64];
  if (gate && *gate == 0) return;
  const int b = blockIdx.x;
  const int t = tauv[b];
  const int kb = min(kbv[b], K);
  if (t <= 0 || kb <= 0 || t > kb + 1) {
    if (COMMIT && threadIdx.x == 0 && trace && r_round < trace_rounds)
      trace[(int64_t)r_round * B + b] = 0;
    return;
  }
  const uint32_t r = rnd[b];
  float* out = y + (int64_t)b * d;
  const int ng = (d + 3) / 4;
  if (t <= kb && reflect) {
    reflection_row(d, yd + (int64_t)b * yc + (int64_t)(t - 1) * yr,
                   mp + (int64_t)b * pc + (int64_t)(t - 1) * pr,
                   mq + (int64_t)b * qc + (int64_t)(t - 1) * qr, out, red);
  } else if (t <= kb) {
    decomposition_row<VEC>(b, d, r, seed, mp + (int64_t)b * pc + (int64_t)(t - 1) * pr,
                      mq + (int64_t)b * qc + (int64_t)(t - 1) * qr,
                      sigma[(int64_t)b * (K + 1) + (t - 1)], dn[(int64_t)b * K + (t - 1)], ures[b],
                      out, red);
  } else if (kb + 1 <= left[b]) {
    // full accept: draw Y_{k+K_b+1} from the target kernel at the last draft
    const float* q = mq + (int64_t)b * qc + (int64_t)kb * qr;
    const float sf = (float)sigma[(int64_t)b * (K + 1) + kb];
    for (int g = threadIdx.x; g < ng; g += blockDim.x) {
      const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, TAG_TARGET << 24, seed));
      const int e0 = 4 * g, cnt = min(4, d - e0);
      for (int c = 0; c < cnt; ++c) out[e0 + c] = q[e0 + c] + sf * get4(z, c);
    }
  } else {
    // the block reached step N: the last draft is Y_N
    const float* src = yd + (int64_t)b * yc + (int64_t)(kb - 1) * yr;
    for (int i = threadIdx.x; i < d; i += blockDim.x) out[i] = src[i];
  }
  if (COMMIT) {
    __syncthreads();  // every thread has read rnd[b] before it changes
    if (threadIdx.x == 0) {
      const int k = kk[b];
      const int knew = min(k + t, N);
      const int cr = min(t, kb);
      kk[b] = knew;
      rnd[b] = r + 1u;
      crow[b] = cr;
      cstep[b] = min(k + cr, N - 1);
      adv[b] = knew - k;
      if (trace && r_round < trace_rounds) trace[(int64_t)r_round * B + b] = t;
    }
  }
}

// Threads per workgroup: one float4 group per thread up to 512 threads.
inline int residual_threads(int d) {
  const int ng = (d + 3) / 4;
  const int t = ((ng + 63) / 64) * 64;
  return t < kMaxThreads ? t : kMaxThreads;
}

}  // namespace

// Rows of the m^p and m^q views and of y all 16-byte aligned, d % 4 == 0.
inline bool residual_vec(int d, sd_stride mps, sd_stride mqs, const float* mp, const float* mq,
                         const float* y) {
  return d % 4 == 0 && mps.chain % 4 == 0 && mps.row % 4 == 0 && mqs.chain % 4 == 0 &&
         mqs.row % 4 == 0 && aligned16(mp) && aligned16(mq) && aligned16(y);
}

hipError_t residual_launch(int B, int K, int d, const float* yd, sd_stride ys, const float* mp,
                           sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                           const int32_t* kb, const int32_t* left, const int32_t* tau,
                           const double* ures, const double* dn, const uint32_t* rnd,
                           uint64_t seed, float* y, hipStream_t s) {
  const bool vec = residual_vec(d, mps, mqs, mp, mq, y);
  return timed("residual_draw", s, [&] {
    (vec ? residual_kernel<false, true> : residual_kernel<false, false>)<<<B, residual_threads(d), 0, s>>>(
        B, K, d, 0, yd, ys.chain, ys.row, mp, mps.chain, mps.row, mq, mqs.chain, mqs.row, sigma,
        kb, left, tau, ures, dn, const_cast<uint32_t*>(rnd), seed, y, nullptr, nullptr, nullptr,
        nullptr, nullptr, 0, 0, false, nullptr);
  });
}

hipError_t reflection_launch(int B, int K, int d, const float* yd, sd_stride ys, const float* mp,
                             sd_stride mps, const float* mq, sd_stride mqs, const double* sigma,
                             const int32_t* kb, const int32_t* left, const int32_t* tau,
                             const uint32_t* rnd, uint64_t seed, float* y, hipStream_t s) {
  return timed("residual_reflect", s, [&] {
    residual_kernel<false, false><<<B, residual_threads(d), 0, s>>>(
        B, K, d, 0, yd, ys.chain, ys.row, mp, mps.chain, mps.row, mq, mqs.chain, mqs.row, sigma,
        kb, left, tau, nullptr, nullptr, const_cast<uint32_t*>(rnd), seed, y, nullptr, nullptr,
        nullptr, nullptr, nullptr, 0, 0, true, nullptr);
  });
}

hipError_t residual_commit_launch(int B, int K, int d, int N, const float* yd, sd_stride ys,
                                  const float* mp, sd_stride mps, const float* mq, sd_stride mqs,
                                  const double* sigma, const int32_t* kb, const int32_t* left,
                                  const int32_t* tau, const double* ures, const double* dn,
                                  uint32_t* rnd, uint64_t seed, float* y, int32_t* k,
                                  int32_t* crow, int32_t* cstep, int32_t* adv, int32_t* trace,
                                  int r, int trace_rounds, hipStream_t s, const int* gate) {
  const bool vec = residual_vec(d, mps, mqs, mp, mq, y);
  return timed("residual_commit", s, [&] {
    (vec ? residual_kernel<true, true> : residual_kernel<true, false>)<<<B, residual_threads(d), 0, s>>>(
        B, K, d, N, yd, ys.chain, ys.row, mp, mps.chain, mps.row, mq, mqs.chain, mqs.row, sigma,
        kb, left, tau, ures, dn, rnd, seed, y, k, crow, cstep, adv, trace, r, trace_rounds, false,
        gate);
  });
}

}  // namespace sd
