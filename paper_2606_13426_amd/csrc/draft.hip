// Free Drafter (Sec. 3.3), chain initialisation and per-round bookkeeping.
//
// The draft recursion is sequential in the draft step i but independent across
// the d coordinates, so each thread owns four consecutive coordinates of one
// chain and walks i = 1..K_b keeping yhat in registers: the state is read once
// and every draft row and draft mean is written once (HBM-bound, no reuse).
#include "common.hpp"
#include "philox.hpp"
#include "rows.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void init_chains_kernel(int d, uint64_t seed, float* y,
                                                               float* x0, int64_t x0c) {
  const int b = blockIdx.y;
  const int g = blockIdx.x * kThreads + threadIdx.x;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, 0u, TAG_INIT << 24, seed));
  float* p = y + (int64_t)b * d + e0;
  const int cnt = min(4, d - e0);
  for (int c = 0; c < cnt; ++c) p[c] = get4(z, c);
  if (x0) {
    float* q = x0 + (int64_t)b * x0c + e0;
    for (int c = 0; c < cnt; ++c) q[c] = get4(z, c);
  }
}

// Draft block of one chain, four coordinates per thread.  The cached target
// score enters only as c2_n S_c.  With CACHE_FROM_MEANS the score is not
// stored: it is the score behind the target mean m^q_c = c1_c x_c + c2_c S_c
// of row crow of the previous round (step cstep), so
//   c2_n S_c = (c2_n / c2_c) (m^q_c - c1_c x_c),
// read from the same x / mq buffers before this chain's rows are overwritten
// (each thread reads and then writes only its own coordinates).
template <bool CACHE_FROM_MEANS>
__global__ __launch_bounds__(kThreads) void draft_kernel(
    Sched sc, const float4* __restrict__ coef, int K, int d, const float* __restrict__ y,
    const float* __restrict__ cs,
    const int32_t* __restrict__ crow, const int32_t* __restrict__ cstep,
    const float* __restrict__ mqprev, int64_t qc, int64_t qr, const int32_t* __restrict__ kk,
    const uint32_t* __restrict__ rnd, uint64_t seed, float* __restrict__ x, int64_t xc,
    int64_t xr, float* __restrict__ mp, int64_t mc, int64_t mr, float* __restrict__ svout,
    bool vec_ok, bool stream, const int* gate, int chain0) {
  if (gate && *gate == 0) return;
  const int b = blockIdx.y;
  const int g = blockIdx.x * kThreads + threadIdx.x;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const int k = kk[b];
  if (k >= sc.N) return;
  const int kb = min(K, sc.N - k);
  const uint32_t r = rnd[b];
  const int cnt = min(4, d - e0);
  const bool vec = vec_ok && cnt == 4;
  float yv[4], sv[4];
  float* xb = x + (int64_t)b * xc + e0;
  float* mb = mp ? mp + (int64_t)b * mc + e0 : nullptr;
  load4(y + (int64_t)b * d + e0, cnt, vec, yv);
  float scale = 1.0f;
  if (CACHE_FROM_MEANS) {
    const int cr = crow[b];
    const float4 cc = step_coef(sc, coef, cstep[b]);
    float xcv[4], qcv[4];
    load4(xb + (int64_t)cr * xr, cnt, vec, xcv);
    load4(mqprev + (int64_t)b * qc + (int64_t)cr * qr + e0, cnt, vec, qcv);
#pragma unroll
    for (int c = 0; c < 4; ++c) sv[c] = qcv[c] - cc.x * xcv[c];  // c2_c S_c
    scale = cc.w;
    if (svout) store4(svout + (int64_t)b * d + e0, cnt, vec, sv);
  } else {
    load4(cs + (int64_t)b * d + e0, cnt, vec, sv);
  }
  store4(xb, cnt, vec, yv, stream);
  draft_rows(sc, coef, K, k, kb, (uint32_t)(chain0 + b), r, seed, g, yv, sv, scale, xb, xr, mb, mr,
             cnt, vec, stream);
}

// One thread per chain, at the start of a round:
//  * books the previous round's outcome (tau histogram, steps advanced) and
//    clears it, so that a round is counted exactly once;
//  * counts the chains still active (a ballot per wavefront) into cnt_cur,
//    which gates every later kernel of the round, and clears the next slot;
//  * writes the block size K_b, the steps left, the step index of every
//    target row and sigma_{k+j} for j = 0..K.
__global__ __launch_bounds__(kThreads) void prepare_kernel(
    Sched sc, int B, int K, const int32_t* __restrict__ kk, int32_t* kb, int32_t* left,
    int32_t* step, double* sigma, int32_t* tau, int32_t* adv, int* cnt_cur, int* cnt_next,
    int64_t* hist, int64_t* steps) {
  __shared__ int h[SD_MAX_BLOCK + 2];
  for (int i = threadIdx.x; i < SD_MAX_BLOCK + 2; i += kThreads) h[i] = 0;
  __syncthreads();
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b == 0) *cnt_next = 0;
  const bool in = b < B;
  const int t = in ? tau[b] : 0;
  const int a = in ? adv[b] : 0;
  const int k = in ? kk[b] : sc.N;
  if (in) {
    if (t > 0 && t < SD_MAX_BLOCK + 2) atomicAdd(&h[t], 1);
    tau[b] = 0;
    adv[b] = 0;
  }
  unsigned long long sa = (unsigned long long)a;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sa += __shfl_xor(sa, o);
  const uint64_t act = __ballot(in && k < sc.N);
  if ((threadIdx.x & 63) == 0) {
    if (act) atomicAdd(cnt_cur, __popcll(act));
    if (sa) atomicAdd((unsigned long long*)steps, sa);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < SD_MAX_BLOCK + 2; i += kThreads)
    if (h[i]) atomicAdd((unsigned long long*)&hist[i], (unsigned long long)h[i]);
  if (!in || k >= sc.N) {
    if (in) kb[b] = 0;
    return;
  }
  kb[b] = min(K, sc.N - k);
  left[b] = sc.N - k;
  for (int j = 0; j <= K; ++j) {
    step[(int64_t)b * (K + 1) + j] = min(k + j, sc.N - 1);
    sigma[(int64_t)b * (K + 1) + j] = sched_sigma(sc, min(k + j, sc.N));
  }
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(kThreads) void chains_active_kernel(int B, int split, int N,
                                                                const int32_t* __restrict__ k,
                                                                int* f0, int* f1) {
  __shared__ int any[2];
  if (threadIdx.x < 2) any[threadIdx.x] = 0;
  __syncthreads();
  int a0 = 0, a1 = 0;
  for (int b = threadIdx.x; b < B; b += kThreads) {
    const int on = k[b] < N ? 1 : 0;
    if (b < split)
      a0 |= on;
    else
      a1 |= on;
  }
  if (a0) atomicOr(&any[0], 1);
  if (a1) atomicOr(&any[1], 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    *f0 = any[0];
    *f1 = any[1];
  }
}

__global__ void fill_i64_kernel(int64_t* p, int64_t n, int64_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void philox_words_kernel(uint64_t seed, int n, const uint32_t* ctr, uint32_t* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint4 w = philox(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3], seed);
  out[4 * i] = w.x;
  out[4 * i + 1] = w.y;
  out[4 * i + 2] = w.z;
  out[4 * i + 3] = w.w;
}

__global__ void philox_normals_kernel(uint64_t seed, uint32_t chain, uint32_t rnd, uint32_t c3,
                                      int d, float* out) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const float4 z = normals4(philox((uint32_t)g, chain, rnd, c3, seed));
  for (int c = 0; c < min(4, d - e0); ++c) out[e0 + c] = get4(z, c);
}

}  // namespace

hipError_t init_chains_launch(int B, int d, uint64_t seed, float* y, float* x0, int64_t x0c,
                              hipStream_t s) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  return timed("init_chains", s,
               [&] { init_chains_kernel<<<grid, kThreads, 0, s>>>(d, seed, y, x0, x0c); });
}

static bool draft_vec(int d, sd_stride xs, sd_stride mps, const float* y, const float* x,
                      const float* mp) {
  return (d % 4 == 0) && (xs.chain % 4 == 0) && (xs.row % 4 == 0) && (mps.chain % 4 == 0) &&
         (mps.row % 4 == 0) && aligned16(y) && aligned16(x) && aligned16(mp);
}

hipError_t draft_launch(const Sched& sc, int B, int K, int d, const float* y, const float* cs,
                        const int32_t* k, const uint32_t* rnd, uint64_t seed, float* x,
                        sd_stride xs, float* mp, sd_stride mps, hipStream_t s, const int* gate) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  const bool vec = draft_vec(d, xs, mps, y, x, mp) && aligned16(cs);
  const bool stream = stream_rows((int64_t)B * (K + 1) * d * 4);
  return timed("draft_block", s, [&] {
    draft_kernel<false><<<grid, kThreads, 0, s>>>(sc, nullptr, K, d, y, cs, nullptr, nullptr, nullptr, 0, 0,
                                                  k, rnd, seed, x, xs.chain, xs.row, mp, mps.chain,
                                                  mps.row, nullptr, vec, stream, gate, 0);
  });
}

hipError_t draft_cached_launch(const Sched& sc, const float4* coef, int B, int K, int d,
                               const float* y,
                               const int32_t* crow, const int32_t* cstep, const float* mqprev,
                               sd_stride mqs, const int32_t* k, const uint32_t* rnd,
                               uint64_t seed, float* x, sd_stride xs, float* sv,
                               hipStream_t s, const int* gate, int chain0, int64_t stream_bytes) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  const bool vec = draft_vec(d, xs, sd_stride{d, d}, y, x, sv) && aligned16(mqprev) &&
                   mqs.chain % 4 == 0 && mqs.row % 4 == 0;
  const bool stream = stream_rows(stream_bytes > 0 ? stream_bytes : (int64_t)B * (K + 1) * d * 4);
  return timed("draft_block", s, [&] {
    draft_kernel<true><<<grid, kThreads, 0, s>>>(sc, coef, K, d, y, nullptr, crow, cstep, mqprev,
                                                 mqs.chain, mqs.row, k, rnd, seed, x, xs.chain,
                                                 xs.row, nullptr, 0, 0, sv, vec, stream, gate,
                                                 chain0);
  });
}

hipError_t prepare_launch(const Sched& sc, int B, int K, const int32_t* k, int32_t* kb,
                          int32_t* left, int32_t* step, double* sigma, int32_t* tau,
                          int32_t* adv, int* cnt_cur, int* cnt_next, int64_t* hist,
                          int64_t* steps, hipStream_t s) {
  const int nb = (B + kThreads - 1) / kThreads;
  return timed("prepare_round", s, [&] {
    prepare_kernel<<<nb, kThreads, 0, s>>>(sc, B, K, k, kb, left, step, sigma, tau, adv, cnt_cur,
                                           cnt_next, hist, steps);
  });
}

hipError_t fill_i32_launch(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  fill_i32_kernel<<<(unsigned)nb, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t chains_active_launch(int B, int split, int N, const int32_t* k, int* f0, int* f1,
                                hipStream_t s) {
  chains_active_kernel<<<1, kThreads, 0, s>>>(B, split, N, k, f0, f1);
  return hipGetLastError();
}

hipError_t fill_i64_launch(int64_t* p, int64_t n, int64_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  fill_i64_kernel<<<(unsigned)nb, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t philox_words_launch(uint64_t seed, int n, const uint32_t* ctr, uint32_t* out,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  philox_words_kernel<<<(n + 255) / 256, 256, 0, s>>>(seed, n, ctr, out);
  return hipGetLastError();
}

hipError_t philox_normals_launch(uint64_t seed, uint32_t chain, uint32_t rnd, uint32_t tag,
                                 uint32_t slot, int d, float* out, hipStream_t s) {
  const int ng = (d + 3) / 4;
  philox_normals_kernel<<<(ng + 255) / 256, 256, 0, s>>>(seed, chain, rnd, (tag << 24) | slot,
                                                         d, out);
  return hipGetLastError();
}

}  // namespace sd
