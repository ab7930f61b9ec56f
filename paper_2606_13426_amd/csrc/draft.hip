// Free Drafter (Sec. 3.3), chain initialisation and per-round bookkeeping.
//
// The draft recursion is sequential in the draft step i but independent across
// the d coordinates, so each thread owns four consecutive coordinates of one
// chain and walks i = 1..K_b keeping yhat in registers: the state is read once
// and every draft row and draft mean is written once (HBM-bound, no reuse).
#include "common.hpp"
#include "philox.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void load4(const float* p, int cnt, bool vec, float (&v)[4]) {
  if (vec) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = c < cnt ? p[c] : 0.0f;
  }
}

__device__ __forceinline__ void store4(float* p, int cnt, bool vec, const float (&v)[4]) {
  if (vec) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (c < cnt) p[c] = v[c];
  }
}

__global__ __launch_bounds__(kThreads) void init_chains_kernel(int d, uint64_t seed, float* y) {
  const int b = blockIdx.y;
  const int g = blockIdx.x * kThreads + threadIdx.x;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, 0u, TAG_INIT << 24, seed));
  float* p = y + (int64_t)b * d + e0;
  const int cnt = min(4, d - e0);
  for (int c = 0; c < cnt; ++c) p[c] = get4(z, c);
}

__global__ __launch_bounds__(kThreads) void draft_kernel(
    Sched sc, int K, int d, const float* __restrict__ y, const float* __restrict__ cs,
    const int32_t* __restrict__ kk, const uint32_t* __restrict__ rnd, uint64_t seed,
    float* __restrict__ x, int64_t xc, int64_t xr, float* __restrict__ mp, int64_t mc,
    int64_t mr, bool vec_ok, const int* gate) {
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
  float yv[4], sv[4], m[4];
  load4(y + (int64_t)b * d + e0, cnt, vec, yv);
  load4(cs + (int64_t)b * d + e0, cnt, vec, sv);
  float* xb = x + (int64_t)b * xc + e0;
  float* mb = mp + (int64_t)b * mc + e0;
  store4(xb, cnt, vec, yv);
  for (int i = 1; i <= kb; ++i) {
    const int n = k + i - 1;
    const float c1 = (float)sched_c1(sc, n);
    const float c2 = (float)sched_c2(sc, n);
    const float sg = (float)sched_sigma(sc, n);
    const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, r, (TAG_DRAFT << 24) | (uint32_t)i, seed));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      m[c] = c1 * yv[c] + c2 * sv[c];
      yv[c] = m[c] + sg * get4(z, c);
    }
    store4(mb + (int64_t)(i - 1) * mr, cnt, vec, m);
    store4(xb + (int64_t)i * xr, cnt, vec, yv);
  }
  // rows past the valid block repeat the last draft / mean, so every row the
  // target call reads is finite
  for (int i = kb + 1; i <= K; ++i) {
    store4(mb + (int64_t)(i - 1) * mr, cnt, vec, m);
    store4(xb + (int64_t)i * xr, cnt, vec, yv);
  }
}

// One thread per chain: the block size K_b, the steps left, the step index of
// every target row and sigma_{k+j} for j = 0..K; thread 0 also clears this
// round's active-chain counter.
__global__ __launch_bounds__(kThreads) void prepare_kernel(Sched sc, int B, int K,
                                                           const int32_t* __restrict__ kk,
                                                           int32_t* kb, int32_t* left,
                                                           int32_t* step, double* sigma,
                                                           int* cnt_zero, const int* gate) {
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b == 0) *cnt_zero = 0;
  if (gate && *gate == 0) return;
  if (b >= B) return;
  const int k = kk[b];
  kb[b] = k < sc.N ? min(K, sc.N - k) : 0;
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

hipError_t init_chains_launch(int B, int d, uint64_t seed, float* y, hipStream_t s) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  return timed("init_chains", s, [&] { init_chains_kernel<<<grid, kThreads, 0, s>>>(d, seed, y); });
}

hipError_t draft_launch(const Sched& sc, int B, int K, int d, const float* y, const float* cs,
                        const int32_t* k, const uint32_t* rnd, uint64_t seed, float* x,
                        sd_stride xs, float* mp, sd_stride mps, hipStream_t s, const int* gate) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  const bool vec = (d % 4 == 0) && (xs.chain % 4 == 0) && (xs.row % 4 == 0) &&
                   (mps.chain % 4 == 0) && (mps.row % 4 == 0) && aligned16(y) &&
                   aligned16(cs) && aligned16(x) && aligned16(mp);
  return timed("draft_block", s, [&] {
    draft_kernel<<<grid, kThreads, 0, s>>>(sc, K, d, y, cs, k, rnd, seed, x, xs.chain, xs.row,
                                           mp, mps.chain, mps.row, vec, gate);
  });
}

hipError_t prepare_launch(const Sched& sc, int B, int K, const int32_t* k, int32_t* kb,
                          int32_t* left, int32_t* step, double* sigma, int* cnt_zero,
                          hipStream_t s, const int* gate) {
  const int nb = (B + kThreads - 1) / kThreads;
  return timed("prepare_round", s, [&] {
    prepare_kernel<<<nb, kThreads, 0, s>>>(sc, B, K, k, kb, left, step, sigma, cnt_zero, gate);
  });
}

hipError_t fill_i32_launch(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = (n + 255) / 256;
  fill_i32_kernel<<<(unsigned)nb, 256, 0, s>>>(p, n, v);
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
