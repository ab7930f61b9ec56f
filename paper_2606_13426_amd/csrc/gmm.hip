// Closed-form Gaussian-mixture target: m^q_n(x) = c1_n x + c2_n s(x) for many
// rows (eq. target-distribution; the B(K+1) states of a round "in parallel").
//
// For a row x at step n with signal level a and s2_m = a^2 var_m + 1 - a^2,
//   logit_m = log w_m - (d/2) log s2_m - (||x||^2 - 2 a x.mu_m + a^2 ||mu_m||^2) / (2 s2_m)
//   r = softmax(logit),  P_m = r_m a / s2_m,  rho = sum_m r_m / s2_m,
//   score = P mu - rho x,   m^q = c1 x + c2 score.
// The two contractions are GEMMs on the matrix cores:
//   gmm_logits:  S = X mu^T   (rows x d by d x M), split over d, with ||x||^2;
//   gmm_softmax: sums the split partials in a fixed order and forms P, rho in float64;
//   gmm_mean:    O = P mu     (rows x M by M x d) with the EM epilogue fused.
// Both GEMMs are "A times B-transposed" over row-major operands whose
// contraction index is contiguous (mu^T is stored at target creation), so one
// tile core serves both: a 64x64 output tile per workgroup, four wavefronts of
// 32x32, k staged through LDS in chunks of 32 and fed to
// v_mfma_f32_32x32x2f32.  Within a chunk, lane half h supplies k = 16h + s to
// MFMA s, so each lane reads its 16 k-values as four 16-byte LDS reads.
#include <vector>

#include "common.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;
constexpr int TILE = 64;
constexpr int KC = 32;
constexpr int LDW = KC + 4;  // LDS row stride in floats (16-byte aligned rows)

typedef float f32x16 __attribute__((ext_vector_type(16)));

struct TileLds {
  float a[TILE * LDW];
  float b[TILE * LDW];
};

// Load rows r0..r0+63, columns k0..k0+31 (< kend) of a row-major matrix into
// two float4 registers per thread: thread t covers rows t/8 and t/8 + 32 and
// columns k0 + 4 (t % 8) .. + 3; out-of-range elements read as zero.
__device__ __forceinline__ void load_chunk(const float* __restrict__ A, int64_t ld, int nrows,
                                           int r0, int k0, int kend, bool vec, float4 (&reg)[2]) {
  const int t = threadIdx.x;
  const int kc = k0 + 4 * (t & 7);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = r0 + (t >> 3) + 32 * h;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < nrows) {
      const float* p = A + (int64_t)r * ld + kc;
      if (vec && kc + 3 < kend) {
        v = *reinterpret_cast<const float4*>(p);
      } else {
        if (kc < kend) v.x = p[0];
        if (kc + 1 < kend) v.y = p[1];
        if (kc + 2 < kend) v.z = p[2];
        if (kc + 3 < kend) v.w = p[3];
      }
    }
    reg[h] = v;
  }
}

__device__ __forceinline__ void store_chunk(float* lds, const float4 (&reg)[2]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h)
    *reinterpret_cast<float4*>(&lds[((t >> 3) + 32 * h) * LDW + 4 * (t & 7)]) = reg[h];
}

__device__ __forceinline__ void mma_chunk(const TileLds& sm, int wr, int wc, f32x16& acc) {
  const int lane = threadIdx.x & 63;
  const int i = lane & 31, h = lane >> 5;
  const float* pa = &sm.a[(wr * 32 + i) * LDW + h * 16];
  const float* pb = &sm.b[(wc * 32 + i) * LDW + h * 16];
  float4 a4[4], b4[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a4[q] = *reinterpret_cast<const float4*>(pa + 4 * q);
    b4[q] = *reinterpret_cast<const float4*>(pb + 4 * q);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].x, b4[q].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].y, b4[q].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].z, b4[q].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].w, b4[q].w, acc, 0, 0, 0);
  }
}

// Accumulate the 64x64 tile (r0, c0) of A[nra][K] * B[nrb][K]^T over k in [kbeg, kend).
// With SQ it also accumulates the float64 squares of the two A rows this thread loads.
template <bool SQ>
__device__ __forceinline__ void nt_tile(TileLds& sm, const float* __restrict__ A, int64_t lda,
                                        int nra, bool veca, const float* __restrict__ Bm,
                                        int64_t ldb, int nrb, bool vecb, int r0, int c0,
                                        int kbeg, int kend, f32x16& acc, double& sq0,
                                        double& sq1) {
  const int w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  float4 ra[2], rb[2];
  load_chunk(A, lda, nra, r0, kbeg, kend, veca, ra);
  load_chunk(Bm, ldb, nrb, c0, kbeg, kend, vecb, rb);
  for (int k0 = kbeg; k0 < kend; k0 += KC) {
    __syncthreads();
    store_chunk(sm.a, ra);
    store_chunk(sm.b, rb);
    if (SQ) {
      sq0 += (double)ra[0].x * ra[0].x + (double)ra[0].y * ra[0].y +
             (double)ra[0].z * ra[0].z + (double)ra[0].w * ra[0].w;
      sq1 += (double)ra[1].x * ra[1].x + (double)ra[1].y * ra[1].y +
             (double)ra[1].z * ra[1].z + (double)ra[1].w * ra[1].w;
    }
    __syncthreads();
    if (k0 + KC < kend) {
      load_chunk(A, lda, nra, r0, k0 + KC, kend, veca, ra);
      load_chunk(Bm, ldb, nrb, c0, k0 + KC, kend, vecb, rb);
    }
    mma_chunk(sm, wr, wc, acc);
  }
}

// Output element v of this lane's 32x32 sub-tile: row and column inside the 64x64 tile.
__device__ __forceinline__ int out_row(int v) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return (w >> 1) * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}
__device__ __forceinline__ int out_col() {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return (w & 1) * 32 + (lane & 31);
}

__global__ __launch_bounds__(kThreads) void gmm_logits_kernel(
    int R, int M, int d, const float* __restrict__ X, int64_t ldx, bool vecx,
    const float* __restrict__ mu, bool vecmu, int ksplit, float* __restrict__ part,
    double* __restrict__ xsq, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  const int r0 = blockIdx.x * TILE, c0 = blockIdx.y * TILE, s = blockIdx.z;
  const int kbeg = s * ksplit, kend = min(d, kbeg + ksplit);
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  double sq[2] = {0.0, 0.0};
  const bool want_sq = blockIdx.y == 0;
  if (want_sq)
    nt_tile<true>(sm, X, ldx, R, vecx, mu, d, M, vecmu, r0, c0, kbeg, kend, acc, sq[0], sq[1]);
  else
    nt_tile<false>(sm, X, ldx, R, vecx, mu, d, M, vecmu, r0, c0, kbeg, kend, acc, sq[0], sq[1]);
  float* ps = part + (int64_t)s * R * M;
  const int col = c0 + out_col();
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = r0 + out_row(v);
    if (row < R && col < M) ps[(int64_t)row * M + col] = acc[v];
  }
  if (want_sq) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      double t = sq[h];
      t += __shfl_xor(t, 1);
      t += __shfl_xor(t, 2);
      t += __shfl_xor(t, 4);
      const int row = r0 + (threadIdx.x >> 3) + 32 * h;
      if ((threadIdx.x & 7) == 0 && row < R) xsq[(int64_t)s * R + row] = t;
    }
  }
}

__global__ __launch_bounds__(kThreads) void gmm_softmax_kernel(
    int R, int M, int d, int S, const float* __restrict__ part, const double* __restrict__ xsq,
    const int32_t* __restrict__ step, Sched sc, const double* __restrict__ var,
    const double* __restrict__ logw, const double* __restrict__ musq, float* __restrict__ P,
    float* __restrict__ rowc, const int* gate) {
  if (gate && *gate == 0) return;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (row >= R) return;
  const int n = step[row];
  const double a = sched_signal(sc, n), a2 = a * a;
  double xs = 0.0;
  for (int s = 0; s < S; ++s) xs += xsq[(int64_t)s * R + row];
  const double hd = 0.5 * (double)d;
  double mx = -INFINITY, sum = 0.0;
  for (int m = lane; m < M; m += 64) {
    double dot = 0.0;
    for (int s = 0; s < S; ++s) dot += (double)part[((int64_t)s * R + row) * M + m];
    const double s2 = a2 * var[m] + 1.0 - a2;
    const double lg = logw[m] - hd * log(s2) - (xs - 2.0 * a * dot + a2 * musq[m]) / (2.0 * s2);
    if (lg > mx) {
      sum = sum * exp(mx - lg) + 1.0;
      mx = lg;
    } else {
      sum += exp(lg - mx);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double omx = __shfl_xor(mx, o), osum = __shfl_xor(sum, o);
    const double nm = fmax(mx, omx);
    const double a1 = mx == -INFINITY ? 0.0 : sum * exp(mx - nm);
    const double a2s = omx == -INFINITY ? 0.0 : osum * exp(omx - nm);
    mx = nm;
    sum = a1 + a2s;
  }
  double rho = 0.0;
  for (int m = lane; m < M; m += 64) {
    double dot = 0.0;
    for (int s = 0; s < S; ++s) dot += (double)part[((int64_t)s * R + row) * M + m];
    const double s2 = a2 * var[m] + 1.0 - a2;
    const double lg = logw[m] - hd * log(s2) - (xs - 2.0 * a * dot + a2 * musq[m]) / (2.0 * s2);
    const double rm = exp(lg - mx) / sum;
    P[(int64_t)row * M + m] = (float)(rm * a / s2);
    rho += rm / s2;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) rho += __shfl_xor(rho, o);
  if (lane == 0) {
    rowc[3 * (int64_t)row + 0] = (float)sched_c1(sc, n);
    rowc[3 * (int64_t)row + 1] = (float)sched_c2(sc, n);
    rowc[3 * (int64_t)row + 2] = (float)rho;
  }
}

__global__ __launch_bounds__(kThreads) void gmm_mean_kernel(
    int R, int M, int d, const float* __restrict__ P, bool vecp, const float* __restrict__ muT,
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ rowc,
    float* __restrict__ mq, int64_t ldq, float* __restrict__ score, int64_t lds,
    const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  const int r0 = blockIdx.x * TILE, c0 = blockIdx.y * TILE;
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  double unused0 = 0.0, unused1 = 0.0;
  nt_tile<false>(sm, P, M, R, vecp, muT, M, d, vecp, r0, c0, 0, M, acc, unused0, unused1);
  const int col = c0 + out_col();
  if (col >= d) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = r0 + out_row(v);
    if (row < R) {
      const float c1 = rowc[3 * (int64_t)row], c2 = rowc[3 * (int64_t)row + 1];
      const float rho = rowc[3 * (int64_t)row + 2];
      const float x = X[(int64_t)row * ldx + col];
      const float sc = acc[v] - rho * x;
      mq[(int64_t)row * ldq + col] = c1 * x + c2 * sc;
      if (score) score[(int64_t)row * lds + col] = sc;
    }
  }
}

struct Plan {
  int S, ksplit;
  size_t off_part, off_xsq, off_p, off_rowc, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Plan make_plan(const Target& t, int R) {
  Plan p{};
  const int tiles = ((R + TILE - 1) / TILE) * ((t.M + TILE - 1) / TILE);
  int S = (512 + tiles - 1) / tiles;
  const int maxS = t.d / 256 > 0 ? t.d / 256 : 1;
  S = S < 1 ? 1 : (S > maxS ? maxS : S);
  int ks = (t.d + S - 1) / S;
  ks = ((ks + KC - 1) / KC) * KC;
  p.ksplit = ks;
  p.S = (t.d + ks - 1) / ks;
  size_t off = 0;
  p.off_part = off;
  off = align256(off + sizeof(float) * (size_t)p.S * R * t.M);
  p.off_xsq = off;
  off = align256(off + sizeof(double) * (size_t)p.S * R);
  p.off_p = off;
  off = align256(off + sizeof(float) * (size_t)R * t.M);
  p.off_rowc = off;
  off = align256(off + sizeof(float) * 3 * (size_t)R);
  p.total = off;
  return p;
}

}  // namespace

size_t target_ws_bytes(const Target& t, int rows) { return make_plan(t, rows).total; }

hipError_t target_mean_launch(const Target& t, int R, const float* x, int64_t ldx,
                              const int32_t* step, float* mq, int64_t ldq, float* score,
                              int64_t lds, void* ws, hipStream_t s, const int* gate) {
  const Plan p = make_plan(t, R);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  double* xsq = reinterpret_cast<double*>(base + p.off_xsq);
  float* P = reinterpret_cast<float*>(base + p.off_p);
  float* rowc = reinterpret_cast<float*>(base + p.off_rowc);
  const bool vecx = (ldx % 4 == 0) && aligned16(x);
  const bool vecmu = (t.d % 4 == 0);
  const bool vecp = (t.M % 4 == 0);
  dim3 g1((R + TILE - 1) / TILE, (t.M + TILE - 1) / TILE, p.S);
  hipError_t e = timed("gmm_logits", s, [&] {
    gmm_logits_kernel<<<g1, kThreads, 0, s>>>(R, t.M, t.d, x, ldx, vecx, t.mu, vecmu, p.ksplit,
                                              part, xsq, gate);
  });
  if (e != hipSuccess) return e;
  const int per = kThreads / 64;
  e = timed("gmm_softmax", s, [&] {
    gmm_softmax_kernel<<<(R + per - 1) / per, kThreads, 0, s>>>(R, t.M, t.d, p.S, part, xsq,
                                                               step, t.sc, t.var, t.logw,
                                                               t.musq, P, rowc, gate);
  });
  if (e != hipSuccess) return e;
  dim3 g2((R + TILE - 1) / TILE, (t.d + TILE - 1) / TILE);
  return timed("gmm_mean", s, [&] {
    gmm_mean_kernel<<<g2, kThreads, 0, s>>>(R, t.M, t.d, P, vecp, t.muT, x, ldx, rowc, mq, ldq,
                                            score, lds, gate);
  });
}

}  // namespace sd
