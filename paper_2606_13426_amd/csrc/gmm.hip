// Closed-form Gaussian-mixture target: m^q_n(x) = c1_n x + c2_n s(x) for many
// rows (eq. target-distribution; the B(K+1) states of a round "in parallel").
//
// For a row x at step n with signal level a and s2_m = a^2 var_m + 1 - a^2,
//   logit_m = log w_m - (d/2) log s2_m - (||x||^2 - 2 a x.mu_m + a^2 ||mu_m||^2) / (2 s2_m)
//   r = softmax(logit),  P_m = r_m a / s2_m,  rho = sum_m r_m / s2_m,
//   score = P mu - rho x,   m^q = c1 x + c2 score.
// The two contractions are GEMMs on the matrix cores:
//   gmm_logits:  S = X mu^T   (rows x d by d x M), split over d, with ||x||^2;
//   gmm_softmax: sums the split partials in a fixed order and forms P, rho (float64 logits);
//   gmm_mean:    O = P mu     (rows x M by M x d) with the EM epilogue fused.
// Both GEMMs are "A times B-transposed" over row-major operands whose
// contraction index is contiguous (mu^T is stored at target creation), on 64x64
// output tiles per workgroup of four wavefronts.  The aligned path (rows
// 16-byte aligned, whole chunks of k) runs them on the bf16 matrix cores
// through exact three-term operand splits (gemm_split.hpp: float32-accurate
// products, mu and mu^T pre-split at target creation).  The unaligned path
// stages k through LDS in chunks of 64 for v_mfma_f32_32x32x2f32 (wavefronts
// of 32x32; lane half h supplies k = 32h + s to MFMA s, eight 16-byte LDS
// reads per lane per chunk).
#include <vector>

#include <type_traits>

#include "bufio.hpp"
#include "common.hpp"
#include "gemm_split.hpp"
#include "philox.hpp"
#include "rows.hpp"
#include "rowsum.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;
constexpr int TILE = 64;
constexpr int KC = 64;
constexpr int LDW = KC + 4;  // LDS row stride in floats (16-byte aligned rows)
constexpr int kFuseSoftmaxMaxM = 256;  // up to this many components the last split does the softmax

typedef float f32x16 __attribute__((ext_vector_type(16)));

struct TileLds {
  float a[TILE * LDW];
  float b[TILE * LDW];
};

// Load rows r0..r0+63, columns k0..k0+63 (< kend) of a row-major matrix into
// four float4 registers per thread: thread t covers rows t/16 + 16 h (h < 4)
// and columns k0 + 4 (t % 16) .. + 3; out-of-range elements read as zero
// (element by element: the unaligned path).
__device__ __forceinline__ void load_chunk(const float* __restrict__ A, int64_t ld, int nrows,
                                           int r0, int k0, int kend, float4 (&reg)[4]) {
  const int t = threadIdx.x;
  const int kc = k0 + 4 * (t & 15);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int r = r0 + (t >> 4) + 16 * h;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < nrows) {
      const float* p = A + (int64_t)r * ld + kc;
      if (kc < kend) v.x = p[0];
      if (kc + 1 < kend) v.y = p[1];
      if (kc + 2 < kend) v.z = p[2];
      if (kc + 3 < kend) v.w = p[3];
    }
    reg[h] = v;
  }
}

// The view of the (at most 64) rows of a tile.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rows(const float* A, int64_t ld, int nrows, int r0) {
  return buf_view(A + (int64_t)r0 * ld, (int64_t)max(0, min(nrows - r0, TILE)) * ld * 4);
}

__device__ __forceinline__ void store_chunk(float* lds, const float4 (&reg)[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 4; ++h)
    *reinterpret_cast<float4*>(&lds[((t >> 4) + 16 * h) * LDW + 4 * (t & 15)]) = reg[h];
}

// One k-chunk of 64 on the matrix cores: lane half h supplies k = 32 h + s to
// MFMA s (s < 32), read as eight 16-byte LDS loads per operand.
__device__ __forceinline__ void mma_chunk(const TileLds& sm, int wr, int wc, f32x16& acc) {
  const int lane = threadIdx.x & 63;
  const int i = lane & 31, h = lane >> 5;
  const float* pa = &sm.a[(wr * 32 + i) * LDW + h * 32];
  const float* pb = &sm.b[(wc * 32 + i) * LDW + h * 32];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    float4 a4[4], b4[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      a4[q] = *reinterpret_cast<const float4*>(pa + 16 * half + 4 * q);
      b4[q] = *reinterpret_cast<const float4*>(pb + 16 * half + 4 * q);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].x, b4[q].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].y, b4[q].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].z, b4[q].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q].w, b4[q].w, acc, 0, 0, 0);
    }
  }
}

// Accumulate the 64x64 tile (r0, c0) of A[nra][K] * B[nrb][K]^T over k in [kbeg, kend),
// starting from the first chunk already loaded into ra, rb (so that a caller
// can issue other loads after the first chunk's: the hardware counts loads in
// order, and the first wait then does not include them).
// With SQ it also accumulates the float64 squares of the four A rows this thread loads.
template <bool SQ>
__device__ __forceinline__ void nt_tile_run(TileLds& sm, const float* __restrict__ A, int64_t lda,
                                            int nra, const float* __restrict__ Bm, int64_t ldb,
                                            int nrb, int r0, int c0, int kbeg, int kend,
                                            float4 (&ra)[4], float4 (&rb)[4], f32x16& acc,
                                            double (&sq)[4]) {
  const int w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  // one chunk: stage it, fetch the next, multiply.  The first chunk is peeled
  // off the loop so that its wait counts only the loads issued before it.
  auto step = [&](int k0) {
    __syncthreads();
    store_chunk(sm.a, ra);
    store_chunk(sm.b, rb);
    if (SQ) {
#pragma unroll
      for (int h = 0; h < 4; ++h)
        sq[h] += (double)ra[h].x * ra[h].x + (double)ra[h].y * ra[h].y +
                 (double)ra[h].z * ra[h].z + (double)ra[h].w * ra[h].w;
    }
    __syncthreads();
    if (k0 + KC < kend) {
      load_chunk(A, lda, nra, r0, k0 + KC, kend, ra);
      load_chunk(Bm, ldb, nrb, c0, k0 + KC, kend, rb);
    }
    mma_chunk(sm, wr, wc, acc);
  };
  if (kbeg < kend) step(kbeg);
  for (int k0 = kbeg + KC; k0 < kend; k0 += KC) step(k0);
}

__device__ __forceinline__ float4 ld4(const float* p, int cnt, bool vec) {
  if (vec && cnt >= 4) return *reinterpret_cast<const float4*>(p);
  return make_float4(cnt > 0 ? p[0] : 0.f, cnt > 1 ? p[1] : 0.f, cnt > 2 ? p[2] : 0.f,
                     cnt > 3 ? p[3] : 0.f);
}

__device__ __forceinline__ void st4(float* p, int cnt, bool vec, float4 v) {
  if (vec && cnt >= 4) {
    *reinterpret_cast<float4*>(p) = v;
  } else {
    if (cnt > 0) p[0] = v.x;
    if (cnt > 1) p[1] = v.y;
    if (cnt > 2) p[2] = v.z;
    if (cnt > 3) p[3] = v.w;
  }
}

__device__ __forceinline__ float comp(const float4& v, int c) {
  return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
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

// The logits GEMM on float32 matrix instructions: the path for rows that are
// not 16-byte aligned or d that is not a whole number of chunks (the aligned
// path is gmm_logits_split_kernel).
__global__ __launch_bounds__(kThreads) void gmm_logits_kernel(
    int R, int M, int d, const float* __restrict__ X, int64_t ldx,
    const float* __restrict__ mu, int ksplit, float* __restrict__ part,
    double* __restrict__ xsq, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  // grid (splits, row tiles, column tiles): the split index varies fastest so
  // that neighbouring workgroups stream neighbouring pieces of the same rows
  const int nsplit = gridDim.x, nrt = gridDim.y;
  const int lin = xcd_tile(nsplit * nrt * gridDim.z);
  const int s = lin % nsplit, rt = (lin / nsplit) % nrt, ct = lin / (nsplit * nrt);
  const int r0 = rt * TILE, c0 = ct * TILE;
  const int kbeg = s * ksplit, kend = min(d, kbeg + ksplit);
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  double sq[4] = {0.0, 0.0, 0.0, 0.0};
  const bool want_sq = ct == 0;
  float4 ra[4], rb[4];
  load_chunk(X, ldx, R, r0, kbeg, kend, ra);
  load_chunk(mu, d, M, c0, kbeg, kend, rb);
  if (want_sq)
    nt_tile_run<true>(sm, X, ldx, R, mu, d, M, r0, c0, kbeg, kend, ra, rb, acc, sq);
  else
    nt_tile_run<false>(sm, X, ldx, R, mu, d, M, r0, c0, kbeg, kend, ra, rb, acc, sq);
  float* ps = part + (int64_t)s * R * M;
  const int col = c0 + out_col();
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = r0 + out_row(v);
    if (row < R && col < M) ps[(int64_t)row * M + col] = acc[v];
  }
  if (want_sq) {
    // the 16 threads of a row are 16 consecutive lanes
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      double t = sq[h];
      t += __shfl_xor(t, 1);
      t += __shfl_xor(t, 2);
      t += __shfl_xor(t, 4);
      t += __shfl_xor(t, 8);
      const int row = r0 + (threadIdx.x >> 4) + 16 * h;
      if ((threadIdx.x & 15) == 0 && row < R) xsq[(int64_t)s * R + row] = t;
    }
  }
}

// The logits GEMM of the aligned float32 path on the bf16 matrix cores
// (gemm_split.hpp): X rows split in registers, mu from its pre-split planes;
// the same outputs and float64 ||x||^2 as gmm_logits_kernel.  The tile is
// kSplitRows = 128 rows of X (two 16-row blocks per wavefront, each B
// fragment read from LDS serving both) by 64 components: half the LDS
// traffic and B loads per output of a 64-row tile, at two wavefronts per
// SIMD (the 32 accumulators and 32 A values per lane need the registers).
static_assert(split::kLdsBytes <= (int)sizeof(TileLds), "the split planes reuse the float32 tile's LDS");
constexpr int kSplitRB = 2, kSplitRows = 64 * kSplitRB;

__global__ __launch_bounds__(kThreads, 2) void gmm_logits_split_kernel(
    int R, int M, int d, const float* __restrict__ X, int64_t ldx,
    const uint16_t* __restrict__ musplit, int ksplit, float* __restrict__ part,
    double* __restrict__ xsq, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  const int nsplit = gridDim.x, nrt = gridDim.y;
  const int lin = xcd_tile(nsplit * nrt * gridDim.z);
  const int s = lin % nsplit, rt = (lin / nsplit) % nrt, ct = lin / (nsplit * nrt);
  const int r0 = rt * kSplitRows, c0 = ct * TILE;
  const int kbeg = s * ksplit, kend = min(d, kbeg + ksplit);
  const size_t plane = (size_t)M * d;
  // rows past R read as zero from the view
  const __amdgpu_buffer_rsrc_t va =
      buf_view(X + (int64_t)r0 * ldx, (int64_t)max(0, min(R - r0, kSplitRows)) * ldx * 4);
  const __amdgpu_buffer_rsrc_t vb[3] = {split::plane_rows(musplit, d, M, c0),
                                        split::plane_rows(musplit + plane, d, M, c0),
                                        split::plane_rows(musplit + 2 * plane, d, M, c0)};
  split::Acc acc[kSplitRB];
  double sq[kSplitRB];
#pragma unroll
  for (int r = 0; r < kSplitRB; ++r) {
    split::zero(acc[r]);
    sq[r] = 0.0;
  }
  split::AChunk ra[kSplitRB];
  split::BChunk rb;
  split::load_b(vb, d, kbeg, rb);
  split::load_a<kSplitRB>(va, ldx, kbeg, ra);
  uint16_t* lds = reinterpret_cast<uint16_t*>(&sm);
  const bool want_sq = ct == 0;
  if (want_sq)
    split::tile_run<true, kSplitRB>(lds, va, ldx, vb, d, kbeg, kend, ra, rb, acc, sq);
  else
    split::tile_run<false, kSplitRB>(lds, va, ldx, vb, d, kbeg, kend, ra, rb, acc, sq);
  float* ps = part + (int64_t)s * R * M;
#pragma unroll
  for (int r = 0; r < kSplitRB; ++r)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int col = c0 + split::out_col(b);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = r0 + split::out_row<kSplitRB>(r, j);
        if (row < R && col < M) ps[(int64_t)row * M + col] = acc[r].c[b][j];
      }
    }
  if (want_sq) {
    // the four lanes of a row are l % 16 + 16 q
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int r = 0; r < kSplitRB; ++r) {
      double t = sq[r];
      t += __shfl_xor(t, 16);
      t += __shfl_xor(t, 32);
      const int row = r0 + 16 * (kSplitRB * w + r) + lane;
      if (lane < 16 && row < R) xsq[(int64_t)s * R + row] = t;
    }
  }
}

// One wavefront per row.  With the per-(step, component) table
// ls[n][m] = (log s2, 1/s2):
//   logit_m = log w_m - (d/2) log s2 - (||x||^2 - 2 a x.mu_m + a^2 ||mu_m||^2) / (2 s2)
// in float64 (kept in registers, up to kMaxPer per lane), then one max
// reduction, one exp per component and one sum reduction.
constexpr int kMaxPer = 16;  // components per lane held in registers (M <= 1024)

template <class TP>
__global__ __launch_bounds__(kThreads) void gmm_softmax_kernel(
    int R, int M, int d, int S, const float* __restrict__ part, const double* __restrict__ xsq,
    const int32_t* __restrict__ step, Sched sc, const double2* __restrict__ ls,
    const double* __restrict__ logw, const double* __restrict__ musq, const float4* __restrict__ coef,
    TP* __restrict__ P, float* __restrict__ rowc, const int* gate) {
  if (gate && *gate == 0) return;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (row >= R) return;
  const int n = step[row];
  const double a = sched_signal(sc, n), a2 = a * a;
  const double2* lsn = ls + (int64_t)n * M;
  double xs = 0.0;
  for (int s = 0; s < S; ++s) xs += xsq[(int64_t)s * R + row];
  const double hd = 0.5 * (double)d;
  // the split partials of x.mu_m, split by split so that the loads of one
  // split (one per component of this lane) are in flight together
  double lg[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) lg[i] = 0.0;
  for (int s = 0; s < S; ++s) {
    const float* ps = part + ((int64_t)s * R + row) * M;
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
      const int m = lane + 64 * i;
      if (m < M) lg[i] += (double)ps[m];
    }
  }
  double mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int m = lane + 64 * i;
    if (m < M) {
      const double2 t = lsn[m];
      lg[i] = logw[m] - hd * t.x - 0.5 * (xs - 2.0 * a * lg[i] + a2 * musq[m]) * t.y;
      mx = fmax(mx, lg[i]);
    } else {
      lg[i] = -INFINITY;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
  float e[kMaxPer];
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    e[i] = lane + 64 * i < M ? __expf((float)(lg[i] - mx)) : 0.0f;
    sum += e[i];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  const double inv = 1.0 / (double)sum;
  double rho = 0.0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int m = lane + 64 * i;
    if (m < M) {
      const double rm = (double)e[i] * inv;
      const double is2 = lsn[m].y;
      const float pm = (float)(rm * a * is2);
      if constexpr (sizeof(TP) == 2)
        P[(int64_t)row * M + m] = __builtin_bit_cast(uint16_t, (__bf16)pm);
      else
        P[(int64_t)row * M + m] = pm;
      rho += rm * is2;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) rho += __shfl_xor(rho, o);
  if (lane == 0) {
    const float4 cf = coef[n];
    rowc[3 * (int64_t)row + 0] = cf.x;
    rowc[3 * (int64_t)row + 1] = cf.y;
    rowc[3 * (int64_t)row + 2] = (float)rho;
  }
}

// The softmax for M % 4 == 0, M <= 4 G: a row is spread over G lanes (G a
// power of two, 16 .. 256) with four consecutive components per lane, so
// every per-component input is one 16-byte load per lane (one per split for
// the logit partials) and a workgroup holds 256 / G rows.  Arithmetic as in
// gmm_softmax_kernel; the max, then the normaliser sum_m e_m together with
// sum_m e_m / s2_m (rho is their ratio), are reduced over the G lanes
// (shuffles within a wavefront, then LDS across the wavefronts of a row).
template <int G>
__device__ __forceinline__ double group_reduce(double v, bool is_max, double* red) {
  constexpr int W = G < 64 ? G : 64;
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) {
    const double u = __shfl_xor(v, o);
    v = is_max ? fmax(v, u) : v + u;
  }
  if constexpr (G > 64) {
    constexpr int NW = G / 64;  // wavefronts per row: the row's are w0 .. w0 + NW - 1
    const int w = threadIdx.x >> 6, w0 = w - w % NW;
    __syncthreads();  // the previous use of red is complete
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    v = red[w0];
#pragma unroll
    for (int i = 1; i < NW; ++i) v = is_max ? fmax(v, red[w0 + i]) : v + red[w0 + i];
  }
  return v;
}

// Both sums of v over the G lanes of a row, as group_reduce.
template <int G>
__device__ __forceinline__ double2 group_sum2(double2 v, double* red) {
  constexpr int W = G < 64 ? G : 64;
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) {
    v.x += __shfl_xor(v.x, o);
    v.y += __shfl_xor(v.y, o);
  }
  if constexpr (G > 64) {
    constexpr int NW = G / 64;
    const int w = threadIdx.x >> 6, w0 = w - w % NW;
    __syncthreads();  // the previous use of red is complete
    if ((threadIdx.x & 63) == 0) {
      red[2 * w] = v.x;
      red[2 * w + 1] = v.y;
    }
    __syncthreads();
    v = make_double2(red[2 * w0], red[2 * w0 + 1]);
#pragma unroll
    for (int i = 1; i < NW; ++i) {
      v.x += red[2 * (w0 + i)];
      v.y += red[2 * (w0 + i) + 1];
    }
  }
  return v;
}

template <int G, class TP>
__global__ __launch_bounds__(kThreads) void gmm_softmax_quad_kernel(
    int R, int M, int d, int S, const float* __restrict__ part, const double* __restrict__ xsq,
    const int32_t* __restrict__ step, Sched sc, const double2* __restrict__ ls,
    const double* __restrict__ logw, const double* __restrict__ musq, const float4* __restrict__ coef,
    TP* __restrict__ P, float* __restrict__ rowc, const int* gate) {
  static_assert(G >= 16 && G <= kThreads && (G & (G - 1)) == 0, "G: a power of two in 16..256");
  if (gate && *gate == 0) return;
  __shared__ double red[2 * (kThreads / 64)];
  constexpr int RPW = kThreads / G;
  const int gl = threadIdx.x % G;
  const int row = blockIdx.x * RPW + (int)threadIdx.x / G;
  const bool on = row < R;
  const int rr = on ? row : R - 1;  // lanes of a missing row follow the last one (no stores)
  const int m0 = 4 * gl;
  const bool has = m0 < M;
  const int mc = has ? m0 : 0;  // loads of lanes past M read component 0 (unused)
  // the partials first (independent of the step), then the step's tables
  double dot[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 8
  for (int sp = 0; sp < S; ++sp) {
    const float4 v = *reinterpret_cast<const float4*>(part + ((int64_t)sp * R + rr) * M + mc);
    dot[0] += (double)v.x;
    dot[1] += (double)v.y;
    dot[2] += (double)v.z;
    dot[3] += (double)v.w;
  }
  double xs = 0.0;
#pragma unroll 8
  for (int sp = 0; sp < S; ++sp) xs += xsq[(int64_t)sp * R + rr];
  const int n = step[rr];
  const double a = sched_signal(sc, n), a2 = a * a, hd = 0.5 * (double)d;
  const double2* lsn = ls + (int64_t)n * M + mc;
  double2 t[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) t[c] = lsn[c];
  const double2 w01 = *reinterpret_cast<const double2*>(logw + mc);
  const double2 w23 = *reinterpret_cast<const double2*>(logw + mc + 2);
  const double2 q01 = *reinterpret_cast<const double2*>(musq + mc);
  const double2 q23 = *reinterpret_cast<const double2*>(musq + mc + 2);
  const double lw[4] = {w01.x, w01.y, w23.x, w23.y}, mq2[4] = {q01.x, q01.y, q23.x, q23.y};
  double lg[4];
  double mx = -INFINITY;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    lg[c] = lw[c] - hd * t[c].x - 0.5 * (xs - 2.0 * a * dot[c] + a2 * mq2[c]) * t[c].y;
    if (has) mx = fmax(mx, lg[c]);
  }
  mx = group_reduce<G>(mx, true, red);
  float e[4];
  float sum = 0.0f;
  double sum_is2 = 0.0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    e[c] = has ? __expf((float)(lg[c] - mx)) : 0.0f;
    sum += e[c];
    sum_is2 += (double)e[c] * t[c].y;
  }
  const double2 tot = group_sum2<G>(make_double2((double)sum, sum_is2), red);
  const double inv = 1.0 / tot.x;
  const double rho = tot.y * inv;
  float pm[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) pm[c] = (float)((double)e[c] * inv * a * t[c].y);
  if (on && has) {
    if constexpr (sizeof(TP) == 2) {
      uint2 pk;
      pk.x = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)pm[0]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)pm[1]) << 16);
      pk.y = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)pm[2]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)pm[3]) << 16);
      *reinterpret_cast<uint2*>(P + (int64_t)row * M + m0) = pk;
    } else {
      *reinterpret_cast<float4*>(P + (int64_t)row * M + m0) = make_float4(pm[0], pm[1], pm[2], pm[3]);
    }
  }
  if (on && gl == 0) {
    const float4 cf = coef[n];
    rowc[3 * (int64_t)row + 0] = cf.x;
    rowc[3 * (int64_t)row + 1] = cf.y;
    rowc[3 * (int64_t)row + 2] = (float)rho;
  }
}

// O = P mu with the EM epilogue on float32 matrix instructions: the path for M
// that is not a whole number of chunks (the aligned path is
// gmm_mean_split_kernel).
__global__ __launch_bounds__(kThreads) void gmm_mean_kernel(
    int R, int M, int d, const float* __restrict__ P, const float* __restrict__ muT,
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ rowc,
    float* __restrict__ mq, int64_t ldq, float* __restrict__ score, int64_t lds,
    const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  __shared__ float rc[3 * TILE];
  const int r0 = blockIdx.x * TILE, c0 = blockIdx.y * TILE;
  const int col = c0 + out_col();
  for (int e = threadIdx.x; e < 3 * TILE; e += kThreads)
    rc[e] = r0 + e / 3 < R ? rowc[3 * (int64_t)r0 + e] : 0.f;
  // the contraction's first operand chunk, then the epilogue's inputs, whose
  // latency then overlaps the contraction
  float4 ra[4], rb[4];
  load_chunk(P, M, R, r0, 0, M, ra);
  load_chunk(muT, M, d, c0, 0, M, rb);
  float xv[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = r0 + out_row(v);
    xv[v] = row < R && col < d ? X[(int64_t)row * ldx + col] : 0.f;
  }
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  double unused[4];
  nt_tile_run<false>(sm, P, M, R, muT, M, d, r0, c0, 0, M, ra, rb, acc, unused);
  if (col >= d) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = r0 + out_row(v);
    if (row < R) {
      const int lr = row - r0;
      const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
      const float sc = acc[v] - rho * xv[v];
      mq[(int64_t)row * ldq + col] = c1 * xv[v] + c2 * sc;
      if (score) score[(int64_t)row * lds + col] = sc;
    }
  }
}

// gmm_mean_kernel's contraction on the bf16 matrix cores (gemm_split.hpp):
// P split in registers, mu^T from its pre-split planes; M a whole number of
// chunks.
__global__ __launch_bounds__(kThreads) void gmm_mean_split_kernel(
    int R, int M, int d, const float* __restrict__ P, const uint16_t* __restrict__ muTs,
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ rowc,
    float* __restrict__ mq, int64_t ldq, float* __restrict__ score, int64_t lds,
    const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  __shared__ float rc[3 * TILE];
  const int r0 = blockIdx.x * TILE, c0 = blockIdx.y * TILE;
  for (int e = threadIdx.x; e < 3 * TILE; e += kThreads)
    rc[e] = r0 + e / 3 < R ? rowc[3 * (int64_t)r0 + e] : 0.f;
  const size_t plane = (size_t)M * d;
  const __amdgpu_buffer_rsrc_t va = tile_rows(P, M, R, r0);
  const __amdgpu_buffer_rsrc_t vb[3] = {split::plane_rows(muTs, M, d, c0),
                                        split::plane_rows(muTs + plane, M, d, c0),
                                        split::plane_rows(muTs + 2 * plane, M, d, c0)};
  split::AChunk sa[1];
  split::BChunk sb;
  split::load_b(vb, M, 0, sb);
  split::load_a<1>(va, M, 0, sa);
  // the epilogue's x, whose latency then overlaps the contraction
  float xv[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int row = r0 + split::out_row<1>(0, j), col = c0 + split::out_col(b);
      xv[b][j] = row < R && col < d ? X[(int64_t)row * ldx + col] : 0.f;
    }
  split::Acc acc[1];
  split::zero(acc[0]);
  double unused[1] = {0.0};
  split::tile_run<false, 1>(reinterpret_cast<uint16_t*>(&sm), va, M, vb, M, 0, M, sa, sb, acc, unused);
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int col = c0 + split::out_col(b);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int lr = split::out_row<1>(0, j), row = r0 + lr;
      if (row < R && col < d) {
        const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
        const float sc = acc[0].c[b][j] - rho * xv[b][j];
        mq[(int64_t)row * ldq + col] = c1 * xv[b][j] + c2 * sc;
        if (score) score[(int64_t)row * lds + col] = sc;
      }
    }
  }
}

// The sampler's second GEMM: O = P mu with the EM epilogue, plus the partial
// log-ratio sums of verification while the tile is on chip.  Rows are
// (chain b, row j) of a [B][K+1][d] block: x row j is draft yhat_{k+j} (row 0
// the state); the draft mean m^p_{k+j} is recomputed from x row j and the
// chain's cache row SV[b] = c2_c S_c exactly as the draft formed it
// (draft_mean, with c2_{k+j} / c2_c from the step tables and the cache step
// cstep[b]).  For j < K and the tile's 64 columns the kernel accumulates, in
// float64 from the float32 values,
//   sum (m^p - m^q)^2   and   sum (yhat_{j+1} - m^p)(m^p - m^q),
// i.e. ||Delta_{j+1}||^2 sigma^2 and Z.Delta sigma^2 (App. A.2), and
// sum (m^p - m^q) G with the residual's G (Alg. 5), into
// lrp[row][column tile][3]; the scan sums the tiles in a fixed order.
// Epilogue layout: the contraction's output is staged in LDS and thread t
// owns columns 4 (t % 16) .. + 3 of tile rows t / 16 + 16 i (i < 4), so a
// wavefront's access to one i is four rows x 256 contiguous bytes; the
// per-row sums are reduced over the 16 lanes of a row (rowsum.hpp).
// VEC: M a whole number of chunks, d a whole number of tiles, rows 16-byte
// aligned; every epilogue access is then an unconditional buffer access
// through a view of the tile's rows (x: 65 rows, the last for the next draft
// of the tile's last row; SV: the tile's chains; m^q: the tile's rows), so
// rows past the block read zero and their stores drop.
// VEC stores m^q with non-temporal stores: of a chain's K + 1 rows the round
// reads back two (the residual's mean and the next cache row).
// VEC also runs the contraction on the bf16 matrix cores from the pre-split
// planes of mu^T (gemm_split.hpp), P split in registers; otherwise it is on
// float32 matrix instructions.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void gmm_mean_lr_kernel(
    int R, int M, int d, int K1, const float* __restrict__ P, const float* __restrict__ muT,
    const uint16_t* __restrict__ muTs, const float* __restrict__ X,
    const float* __restrict__ rowc, const float* __restrict__ SV,
    const int32_t* __restrict__ cstep, const float4* __restrict__ coef, float* __restrict__ mq,
    double* __restrict__ lrp, const uint32_t* __restrict__ rnd, uint64_t seed, const int* gate,
    int chain0) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  __shared__ float rc[3 * TILE];
  __shared__ float cscale[TILE];  // 1 / c2 at each chain's cache step
  // grid (column tiles, row tiles): the column tile varies fastest so that
  // neighbouring workgroups stream neighbouring pieces of the same rows
  const int nct = gridDim.x;
  const int lin = xcd_tile(nct * gridDim.y);
  const int ct = lin % nct, rt = lin / nct;
  const int r0 = rt * TILE, c0 = ct * TILE;
  const int K = K1 - 1, B = R / K1;
  const int cg = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int col = c0 + 4 * cg;
  const int cnt = max(0, min(4, d - col));
  const int b_first = r0 / K1;
  const int nchain = min((min(r0 + TILE, R) - 1) / K1 - b_first + 1, TILE);
  // the contraction's first operand chunk, then every global load of the
  // epilogue, whose latency then overlaps the contraction
  const __amdgpu_buffer_rsrc_t va = tile_rows(P, M, R, r0);
  float4 ra[4], rb[4];
  split::AChunk sa[1];
  split::BChunk sb;
  __amdgpu_buffer_rsrc_t vbs[3];
  if constexpr (VEC) {
    const size_t plane = (size_t)M * d;
#pragma unroll
    for (int p = 0; p < 3; ++p) vbs[p] = split::plane_rows(muTs + p * plane, M, d, c0);
    split::load_b(vbs, M, 0, sb);
    split::load_a<1>(va, M, 0, sa);
  } else {
    load_chunk(P, M, R, r0, 0, M, ra);
    load_chunk(muT, M, d, c0, 0, M, rb);
  }
  // small per-row and per-chain inputs next (the epilogue's coefficients and
  // the rounds of the residual's G), so that their waits exclude the bulk
  // (unconditional loads from clamped indices, unused where out of range)
  const float rcv = rowc[min(3 * (int64_t)r0 + threadIdx.x, 3 * (int64_t)R - 1)];
  constexpr int kGItems = 3;  // ceil(16 x chains / 256): at most 33 chains meet a tile
  uint32_t rn[kGItems];
#pragma unroll
  for (int u = 0; u < kGItems; ++u)
    rn[u] = rnd[min(b_first + (int)((threadIdx.x + kThreads * u) >> 4), B - 1)];
  // (the step index only: the table lookup that depends on it waits until
  // after the contraction, so that no wait here covers the bulk loads)
  const int csi = cstep[min(b_first + (int)threadIdx.x, B - 1)];
  // keep that issue order: the scheduler must not hoist the bulk loads above
  __builtin_amdgcn_sched_barrier(0);
  __amdgpu_buffer_rsrc_t vx, vp, vq;
  if constexpr (VEC) {
    vx = buf_view(X + (int64_t)r0 * d, (int64_t)min(R - r0, TILE + 1) * d * 4);
    vp = buf_view(SV + (int64_t)b_first * d, (int64_t)min(B - b_first, nchain) * d * 4);
    vq = buf_view(mq + (int64_t)r0 * d, (int64_t)min(R - r0, TILE) * d * 4);
  }
  // VEC: the thread's rows are the four consecutive tile rows 4 rg + i, so the
  // next draft of a row is the x of the next one (one extra load for the
  // last) and the rows meet at most two chains (K + 1 >= 4: two cache-row
  // loads); otherwise rows rg + 16 i
  const int lrb = VEC ? 4 * rg : rg, lstep = VEC ? 1 : 16;
  float4 xv[4], yv[4], pv[4];
  float4 xnext, svl, svh;  // VEC: x of the row after the four, cache rows of their chains
  const int bl = (r0 + lrb) / K1;
  if constexpr (VEC) {
    // rows past the block land past a view
#pragma unroll
    for (int i = 0; i < 4; ++i) xv[i] = buf_ld4(vx, (uint32_t)(((lrb + i) * d + col) * 4));
    xnext = buf_ld4(vx, (uint32_t)(((lrb + 4) * d + col) * 4));
    svl = buf_ld4(vp, (uint32_t)(((bl - b_first) * d + col) * 4));
    svh = buf_ld4(vp, (uint32_t)((((r0 + lrb + 3) / K1 - b_first) * d + col) * 4));
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lr = rg + 16 * i, row = r0 + lr;
    const int b = row / K1, j = row - b * K1;
    if constexpr (!VEC) {
      const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
      const float* px = X + (int64_t)row * d + col;
      xv[i] = row < R && cnt > 0 ? ld4(px, cnt, false) : z4;
      const bool dr = row < R && cnt > 0 && j < K1 - 1;
      yv[i] = dr ? ld4(px + d, cnt, false) : z4;
      pv[i] = dr ? ld4(SV + (int64_t)b * d + col, cnt, false) : z4;
    }
  }
  if constexpr (VEC) {
    split::Acc acc[1];
    split::zero(acc[0]);
    double unused[1] = {0.0};
    split::tile_run<false, 1>(reinterpret_cast<uint16_t*>(&sm), va, M, vbs, M, 0, M, sa, sb, acc,
                              unused);
    __syncthreads();  // every wavefront is done with the operand planes
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        sm.a[split::out_row<1>(0, j) * LDW + split::out_col(b)] = acc[0].c[b][j];
  } else {
    f32x16 acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
    double unused[4];
    nt_tile_run<false>(sm, P, M, R, muT, M, d, r0, c0, 0, M, ra, rb, acc, unused);
    __syncthreads();  // every wavefront is done with the operand tiles
    const int cw = out_col();
#pragma unroll
    for (int v = 0; v < 16; ++v) sm.a[out_row(v) * LDW + cw] = acc[v];
  }
  if (threadIdx.x < 3 * TILE) rc[threadIdx.x] = r0 + (int)threadIdx.x / 3 < R ? rcv : 0.f;
  if (threadIdx.x < TILE) cscale[threadIdx.x] = coef[csi].w;
  // G of the residual (RESID stream of each chain's current round) depends
  // only on the chain and the coordinate: drawn once per chain of the tile
  // into sm.b (item e: chain e / 16, coordinates 4 (e % 16) ..)
#pragma unroll
  for (int u = 0; u < kGItems; ++u) {
    const int e = threadIdx.x + kThreads * u;
    if (e < nchain * 16)
      *reinterpret_cast<float4*>(&sm.b[(e >> 4) * LDW + 4 * (e & 15)]) =
          normals4(philox((uint32_t)((c0 >> 2) + (e & 15)), (uint32_t)(chain0 + b_first + (e >> 4)), rn[u],
                          TAG_RESID << 24, seed));
  }
  __syncthreads();
  double s2[4], sz[4], sgd[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    s2[i] = sz[i] = sgd[i] = 0.0;
    const int lr = lrb + lstep * i, row = r0 + lr;
    const int b = row / K1, j = row - b * K1;
    const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
    const float4 ov = *reinterpret_cast<const float4*>(&sm.a[lr * LDW + 4 * cg]);
    const float4 x = xv[i];
    float4 y, sv;
    if constexpr (VEC) {
      y = i < 3 ? xv[i < 3 ? i + 1 : 3] : xnext;
      sv = b == bl ? svl : svh;
    } else {
      y = yv[i];
      sv = pv[i];
    }
    const float4 qv = make_float4(c1 * x.x + c2 * (ov.x - rho * x.x),
                                  c1 * x.y + c2 * (ov.y - rho * x.y),
                                  c1 * x.z + c2 * (ov.z - rho * x.z),
                                  c1 * x.w + c2 * (ov.w - rho * x.w));
    if constexpr (VEC) {
      buf_st4_stream(vq, (uint32_t)((lr * d + col) * 4), qv);
    } else {
      if (row >= R || cnt == 0) continue;
      st4(mq + (int64_t)row * d + col, cnt, false, qv);
    }
    if constexpr (VEC) {
      // all four columns exist; every row is computed and kept only when it
      // is a draft row of the block (a select, no branch: rows past R read
      // zeros and their chain index stays inside sm.b and cscale)
      const bool keep = row < R && j < K1 - 1;
      const float4 gv = *reinterpret_cast<const float4*>(&sm.b[(b - b_first) * LDW + 4 * cg]);
      const float c2s = c2 * cscale[b - b_first];
      double a2 = 0.0, az = 0.0, ag = 0.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float pe = draft_mean(c1, comp(x, e), c2s, comp(sv, e));  // m^p
        const double dd = (double)pe - (double)comp(qv, e);
        const double zz = (double)comp(y, e) - (double)pe;
        a2 = fma(dd, dd, a2);
        az = fma(zz, dd, az);
        ag = fma((double)comp(gv, e), dd, ag);
      }
      s2[i] = keep ? a2 : 0.0;
      sz[i] = keep ? az : 0.0;
      sgd[i] = keep ? ag : 0.0;
    } else if (row < R && j < K1 - 1) {
      const float4 gv = *reinterpret_cast<const float4*>(&sm.b[(b - b_first) * LDW + 4 * cg]);
      const float c2s = c2 * cscale[b - b_first];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < cnt) {
          const float pe = draft_mean(c1, comp(x, e), c2s, comp(sv, e));  // m^p
          const double dd = (double)pe - (double)comp(qv, e);
          const double zz = (double)comp(y, e) - (double)pe;
          s2[i] = fma(dd, dd, s2[i]);
          sz[i] = fma(zz, dd, sz[i]);
          sgd[i] = fma((double)comp(gv, e), dd, sgd[i]);
        }
      }
    }
  }
  // every lane of the group takes part (rows past R and empty columns add zeros)
  const double t2 = reduce_rows16<4>(s2, cg), tz = reduce_rows16<4>(sz, cg),
               tg = reduce_rows16<4>(sgd, cg);
  const int row = r0 + lrb + lstep * row_of<4>(cg);
  if ((cg & 3) == 0 && row < R) {
    double* o = lrp + ((int64_t)row * nct + ct) * 3;
    o[0] = t2;
    o[1] = tz;
    o[2] = tg;
  }
}

// The softmax for M <= 64 (M % 4 == 0): sixteen lanes per row, four
// components per lane read as one float4 per split, four rows per wavefront;
// the same arithmetic as gmm_softmax_kernel with 16-lane reductions.
__global__ __launch_bounds__(kThreads) void gmm_softmax_small_kernel(
    int R, int M, int d, int S, const float* __restrict__ part, const double* __restrict__ xsq,
    const int32_t* __restrict__ step, Sched sc, const double2* __restrict__ ls,
    const double* __restrict__ logw, const double* __restrict__ musq, const float4* __restrict__ coef,
    float* __restrict__ P, float* __restrict__ rowc, const int* gate) {
  if (gate && *gate == 0) return;
  const int q = threadIdx.x & 15;
  const int row = blockIdx.x * (kThreads / 16) + (threadIdx.x >> 4);
  const bool on = row < R;
  const int rr = on ? row : R - 1;  // lanes of a missing row follow the last one (no stores)
  const int n = step[rr];
  const double a = sched_signal(sc, n), a2 = a * a, hd = 0.5 * (double)d;
  double xs = 0.0;
#pragma unroll 8
  for (int sp = 0; sp < S; ++sp) xs += xsq[(int64_t)sp * R + rr];
  const int m0 = 4 * q;
  const bool has = m0 < M;
  double dot[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 8
  for (int sp = 0; sp < S; ++sp) {
    if (has) {
      const float4 v = *reinterpret_cast<const float4*>(part + ((int64_t)sp * R + rr) * M + m0);
      dot[0] += (double)v.x;
      dot[1] += (double)v.y;
      dot[2] += (double)v.z;
      dot[3] += (double)v.w;
    }
  }
  const double2* lsn = ls + (int64_t)n * M;
  double lg[4];
  double mx = -INFINITY;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    lg[c] = -INFINITY;
    if (has) {
      const int m = m0 + c;
      const double2 t = lsn[m];
      lg[c] = logw[m] - hd * t.x - 0.5 * (xs - 2.0 * a * dot[c] + a2 * musq[m]) * t.y;
      mx = fmax(mx, lg[c]);
    }
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
  float e[4];
  float sum = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    e[c] = has ? __expf((float)(lg[c] - mx)) : 0.0f;
    sum += e[c];
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  const double inv = 1.0 / (double)sum;
  double rho = 0.0;
  float pv[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    pv[c] = 0.0f;
    if (has) {
      const double rm = (double)e[c] * inv;
      const double is2 = lsn[m0 + c].y;
      pv[c] = (float)(rm * a * is2);
      rho += rm * is2;
    }
  }
  if (on && has)
    *reinterpret_cast<float4*>(P + (int64_t)row * M + m0) = make_float4(pv[0], pv[1], pv[2], pv[3]);
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) rho += __shfl_xor(rho, o);
  if (q == 0 && on) {
    const float4 cf = coef[n];
    rowc[3 * (int64_t)row + 0] = cf.x;
    rowc[3 * (int64_t)row + 1] = cf.y;
    rowc[3 * (int64_t)row + 2] = (float)rho;
  }
}

struct Plan {
  int S, ksplit;
  size_t off_part, off_xsq, off_p, off_rowc, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Split of the logits GEMM over d: the number of k-chunks per split and the
// number of splits minimise (rounds of workgroups over 512 slots, two per
// compute unit) x (chunks per workgroup), i.e. the critical path, preferring
// fewer splits on ties.
// Buffers for R rows; the split is chosen for plan_rows rows (0: R).
Plan make_plan(const Target& t, int R, int plan_rows = 0) {
  Plan p{};
  // the aligned path's tiles (kSplitRows rows, two workgroups per compute
  // unit); the unaligned kernel takes the same splits
  const int Rp = plan_rows > 0 ? plan_rows : R;
  const int tiles = ((Rp + kSplitRows - 1) / kSplitRows) * ((t.M + TILE - 1) / TILE);
  const int nchunks = (t.d + KC - 1) / KC;
  constexpr int kSlots = 512, kMaxSplits = 32;
  int best_cost = 1 << 30, best_per = nchunks;
  for (int S = 1; S <= kMaxSplits && S <= nchunks; ++S) {
    const int per = (nchunks + S - 1) / S;
    const int splits = (nchunks + per - 1) / per;
    const int cost = ((tiles * splits + kSlots - 1) / kSlots) * per;
    if (cost < best_cost) {
      best_cost = cost;
      best_per = per;
    }
  }
  p.ksplit = best_per * KC;
  p.S = (t.d + p.ksplit - 1) / p.ksplit;
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

// The logits GEMM (buffer path when d is a whole number of chunks, rows are
// aligned and a tile's rows fit 32-bit offsets).
hipError_t logits_launch(const Target& t, const Plan& p, int R, const float* x, int64_t ldx,
                         float* part, double* xsq, hipStream_t s, const int* gate) {
  const bool vec = t.d % KC == 0 && ldx % 4 == 0 && aligned16(x) &&
                   (int64_t)kSplitRows * ldx * 4 < ((int64_t)1 << 31) &&
                   (int64_t)TILE * t.d * 2 < ((int64_t)1 << 31);
  if (vec)
    return launch_timed("gmm_logits", gmm_logits_split_kernel,
                        dim3(p.S, (R + kSplitRows - 1) / kSplitRows, (t.M + TILE - 1) / TILE),
                        dim3(kThreads), s, R, t.M, t.d, x, ldx, t.mu_split, p.ksplit, part, xsq, gate);
  return launch_timed("gmm_logits", gmm_logits_kernel,
                      dim3(p.S, (R + TILE - 1) / TILE, (t.M + TILE - 1) / TILE), dim3(kThreads), s,
                      R, t.M, t.d, x, ldx, t.mu, p.ksplit, part, xsq, gate);
}

}  // namespace

size_t target_ws_bytes(const Target& t, int rows, int plan_rows) {
  return t.prec == SD_BF16 ? target_ws_bytes_bf16(t, rows, plan_rows)
                           : make_plan(t, rows, plan_rows).total;
}

hipError_t gmm_softmax_launch(const Target& t, int R, int S, const float* part, const double* xsq,
                              const int32_t* step, void* P, bool p_bf16, float* rowc,
                              hipStream_t s, const int* gate) {
  if (!p_bf16 && t.M <= 64 && t.M % 4 == 0) {
    const int nbs = (R + kThreads / 16 - 1) / (kThreads / 16);
    return launch_timed("gmm_softmax", gmm_softmax_small_kernel, dim3(nbs), dim3(kThreads), s, R,
                        t.M, t.d, S, part, xsq, step, t.sc, t.ls, t.logw, t.musq, t.coef,
                        static_cast<float*>(P), rowc, gate);
  }
  if (t.M % 4 == 0 && t.M <= 4 * kThreads) {
    // G lanes per row: the smallest power of two >= M / 4, at least 16
    int g = 16;
    while (4 * g < t.M) g <<= 1;
    const int nbq = (R + kThreads / g - 1) / (kThreads / g);
    auto launch = [&](auto gtag) {
      constexpr int GG = decltype(gtag)::value;
      if (p_bf16)
        return launch_timed("gmm_softmax", gmm_softmax_quad_kernel<GG, uint16_t>, dim3(nbq),
                            dim3(kThreads), s, R, t.M, t.d, S, part, xsq, step, t.sc, t.ls, t.logw,
                            t.musq, t.coef, static_cast<uint16_t*>(P), rowc, gate);
      return launch_timed("gmm_softmax", gmm_softmax_quad_kernel<GG, float>, dim3(nbq),
                          dim3(kThreads), s, R, t.M, t.d, S, part, xsq, step, t.sc, t.ls, t.logw,
                          t.musq, t.coef, static_cast<float*>(P), rowc, gate);
    };
    switch (g) {
      case 16: return launch(std::integral_constant<int, 16>{});
      case 32: return launch(std::integral_constant<int, 32>{});
      case 64: return launch(std::integral_constant<int, 64>{});
      case 128: return launch(std::integral_constant<int, 128>{});
      default: return launch(std::integral_constant<int, 256>{});
    }
  }
  const int per = kThreads / 64;
  const int nb = (R + per - 1) / per;
  if (p_bf16)
    return launch_timed("gmm_softmax", gmm_softmax_kernel<uint16_t>, dim3(nb), dim3(kThreads), s, R,
                        t.M, t.d, S, part, xsq, step, t.sc, t.ls, t.logw, t.musq, t.coef,
                        static_cast<uint16_t*>(P), rowc, gate);
  return launch_timed("gmm_softmax", gmm_softmax_kernel<float>, dim3(nb), dim3(kThreads), s, R, t.M,
                      t.d, S, part, xsq, step, t.sc, t.ls, t.logw, t.musq, t.coef,
                      static_cast<float*>(P), rowc, gate);
}

hipError_t target_mean_launch(const Target& t, int R, const float* x, int64_t ldx,
                              const int32_t* step, float* mq, int64_t ldq, float* score,
                              int64_t lds, void* ws, hipStream_t s, const int* gate,
                              int plan_rows) {
  if (t.prec == SD_BF16)
    return target_mean_bf16_launch(t, R, x, ldx, step, mq, ldq, score, lds, ws, s, gate,
                                   plan_rows);
  const Plan p = make_plan(t, R, plan_rows);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  double* xsq = reinterpret_cast<double*>(base + p.off_xsq);
  float* P = reinterpret_cast<float*>(base + p.off_p);
  float* rowc = reinterpret_cast<float*>(base + p.off_rowc);
  hipError_t e = logits_launch(t, p, R, x, ldx, part, xsq, s, gate);
  if (e != hipSuccess) return e;
  e = gmm_softmax_launch(t, R, p.S, part, xsq, step, P, false, rowc, s, gate);
  if (e != hipSuccess) return e;
  dim3 g2((R + TILE - 1) / TILE, (t.d + TILE - 1) / TILE);
  const bool vec = t.M % KC == 0 && t.M < 1 << 22;
  if (vec)
    return launch_timed("gmm_mean", gmm_mean_split_kernel, g2, dim3(kThreads), s, R, t.M, t.d, P,
                        t.muT_split, x, ldx, rowc, mq, ldq, score, lds, gate);
  return launch_timed("gmm_mean", gmm_mean_kernel, g2, dim3(kThreads), s, R, t.M, t.d, P, t.muT, x,
                      ldx, rowc, mq, ldq, score, lds, gate);
}

hipError_t target_mean_lr_launch(const Target& t, int R, int K1, const float* x,
                                 const int32_t* step, float* mq, const float* sv,
                                 const int32_t* cstep, double* lrp, const uint32_t* rnd,
                                 uint64_t seed, void* ws, hipStream_t s, const int* gate,
                                 int plan_rows, int chain0) {
  if (t.prec == SD_BF16)
    return target_mean_lr_bf16_launch(t, R, K1, x, step, mq, sv, cstep, lrp, rnd, seed, ws, s,
                                      gate, plan_rows, chain0);
  const Plan p = make_plan(t, R, plan_rows);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  double* xsq = reinterpret_cast<double*>(base + p.off_xsq);
  float* P = reinterpret_cast<float*>(base + p.off_p);
  float* rowc = reinterpret_cast<float*>(base + p.off_rowc);
  hipError_t e = logits_launch(t, p, R, x, t.d, part, xsq, s, gate);
  if (e != hipSuccess) return e;
  e = gmm_softmax_launch(t, R, p.S, part, xsq, step, P, false, rowc, s, gate);
  if (e != hipSuccess) return e;
  dim3 g2((t.d + TILE - 1) / TILE, (R + TILE - 1) / TILE);
  // the buffer path: whole chunks of M and tiles of d, aligned rows, at least
  // four rows per chain, and 32-bit offsets inside a tile's views
  const bool vec = t.M % KC == 0 && t.d % TILE == 0 && aligned16(x) && aligned16(mq) &&
                   aligned16(sv) && K1 >= 4 &&
                   (int64_t)(TILE + 2) * t.d * 4 < ((int64_t)1 << 31) && t.M < 1 << 22;
  return launch_timed("gmm_mean_lr", vec ? gmm_mean_lr_kernel<true> : gmm_mean_lr_kernel<false>, g2,
                      dim3(kThreads), s, R, t.M, t.d, K1, P, t.muT,
                      t.muT_split, x, rowc, sv, cstep, t.coef, mq, lrp, rnd, seed, gate, chain0);
}

int lr_tiles(const Target& t, int K1) {
  return t.prec == SD_BF16 ? lr_tiles_bf16(t, K1) : (t.d + TILE - 1) / TILE;
}

}  // namespace sd
