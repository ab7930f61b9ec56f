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
// contraction index is contiguous (mu^T is stored at target creation), so one
// tile core serves both: a 64x64 output tile per workgroup, four wavefronts of
// 32x32, k staged through LDS in chunks of 64 and fed to
// v_mfma_f32_32x32x2f32.  Within a chunk, lane half h supplies k = 32h + s to
// MFMA s, so each lane reads its 32 k-values as eight 16-byte LDS reads.
#include <vector>

#include "common.hpp"
#include "philox.hpp"

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
// and columns k0 + 4 (t % 16) .. + 3; out-of-range elements read as zero.
__device__ __forceinline__ void load_chunk(const float* __restrict__ A, int64_t ld, int nrows,
                                           int r0, int k0, int kend, bool vec, float4 (&reg)[4]) {
  const int t = threadIdx.x;
  const int kc = k0 + 4 * (t & 15);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int r = r0 + (t >> 4) + 16 * h;
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

// Accumulate the 64x64 tile (r0, c0) of A[nra][K] * B[nrb][K]^T over k in [kbeg, kend).
// With SQ it also accumulates the float64 squares of the four A rows this thread loads.
template <bool SQ>
__device__ __forceinline__ void nt_tile(TileLds& sm, const float* __restrict__ A, int64_t lda,
                                        int nra, bool veca, const float* __restrict__ Bm,
                                        int64_t ldb, int nrb, bool vecb, int r0, int c0,
                                        int kbeg, int kend, f32x16& acc, double (&sq)[4]) {
  const int w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  float4 ra[4], rb[4];
  load_chunk(A, lda, nra, r0, kbeg, kend, veca, ra);
  load_chunk(Bm, ldb, nrb, c0, kbeg, kend, vecb, rb);
  for (int k0 = kbeg; k0 < kend; k0 += KC) {
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
  if (want_sq)
    nt_tile<true>(sm, X, ldx, R, vecx, mu, d, M, vecmu, r0, c0, kbeg, kend, acc, sq);
  else
    nt_tile<false>(sm, X, ldx, R, vecx, mu, d, M, vecmu, r0, c0, kbeg, kend, acc, sq);
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
  double lg[kMaxPer];
  double mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int m = lane + 64 * i;
    lg[i] = -INFINITY;
    if (m < M) {
      double dot = 0.0;
      for (int s = 0; s < S; ++s) dot += (double)part[((int64_t)s * R + row) * M + m];
      const double2 t = lsn[m];
      lg[i] = logw[m] - hd * t.x - 0.5 * (xs - 2.0 * a * dot + a2 * musq[m]) * t.y;
      mx = fmax(mx, lg[i]);
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

__global__ __launch_bounds__(kThreads) void gmm_mean_kernel(
    int R, int M, int d, const float* __restrict__ P, bool vecp, const float* __restrict__ muT,
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
  // the epilogue's inputs are fetched before the contraction so that their
  // latency overlaps it
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
  nt_tile<false>(sm, P, M, R, vecp, muT, M, d, vecp, r0, c0, 0, M, acc, unused);
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

// The sampler's second GEMM: O = P mu with the EM epilogue, plus the partial
// log-ratio sums of verification while the tile is on chip.  Rows are
// (chain b, row j) of a [B][K+1][d] block: x row j is draft yhat_{k+j} (row 0
// the state) and MP [B][K][d] holds m^p_{k+j}.  For j < K and the tile's 64
// columns the kernel accumulates, in float64 from the float32 values,
//   sum (m^p - m^q)^2   and   sum (yhat_{j+1} - m^p)(m^p - m^q),
// i.e. ||Delta_{j+1}||^2 sigma^2 and Z.Delta sigma^2 (App. A.2), and
// sum (m^p - m^q) G with the residual's G (Alg. 5), into
// lrp[row][column tile][3]; the scan sums the tiles in a fixed order.  The
// contraction's output is staged in LDS so that the epilogue runs
// row-contiguous (four threads per row, sixteen columns each).
__global__ __launch_bounds__(kThreads) void gmm_mean_lr_kernel(
    int R, int M, int d, int K1, const float* __restrict__ P, bool vecp,
    const float* __restrict__ muT, const float* __restrict__ X, const float* __restrict__ rowc,
    const float* __restrict__ MP, float* __restrict__ mq, double* __restrict__ lrp, bool vecd,
    const uint32_t* __restrict__ rnd, uint64_t seed, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ TileLds sm;
  __shared__ float rc[3 * TILE];
  // grid (column tiles, row tiles): the column tile varies fastest so that
  // neighbouring workgroups stream neighbouring pieces of the same rows
  const int nct = gridDim.x;
  const int lin = xcd_tile(nct * gridDim.y);
  const int ct = lin % nct, rt = lin / nct;
  const int r0 = rt * TILE, c0 = ct * TILE;
  // Every global load of the epilogue is issued first, together with the
  // first operand chunk, so that one memory latency covers them all: thread t
  // owns row r0 + t/4 and columns c0 + 16 (t % 4) .. + 15 in the epilogue.
  const int lr = threadIdx.x >> 2, cb = 16 * (threadIdx.x & 3);
  const int row = r0 + lr;
  const int b = row / K1, j = row - b * K1;
  const bool has_row = row < R;
  const bool has_draft = has_row && j < K1 - 1;
  float xv[16], yv[16], pv[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int col = c0 + cb + 4 * q;
    const int cnt = col < d ? min(4, d - col) : 0;
    const bool vec = vecd && cnt == 4;
    const float* px = X + (int64_t)row * d + col;
    const float* pp = MP + ((int64_t)b * (K1 - 1) + j) * d + col;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      xv[4 * q + c] = 0.f;
      yv[4 * q + c] = 0.f;
      pv[4 * q + c] = 0.f;
    }
    if (has_row && cnt > 0) {
      if (vec) {
        const float4 a = *reinterpret_cast<const float4*>(px);
        xv[4 * q] = a.x; xv[4 * q + 1] = a.y; xv[4 * q + 2] = a.z; xv[4 * q + 3] = a.w;
      } else {
        for (int c = 0; c < cnt; ++c) xv[4 * q + c] = px[c];
      }
    }
    if (has_draft && cnt > 0) {
      if (vec) {
        const float4 a = *reinterpret_cast<const float4*>(px + d);
        yv[4 * q] = a.x; yv[4 * q + 1] = a.y; yv[4 * q + 2] = a.z; yv[4 * q + 3] = a.w;
        const float4 m = *reinterpret_cast<const float4*>(pp);
        pv[4 * q] = m.x; pv[4 * q + 1] = m.y; pv[4 * q + 2] = m.z; pv[4 * q + 3] = m.w;
      } else {
        for (int c = 0; c < cnt; ++c) {
          yv[4 * q + c] = px[d + c];
          pv[4 * q + c] = pp[c];
        }
      }
    }
  }
  for (int e = threadIdx.x; e < 3 * TILE; e += kThreads)
    rc[e] = r0 + e / 3 < R ? rowc[3 * (int64_t)r0 + e] : 0.f;
  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
  double unused[4];
  nt_tile<false>(sm, P, M, R, vecp, muT, M, d, vecp, r0, c0, 0, M, acc, unused);
  __syncthreads();  // every wavefront is done with the operand tiles
  {
    const int cw = out_col();
#pragma unroll
    for (int v = 0; v < 16; ++v) sm.a[out_row(v) * LDW + cw] = acc[v];
  }
  // G of the residual (RESID stream of each chain's current round) depends
  // only on the chain and the coordinate: draw it once per chain of the tile
  // into sm.b (at most 64 chains x 64 coordinates).
  const int b_first = r0 / K1;
  const int nchain = min((min(r0 + TILE, R) - 1) / K1 - b_first + 1, TILE);
  for (int e = threadIdx.x; e < nchain * 16; e += kThreads) {
    const int cl = e >> 4, gq = e & 15;
    const int bb = b_first + cl;
    const float4 z = normals4(philox((uint32_t)((c0 >> 2) + gq), (uint32_t)bb, rnd[bb],
                                     TAG_RESID << 24, seed));
    *reinterpret_cast<float4*>(&sm.b[cl * LDW + 4 * gq]) = z;
  }
  __syncthreads();
  double s2 = 0.0, sz = 0.0, sgd = 0.0;
  if (has_row) {
    const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
    const float* gz = &sm.b[(b - b_first) * LDW];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int cl = cb + 4 * q, col = c0 + cl;
      const int cnt = col < d ? min(4, d - col) : 0;
      float qv[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float x = xv[4 * q + c];
        qv[c] = c1 * x + c2 * (sm.a[lr * LDW + cl + c] - rho * x);
      }
      float* pq = mq + (int64_t)row * d + col;
      if (vecd && cnt == 4) {
        *reinterpret_cast<float4*>(pq) = make_float4(qv[0], qv[1], qv[2], qv[3]);
      } else {
        for (int c = 0; c < cnt; ++c) pq[c] = qv[c];
      }
      if (has_draft) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          if (c < cnt) {
            const double dd = (double)pv[4 * q + c] - (double)qv[c];
            const double zz = (double)yv[4 * q + c] - (double)pv[4 * q + c];
            s2 = fma(dd, dd, s2);
            sz = fma(zz, dd, sz);
            sgd = fma((double)gz[cl + c], dd, sgd);
          }
        }
      }
    }
  }
  s2 += __shfl_xor(s2, 1);
  s2 += __shfl_xor(s2, 2);
  sz += __shfl_xor(sz, 1);
  sz += __shfl_xor(sz, 2);
  sgd += __shfl_xor(sgd, 1);
  sgd += __shfl_xor(sgd, 2);
  if ((threadIdx.x & 3) == 0 && has_row) {
    double* o = lrp + ((int64_t)row * nct + ct) * 3;
    o[0] = s2;
    o[1] = sz;
    o[2] = sgd;
  }
}

struct Plan {
  int S, ksplit;
  size_t off_part, off_xsq, off_p, off_rowc, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Split of the logits GEMM over d: the number of k-chunks per split and the
// number of splits minimise (workgroups per CU, rounded up) x (chunks per
// workgroup), i.e. the critical path over 256 compute units, preferring fewer
// splits on ties.
Plan make_plan(const Target& t, int R) {
  Plan p{};
  const int tiles = ((R + TILE - 1) / TILE) * ((t.M + TILE - 1) / TILE);
  const int nchunks = (t.d + KC - 1) / KC;
  int best_cost = 1 << 30, best_per = nchunks;
  for (int S = 1; S <= 8 && S <= nchunks; ++S) {
    const int per = (nchunks + S - 1) / S;
    const int splits = (nchunks + per - 1) / per;
    const int cost = ((tiles * splits + 255) / 256) * per;
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

}  // namespace

size_t target_ws_bytes(const Target& t, int rows) {
  return t.prec == SD_BF16 ? target_ws_bytes_bf16(t, rows) : make_plan(t, rows).total;
}

hipError_t gmm_softmax_launch(const Target& t, int R, int S, const float* part, const double* xsq,
                              const int32_t* step, void* P, bool p_bf16, float* rowc,
                              hipStream_t s, const int* gate) {
  const int per = kThreads / 64;
  const int nb = (R + per - 1) / per;
  return timed("gmm_softmax", s, [&] {
    if (p_bf16)
      gmm_softmax_kernel<<<nb, kThreads, 0, s>>>(R, t.M, t.d, S, part, xsq, step, t.sc, t.ls,
                                                 t.logw, t.musq, t.coef,
                                                 static_cast<uint16_t*>(P), rowc, gate);
    else
      gmm_softmax_kernel<<<nb, kThreads, 0, s>>>(R, t.M, t.d, S, part, xsq, step, t.sc, t.ls,
                                                 t.logw, t.musq, t.coef, static_cast<float*>(P),
                                                 rowc, gate);
  });
}

hipError_t target_mean_launch(const Target& t, int R, const float* x, int64_t ldx,
                              const int32_t* step, float* mq, int64_t ldq, float* score,
                              int64_t lds, void* ws, hipStream_t s, const int* gate) {
  if (t.prec == SD_BF16)
    return target_mean_bf16_launch(t, R, x, ldx, step, mq, ldq, score, lds, ws, s, gate);
  const Plan p = make_plan(t, R);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  double* xsq = reinterpret_cast<double*>(base + p.off_xsq);
  float* P = reinterpret_cast<float*>(base + p.off_p);
  float* rowc = reinterpret_cast<float*>(base + p.off_rowc);
  const bool vecx = (ldx % 4 == 0) && aligned16(x);
  const bool vecmu = (t.d % 4 == 0);
  const bool vecp = (t.M % 4 == 0);
  dim3 g1(p.S, (R + TILE - 1) / TILE, (t.M + TILE - 1) / TILE);
  hipError_t e = timed("gmm_logits", s, [&] {
    gmm_logits_kernel<<<g1, kThreads, 0, s>>>(R, t.M, t.d, x, ldx, vecx, t.mu, vecmu, p.ksplit,
                                              part, xsq, gate);
  });
  if (e != hipSuccess) return e;
  e = gmm_softmax_launch(t, R, p.S, part, xsq, step, P, false, rowc, s, gate);
  if (e != hipSuccess) return e;
  dim3 g2((R + TILE - 1) / TILE, (t.d + TILE - 1) / TILE);
  return timed("gmm_mean", s, [&] {
    gmm_mean_kernel<<<g2, kThreads, 0, s>>>(R, t.M, t.d, P, vecp, t.muT, x, ldx, rowc, mq, ldq,
                                            score, lds, gate);
  });
}

hipError_t target_mean_lr_launch(const Target& t, int R, int K1, const float* x,
                                 const int32_t* step, float* mq, const float* mp, double* lrp,
                                 const uint32_t* rnd, uint64_t seed, void* ws, hipStream_t s,
                                 const int* gate) {
  if (t.prec == SD_BF16)
    return target_mean_lr_bf16_launch(t, R, K1, x, step, mq, mp, lrp, rnd, seed, ws, s, gate);
  const Plan p = make_plan(t, R);
  char* base = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(base + p.off_part);
  double* xsq = reinterpret_cast<double*>(base + p.off_xsq);
  float* P = reinterpret_cast<float*>(base + p.off_p);
  float* rowc = reinterpret_cast<float*>(base + p.off_rowc);
  const bool vecd = (t.d % 4 == 0) && aligned16(x) && aligned16(mq) && aligned16(mp);
  const bool vecp = (t.M % 4 == 0);
  dim3 g1(p.S, (R + TILE - 1) / TILE, (t.M + TILE - 1) / TILE);
  hipError_t e = timed("gmm_logits", s, [&] {
    gmm_logits_kernel<<<g1, kThreads, 0, s>>>(R, t.M, t.d, x, t.d, vecd, t.mu, t.d % 4 == 0,
                                              p.ksplit, part, xsq, gate);
  });
  if (e != hipSuccess) return e;
  e = gmm_softmax_launch(t, R, p.S, part, xsq, step, P, false, rowc, s, gate);
  if (e != hipSuccess) return e;
  dim3 g2((t.d + TILE - 1) / TILE, (R + TILE - 1) / TILE);
  return timed("gmm_mean_lr", s, [&] {
    gmm_mean_lr_kernel<<<g2, kThreads, 0, s>>>(R, t.M, t.d, K1, P, vecp, t.muT, x, rowc, mp, mq,
                                               lrp, vecd, rnd, seed, gate);
  });
}

int lr_tiles(const Target& t) {
  return t.prec == SD_BF16 ? lr_tiles_bf16(t) : (t.d + TILE - 1) / TILE;
}

}  // namespace sd
