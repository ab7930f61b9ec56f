// Gaussian-mixture target with bf16 operands on the matrix cores (float32
// accumulation), for the large configurations: the same three steps as the
// float32 path (logits GEMM split over d, float64 softmax, mean GEMM with the
// EM epilogue) on tiles of v_mfma_f32_32x32x16_bf16.
//   gmm_logits_bf16: S = X mu^T, X float32 rounded to bf16 on staging, mu bf16;
//                    ||x||^2 from the unrounded float32 values (float64
//                    sums; on 256 x 256 tiles of float32 partials of four);
//                    256 x 256 tiles (gemm_bf16_wide.hpp) when d is a whole
//                    number of chunks and rows are aligned, else 128 x 128;
//   softmax:         the float32 path's kernels, writing P in bf16;
//   gmm_mean_bf16 / gmm_mean_lr_bf16: O = P mu (mu^T stored as bf16) and the
//                    epilogue in float32, the latter with the verification
//                    partial sums of the sampler (as the float32 path).
// The mean GEMMs' 128 x 128 accumulator tile is handed to the epilogue
// through LDS in two passes of 64 columns, each over the operand buffers'
// storage.
#include "bufio.hpp"
#include "common.hpp"
#include "gemm_bf16.hpp"
#include "gemm_bf16_wide.hpp"
#include "philox.hpp"
#include "rows.hpp"
#include "rowsum.hpp"

namespace sd {
namespace {

using namespace bf16;

constexpr int LDO = 68;         // staging row stride in floats (one 64-column pass)
constexpr int kMaxChains = 65;  // chains that 128 rows of [B][K+1] can touch (K+1 >= 2)

static_assert(sizeof(float) * TM * LDO <= sizeof(OperandLds), "staging must fit one operand buffer");
static_assert(sizeof(float) * kMaxChains * LDO <= sizeof(OperandLds), "G must fit one operand buffer");

template <bool VEC>
__global__ __launch_bounds__(kThreads, 2) void gmm_logits_bf16_kernel(
    int R, int M, int d, const float* __restrict__ X, int64_t ldx,
    const uint16_t* __restrict__ mu, int ksplit, float* __restrict__ part,
    double* __restrict__ xsq, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ OperandLds sm[2];
  // grid (column tiles, row tiles, splits).  Each XCD takes a contiguous range
  // of the tile order (column tile fastest, split slowest): the column tiles
  // that share a block of X run together and read it once into that XCD's L2,
  // and one XCD keeps to one k-range of mu while it walks the row tiles.
  const int nct = gridDim.x, nrt = gridDim.y;
  const int lin = xcd_tile(nct * nrt * gridDim.z);
  const int ct = lin % nct, rt = (lin / nct) % nrt, s = lin / (nct * nrt);
  const int r0 = rt * TM, c0 = ct * TN;
  const int kbeg = s * ksplit, kend = min(d, kbeg + ksplit);
  f32x16 acc[2][2];
  zero(acc);
  double sq[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  const bool want_sq = ct == 0;
  if (want_sq)
    tile<true, VEC>(sm, X, ldx, R, mu, d, M, r0, c0, kbeg, kend, acc, sq);
  else
    tile<false, VEC>(sm, X, ldx, R, mu, d, M, r0, c0, kbeg, kend, acc, sq);
  float* ps = part + (int64_t)s * R * M;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int col = c0 + out_col(qb);
    if (col >= M) continue;
#pragma unroll
    for (int qa = 0; qa < 2; ++qa)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = r0 + out_row(qa, v);
        if (row < R) ps[(int64_t)row * M + col] = acc[qa][qb][v];
      }
  }
  if (want_sq) {
    // the 16 threads that loaded a row are 16 consecutive lanes
#pragma unroll
    for (int h = 0; h < 8; ++h) {
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

// The logits GEMM on 256 x 256 tiles (one workgroup per compute unit), for
// the aligned case: d a whole number of chunks, rows of X 16-byte aligned.
// Grid and tile order as gmm_logits_bf16_kernel.  The ||x||^2 partials of a
// row are taken by one of the column tiles: a thread's loaded rows h (< 8)
// go to column tile h % nct, so the column tiles (that run side by side)
// share the work instead of column tile 0 doing all of it.
__global__ __launch_bounds__(bf16w::kThreads, 2) void gmm_logits_bf16_wide_kernel(
    int R, int M, int d, const float* __restrict__ X, int64_t ldx,
    const uint16_t* __restrict__ mu, int ksplit, float* __restrict__ part,
    double* __restrict__ xsq, const int* gate) {
  using namespace bf16w;
  if (gate && *gate == 0) return;
  __shared__ bf16w::OperandLds sm[2];
  const int nct = gridDim.x, nrt = gridDim.y;
  const int lin = xcd_tile(nct * nrt * gridDim.z);
  const int ct = lin % nct, rt = (lin / nct) % nrt, s = lin / (nct * nrt);
  const int r0 = rt * WT, c0 = ct * WT;
  const int kbeg = s * ksplit, kend = min(d, kbeg + ksplit);
  bf16w::f32x16 acc[4][2];
  bf16w::zero(acc);
  double sq[8];
#pragma unroll
  for (int h = 0; h < 8; ++h) sq[h] = 0.0;
  const __amdgpu_buffer_rsrc_t va = bf16w::tile_view(X, ldx, R, r0);
  const __amdgpu_buffer_rsrc_t vb = bf16w::tile_view(mu, (int64_t)d, M, c0);
  uint32_t sqmask = 0;
#pragma unroll
  for (int h = 0; h < 8; ++h) sqmask |= (h % nct == ct ? 1u : 0u) << h;
  bf16w::tile<true, float>(sm, va, ldx, vb, d, kbeg, kend, acc, sq, sqmask);
  float* ps = part + (int64_t)s * R * M;
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int col = c0 + bf16w::out_col(qb);
    if (col >= M) continue;
#pragma unroll
    for (int qa = 0; qa < 4; ++qa)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = r0 + bf16w::out_row(qa, v);
        if (row < R) ps[(int64_t)row * M + col] = acc[qa][qb][v];
      }
  }
  // the 16 threads that loaded a row are 16 consecutive lanes
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    if (!(sqmask >> h & 1u)) continue;
    double t = sq[h];
    t += __shfl_xor(t, 1);
    t += __shfl_xor(t, 2);
    t += __shfl_xor(t, 4);
    t += __shfl_xor(t, 8);
    const int row = r0 + (threadIdx.x >> 4) + 32 * h;
    if ((threadIdx.x & 15) == 0 && row < R) xsq[(int64_t)s * R + row] = t;
  }
}

// Tile of a (column tiles) x (row tiles) grid for the mean GEMM.  Its B
// operand is the slice of mu^T of the column tile, re-read by every row tile,
// so each XCD owns a contiguous eighth of the column tiles and walks all row
// tiles over them (the slices stay in its L2); inside an XCD consecutive
// workgroups take consecutive column tiles of one row tile (shared P rows).
__device__ __forceinline__ void col_major_xcd(int nct, int nrt, int& ct, int& rt) {
  const int L = blockIdx.x + gridDim.x * blockIdx.y;
  if (nct % 8 != 0) {
    ct = L % nct;
    rt = L / nct;
    return;
  }
  const int per = nct / 8, i = L / 8;
  ct = (L % 8) * per + i % per;
  rt = i / per;
}

// Pass p of the epilogue stages accumulator blocks qb = p of every wavefront:
// tile columns 64 wc + 32 p + (0..31) go to staging columns 32 wc + (0..31).
__device__ __forceinline__ void stage(float* stg, const f32x16 (&acc)[2][2], int p) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int sc = 32 * (w & 1) + (lane & 31);
#pragma unroll
  for (int qa = 0; qa < 2; ++qa)
#pragma unroll
    for (int v = 0; v < 16; ++v) stg[out_row(qa, v) * LDO + sc] = acc[qa][p][v];
}

// Epilogue layout.  Thread t owns staging columns 4 cg .. 4 cg + 3 (cg = t % 16)
// of tile rows rg + 16 i (rg = t / 16, i < 8): tile columns
// 64 (cg / 8) + 32 p + 4 (cg % 8) .. + 3 in pass p.  A wavefront's load of one
// i covers four rows x 2 x 128 contiguous bytes, so global accesses are
// whole cache lines.
__device__ __forceinline__ int epi_col(int cg, int p) { return 64 * (cg >> 3) + 32 * p + 4 * (cg & 7); }

__device__ __forceinline__ void load_rc(float* rc, const float* __restrict__ rowc, int r0, int R) {
  for (int e = threadIdx.x; e < 3 * TM; e += kThreads)
    rc[e] = r0 + e / 3 < R ? rowc[3 * (int64_t)r0 + e] : 0.f;
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

// Public target call: m^q = c1 x + c2 (O - rho x) (and the score if asked).
template <bool VEC>
__global__ __launch_bounds__(kThreads, 2) void gmm_mean_bf16_kernel(
    int R, int M, int d, const uint16_t* __restrict__ P,
    const uint16_t* __restrict__ muT, const float* __restrict__ X, int64_t ldx, bool vecx,
    const float* __restrict__ rowc, float* __restrict__ mq, int64_t ldq, bool vecq,
    float* __restrict__ score, int64_t lds, bool vecs, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ OperandLds sm[2];
  __shared__ float rc[3 * TM];
  const int nct = gridDim.x;
  int ct, rt;
  col_major_xcd(nct, gridDim.y, ct, rt);
  const int r0 = rt * TM, c0 = ct * TN;
  load_rc(rc, rowc, r0, R);
  f32x16 acc[2][2];
  zero(acc);
  double unused[8];
  tile<false, VEC>(sm, P, M, R, muT, M, d, r0, c0, 0, M, acc, unused);
  float* stg = reinterpret_cast<float*>(&sm[0]);
  const int cg = threadIdx.x & 15, rg = threadIdx.x >> 4;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    __syncthreads();  // the operand tiles (p = 0) or the previous pass are consumed
    stage(stg, acc, p);
    __syncthreads();
    const int col = c0 + epi_col(cg, p);
    const int cnt = min(4, d - col);
    if (cnt <= 0) continue;
    float4 xv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = r0 + rg + 16 * i;
      xv[i] = row < R ? ld4(X + (int64_t)row * ldx + col, cnt, vecx) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int lr = rg + 16 * i, row = r0 + lr;
      if (row >= R) continue;
      const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
      const float4 ov = *reinterpret_cast<const float4*>(&stg[lr * LDO + 4 * cg]);
      const float4 x = xv[i];
      const float4 sv = make_float4(ov.x - rho * x.x, ov.y - rho * x.y, ov.z - rho * x.z,
                                    ov.w - rho * x.w);
      st4(mq + (int64_t)row * ldq + col, cnt, vecq,
          make_float4(c1 * x.x + c2 * sv.x, c1 * x.y + c2 * sv.y, c1 * x.z + c2 * sv.z,
                      c1 * x.w + c2 * sv.w));
      if (score) st4(score + (int64_t)row * lds + col, cnt, vecs, sv);
    }
  }
}

// The aligned epilogue of the sampler's mean GEMM (d a whole number of tiles,
// rows 16-byte aligned, at least eight rows per chain for the cache-row
// loads: K + 1 >= 8).  Thread t owns staging columns 4 (t % 16) .. + 3 of the
// eight consecutive tile rows 8 (t / 16) .. + 7, so the next draft yhat_{j+1}
// of a row is the x of the thread's next row (one extra load for the last),
// and the eight rows meet at most two chains (two cache-row loads).  Every
// global load of both passes is issued before the first store (stores and
// loads share one in-order counter), through buffer views of the tile's rows
// (rows past the block read zero; their stores drop).  m^q goes out with
// non-temporal stores: the round reads back two of a chain's K + 1 rows.
__device__ __forceinline__ void mean_lr_epilogue_vec(
    float* stg, float* gz, const float* cscale, const float* rc, const f32x16 (&acc)[2][2], int R,
    int d, int K1, int r0, int c0, int ct, int nct, int b_first, int nchain,
    const float* __restrict__ X, const float* __restrict__ SV, float* __restrict__ mq,
    double* __restrict__ lrp, const uint32_t* __restrict__ rnd, uint64_t seed) {
  const int cg = threadIdx.x & 15, lr0 = 8 * (threadIdx.x >> 4);
  const int B = R / K1;
  const __amdgpu_buffer_rsrc_t vx = buf_view(X + (int64_t)r0 * d, (int64_t)min(R - r0, TM + 1) * d * 4);
  const __amdgpu_buffer_rsrc_t vs = buf_view(SV + (int64_t)b_first * d, (int64_t)min(B - b_first, nchain) * d * 4);
  const __amdgpu_buffer_rsrc_t vq = buf_view(mq + (int64_t)r0 * d, (int64_t)min(R - r0, TM) * d * 4);
  const int bl = (r0 + lr0) / K1, bh = min((r0 + lr0 + 7) / K1, B);  // chains of the eight rows
  // the chains' rounds for the G draws (items e = t + 256 u: chain e / 16)
  constexpr int kMaxChainsVec = TM / 8 + 2;  // chains that 128 rows can touch with K + 1 >= 8
  constexpr int kGItems = (kMaxChainsVec * 16 + kThreads - 1) / kThreads;
  uint32_t rn[kGItems];
#pragma unroll
  for (int u = 0; u < kGItems; ++u)
    rn[u] = rnd[min(b_first + (int)((threadIdx.x + kThreads * u) >> 4), B - 1)];
  float4 xv[2][9], sl[2], sh[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int col = c0 + epi_col(cg, p);
#pragma unroll
    for (int i = 0; i < 9; ++i) xv[p][i] = buf_ld4(vx, (uint32_t)(((lr0 + i) * d + col) * 4));
    sl[p] = buf_ld4(vs, (uint32_t)(((bl - b_first) * d + col) * 4));
    sh[p] = buf_ld4(vs, (uint32_t)(((bh - b_first) * d + col) * 4));
  }
  double t2 = 0.0, tz = 0.0, tg = 0.0;  // this lane's row (see reduce_rows16), both passes
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    __syncthreads();  // the operand tiles (p = 0) or the previous pass are consumed
    stage(stg, acc, p);
#pragma unroll
    for (int u = 0; u < kGItems; ++u) {
      const int e = threadIdx.x + kThreads * u;
      if (e < nchain * 16) {
        const int tcol = c0 + epi_col(e & 15, p);
        *reinterpret_cast<float4*>(&gz[(e >> 4) * LDO + 4 * (e & 15)]) =
            normals4(philox((uint32_t)(tcol >> 2), (uint32_t)(b_first + (e >> 4)), rn[u],
                            TAG_RESID << 24, seed));
      }
    }
    __syncthreads();
    const int col = c0 + epi_col(cg, p);
    double s2[8], sz[8], sgd[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s2[i] = sz[i] = sgd[i] = 0.0;
      const int lr = lr0 + i, row = r0 + lr;
      const int b = row / K1, j = row - b * K1;
      const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
      const float4 ov = *reinterpret_cast<const float4*>(&stg[lr * LDO + 4 * cg]);
      const float4 x = xv[p][i], y = xv[p][i + 1];
      const float4 qv = make_float4(c1 * x.x + c2 * (ov.x - rho * x.x),
                                    c1 * x.y + c2 * (ov.y - rho * x.y),
                                    c1 * x.z + c2 * (ov.z - rho * x.z),
                                    c1 * x.w + c2 * (ov.w - rho * x.w));
      buf_st4_stream(vq, (uint32_t)((lr * d + col) * 4), qv);
      // every row is computed and kept only when it is a draft row of the
      // block (a select: rows past R read zeros and their chain index stays
      // inside gz and cscale)
      const bool keep = row < R && j < K1 - 1;
      const float4 sv = b == bl ? sl[p] : sh[p];
      const float4 gv = *reinterpret_cast<const float4*>(&gz[(b - b_first) * LDO + 4 * cg]);
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
    }
    t2 += reduce_rows16<8>(s2, cg);
    tz += reduce_rows16<8>(sz, cg);
    tg += reduce_rows16<8>(sgd, cg);
  }
  const int row = r0 + lr0 + row_of<8>(cg);
  if ((cg & 1) == 0 && row < R) {
    double* o = lrp + ((int64_t)row * nct + ct) * 3;
    o[0] = t2;
    o[1] = tz;
    o[2] = tg;
  }
}

// The sampler's mean GEMM on its [B][K+1][d] block with the verification
// partials: for draft rows j < K and this tile's columns, float64 sums of
// (m^p - m^q)^2, (yhat_{j+1} - m^p)(m^p - m^q) and G (m^p - m^q), G the
// residual's normals of the chain's round, into lrp[row][column tile][3].
// m^p is recomputed from x row j and the chain's cache row SV[b] as the draft
// formed it (draft_mean; c2_{k+j} / c2_c from the tables and cstep[b]).
template <bool VEC>
__global__ __launch_bounds__(kThreads, 2) void gmm_mean_lr_bf16_kernel(
    int R, int M, int d, int K1, const uint16_t* __restrict__ P,
    const uint16_t* __restrict__ muT, const float* __restrict__ X, const float* __restrict__ rowc,
    const float* __restrict__ SV, const int32_t* __restrict__ cstep,
    const float4* __restrict__ coef, float* __restrict__ mq, double* __restrict__ lrp, bool vecd,
    const uint32_t* __restrict__ rnd, uint64_t seed, const int* gate) {
  if (gate && *gate == 0) return;
  __shared__ OperandLds sm[2];
  __shared__ float rc[3 * TM];
  __shared__ float cscale[kMaxChains];  // 1 / c2 at each chain's cache step
  const int nct = gridDim.x;
  int ct, rt;
  col_major_xcd(nct, gridDim.y, ct, rt);
  const int r0 = rt * TM, c0 = ct * TN;
  load_rc(rc, rowc, r0, R);
  f32x16 acc[2][2];
  zero(acc);
  double unused[8];
  // the cache steps of the tile's chains, fetched before the contraction (an
  // unconditional load from a clamped index; the table lookup that depends on
  // it comes after, so that no early wait stalls the workgroup)
  const int B = R / K1;
  const int csi = cstep[min(r0 / K1 + (int)threadIdx.x, B - 1)];
  tile<false, VEC>(sm, P, M, R, muT, M, d, r0, c0, 0, M, acc, unused);
  float* stg = reinterpret_cast<float*>(&sm[0]);
  float* gz = reinterpret_cast<float*>(&sm[1]);
  const int cg = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int b_first = r0 / K1;
  const int nchain = min((min(r0 + TM, R) - 1) / K1 - b_first + 1, kMaxChains);
  if ((int)threadIdx.x < nchain) cscale[threadIdx.x] = coef[csi].w;
  if constexpr (VEC) {
    mean_lr_epilogue_vec(stg, gz, cscale, rc, acc, R, d, K1, r0, c0, ct, nct, b_first, nchain, X,
                         SV, mq, lrp, rnd, seed);
    return;
  }
  double t2 = 0.0, tz = 0.0, tg = 0.0;  // this lane's row (see reduce_rows16), both passes
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    __syncthreads();
    stage(stg, acc, p);
    // G of this pass's columns for every chain of the tile, four coordinates
    // (one Philox block) per item, at the staging column of those coordinates
    for (int e = threadIdx.x; e < nchain * 16; e += kThreads) {
      const int cl = e >> 4, gq = e & 15;
      const int bb = b_first + cl;
      const int tcol = c0 + epi_col(gq, p);
      const float4 z = normals4(philox((uint32_t)(tcol >> 2), (uint32_t)bb, rnd[bb],
                                       TAG_RESID << 24, seed));
      *reinterpret_cast<float4*>(&gz[cl * LDO + 4 * gq]) = z;
    }
    __syncthreads();
    const int col = c0 + epi_col(cg, p);
    const int cnt = max(0, min(4, d - col));
    // every global load of the pass first, then the arithmetic
    float4 xv[8], yv[8], pv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = r0 + rg + 16 * i;
      const int b = row / K1, j = row - b * K1;
      const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
      const float* px = X + (int64_t)row * d + col;
      xv[i] = row < R && cnt > 0 ? ld4(px, cnt, vecd) : z4;
      const bool dr = row < R && cnt > 0 && j < K1 - 1;
      yv[i] = dr ? ld4(px + d, cnt, vecd) : z4;
      pv[i] = dr ? ld4(SV + (int64_t)b * d + col, cnt, vecd) : z4;  // the chain's cache row
    }
    double s2[8], sz[8], sgd[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s2[i] = sz[i] = sgd[i] = 0.0;
      const int lr = rg + 16 * i, row = r0 + lr;
      if (row >= R || cnt == 0) continue;
      const int b = row / K1, j = row - b * K1;
      const float c1 = rc[3 * lr], c2 = rc[3 * lr + 1], rho = rc[3 * lr + 2];
      const float4 ov = *reinterpret_cast<const float4*>(&stg[lr * LDO + 4 * cg]);
      const float4 x = xv[i];
      const float4 qv = make_float4(c1 * x.x + c2 * (ov.x - rho * x.x),
                                    c1 * x.y + c2 * (ov.y - rho * x.y),
                                    c1 * x.z + c2 * (ov.z - rho * x.z),
                                    c1 * x.w + c2 * (ov.w - rho * x.w));
      st4(mq + (int64_t)row * d + col, cnt, vecd, qv);
      if (j < K1 - 1) {
        const float4 gv = *reinterpret_cast<const float4*>(&gz[(b - b_first) * LDO + 4 * cg]);
        const float c2s = c2 * cscale[b - b_first];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (e < cnt) {
            const float pe = draft_mean(c1, comp(x, e), c2s, comp(pv[i], e));  // m^p
            const double dd = (double)pe - (double)comp(qv, e);
            const double zz = (double)comp(yv[i], e) - (double)pe;
            s2[i] = fma(dd, dd, s2[i]);
            sz[i] = fma(zz, dd, sz[i]);
            sgd[i] = fma((double)comp(gv, e), dd, sgd[i]);
          }
        }
      }
    }
    // every lane of the group takes part (rows past R and empty columns add zeros)
    t2 += reduce_rows16<8>(s2, cg);
    tz += reduce_rows16<8>(sz, cg);
    tg += reduce_rows16<8>(sgd, cg);
  }
  const int row = r0 + rg + 16 * row_of<8>(cg);
  if ((cg & 1) == 0 && row < R) {
    double* o = lrp + ((int64_t)row * nct + ct) * 3;
    o[0] = t2;
    o[1] = tz;
    o[2] = tg;
  }
}

struct Plan {
  int S, ksplit;
  bool wide;  // the logits GEMM may run on 256 x 256 tiles (d a whole number of chunks)
  size_t off_part, off_xsq, off_p, off_rowc, total;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Split of the logits GEMM over d, chosen as in the float32 path: the
// chunks per split and the splits minimise (workgroups per slot, rounded up)
// x (chunks per workgroup), over 256 slots of one 256 x 256 workgroup per
// compute unit when d is a whole number of chunks, else over 512 slots of two
// 128 x 128 workgroups per compute unit.
Plan make_plan(const Target& t, int R) {
  Plan p{};
  p.wide = t.d % KC == 0;
  const int tm = p.wide ? bf16w::WT : TM, tn = p.wide ? bf16w::WT : TN;
  const int slots = p.wide ? 256 : 512;
  const int tiles = ((R + tm - 1) / tm) * ((t.M + tn - 1) / tn);
  const int nchunks = (t.d + KC - 1) / KC;
  int best_cost = 1 << 30, best_per = nchunks;
  for (int S = 1; S <= 8 && S <= nchunks; ++S) {
    const int per = (nchunks + S - 1) / S;
    const int splits = (nchunks + per - 1) / per;
    const int cost = ((tiles * splits + slots - 1) / slots) * per;
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
  off = align256(off + sizeof(uint16_t) * (size_t)R * t.M);
  p.off_rowc = off;
  off = align256(off + sizeof(float) * 3 * (size_t)R);
  p.total = off;
  return p;
}

struct Bufs {
  float* part;
  double* xsq;
  uint16_t* P;
  float* rowc;
};

Bufs carve(const Plan& p, void* ws) {
  char* base = static_cast<char*>(ws);
  return Bufs{reinterpret_cast<float*>(base + p.off_part),
              reinterpret_cast<double*>(base + p.off_xsq),
              reinterpret_cast<uint16_t*>(base + p.off_p),
              reinterpret_cast<float*>(base + p.off_rowc)};
}

hipError_t logits_and_softmax(const Target& t, const Plan& p, const Bufs& w, int R,
                              const float* x, int64_t ldx, bool vecx, const int32_t* step,
                              hipStream_t s, const int* gate) {
  dim3 g1((t.M + TN - 1) / TN, (R + TM - 1) / TM, p.S);
  // the buffer-load path: whole chunks of k and 32-bit offsets inside a tile
  const bool vec = vecx && t.d % KC == 0 && ldx < (int64_t)1 << 22 && t.d < 1 << 22;
  const bool wide = vec && p.wide && ldx < (int64_t)1 << 21 && t.d < 1 << 21;
  hipError_t e;
  if (wide)
    e = launch_timed("gmm_logits_bf16", gmm_logits_bf16_wide_kernel,
                     dim3((t.M + bf16w::WT - 1) / bf16w::WT, (R + bf16w::WT - 1) / bf16w::WT, p.S),
                     dim3(bf16w::kThreads), s, R, t.M, t.d, x, ldx, t.mu16, p.ksplit, w.part, w.xsq,
                     gate);
  else
    e = launch_timed("gmm_logits_bf16", vec ? gmm_logits_bf16_kernel<true> : gmm_logits_bf16_kernel<false>,
                     g1, dim3(kThreads), s, R, t.M, t.d, x, ldx, t.mu16, p.ksplit, w.part, w.xsq,
                     gate);
  if (e != hipSuccess) return e;
  return gmm_softmax_launch(t, R, p.S, w.part, w.xsq, step, w.P, true, w.rowc, s, gate);
}

}  // namespace

size_t target_ws_bytes_bf16(const Target& t, int rows) { return make_plan(t, rows).total; }

hipError_t target_mean_bf16_launch(const Target& t, int R, const float* x, int64_t ldx,
                                   const int32_t* step, float* mq, int64_t ldq, float* score,
                                   int64_t lds, void* ws, hipStream_t s, const int* gate) {
  const Plan p = make_plan(t, R);
  const Bufs w = carve(p, ws);
  const bool vecx = (ldx % 4 == 0) && aligned16(x);
  hipError_t e = logits_and_softmax(t, p, w, R, x, ldx, vecx, step, s, gate);
  if (e != hipSuccess) return e;
  const bool vecq = (ldq % 4 == 0) && aligned16(mq);
  const bool vecs = score && (lds % 4 == 0) && aligned16(score);
  dim3 g2((t.d + TN - 1) / TN, (R + TM - 1) / TM);
  return timed("gmm_mean_bf16", s, [&] {
    if (t.M % KC == 0)
      gmm_mean_bf16_kernel<true><<<g2, kThreads, 0, s>>>(R, t.M, t.d, w.P, t.muT16, x, ldx, vecx,
                                                         w.rowc, mq, ldq, vecq, score, lds, vecs,
                                                         gate);
    else
      gmm_mean_bf16_kernel<false><<<g2, kThreads, 0, s>>>(R, t.M, t.d, w.P, t.muT16, x, ldx, vecx,
                                                          w.rowc, mq, ldq, vecq, score, lds, vecs,
                                                          gate);
  });
}

hipError_t target_mean_lr_bf16_launch(const Target& t, int R, int K1, const float* x,
                                      const int32_t* step, float* mq, const float* sv,
                                      const int32_t* cstep, double* lrp, const uint32_t* rnd,
                                      uint64_t seed, void* ws, hipStream_t s, const int* gate) {
  const Plan p = make_plan(t, R);
  const Bufs w = carve(p, ws);
  const bool vecd = (t.d % 4 == 0) && aligned16(x) && aligned16(mq) && aligned16(sv);
  hipError_t e = logits_and_softmax(t, p, w, R, x, t.d, vecd, step, s, gate);
  if (e != hipSuccess) return e;
  dim3 g2((t.d + TN - 1) / TN, (R + TM - 1) / TM);
  // the buffer path: whole chunks of M, whole tiles of d, aligned rows, at
  // least eight rows per chain, 32-bit offsets inside a tile's views
  const bool vec = t.M % KC == 0 && t.d % TN == 0 && vecd && K1 >= 8 &&
                   (int64_t)(TM + 2) * t.d * 4 < ((int64_t)1 << 31);
  return launch_timed("gmm_mean_lr_bf16",
                      vec ? gmm_mean_lr_bf16_kernel<true> : gmm_mean_lr_bf16_kernel<false>, g2,
                      dim3(kThreads), s, R, t.M, t.d, K1, w.P, t.muT16, x, w.rowc, sv, cstep, t.coef,
                      mq, lrp, vecd, rnd, seed, gate);
}

int lr_tiles_bf16(const Target& t) { return (t.d + TN - 1) / TN; }

}  // namespace sd
