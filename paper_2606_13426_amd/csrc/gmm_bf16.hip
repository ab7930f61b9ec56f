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
//                    partial sums of the sampler (as the float32 path); the
//                    sampler's call with at least 512 components runs on the
//                    chain-aligned 288 x 256 tiles of gemm_bf16_big.hpp.
// The mean GEMMs' 128 x 128 accumulator tile is handed to the epilogue
// through LDS in two passes of 64 columns, each over the operand buffers'
// storage.
#include "bufio.hpp"
#include "common.hpp"
#include "gemm_bf16.hpp"
#include "gemm_bf16_big.hpp"
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
    double* __restrict__ lrp, const uint32_t* __restrict__ rnd, uint64_t seed, int chain0) {
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
            normals4(philox((uint32_t)(tcol >> 2), (uint32_t)(chain0 + b_first + (e >> 4)), rn[u],
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
    const uint32_t* __restrict__ rnd, uint64_t seed, const int* gate, int chain0) {
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
                         SV, mq, lrp, rnd, seed, chain0);
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
      const float4 z = normals4(philox((uint32_t)(tcol >> 2), (uint32_t)(chain0 + bb), rnd[bb],
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

// The sampler's mean GEMM on the 288-row tiles of gemm_bf16_big.hpp whose
// rows are whole chains: tile rt holds the CT chains rt CT .. (CT K1 <= 288
// rows), so no chain straddles two tiles.  Same outputs as
// gmm_mean_lr_bf16_kernel (m^q, and the float64 partials of ||m^p - m^q||^2,
// (yhat_{j+1} - m^p).(m^p - m^q) and G.(m^p - m^q) per draft row and column
// tile).  The epilogue works on the accumulators where they are: each lane
// holds four consecutive columns of one row per block, so x and m^q move as
// 16-byte row segments, the next draft comes from the neighbouring lane, G
// and the chains' cache rows are staged once in LDS, and the per-row sums are
// combined over the four lanes of a row and the column wavefronts in a fixed
// order.  Needs d % TC == 0, M % KC == 0, aligned rows and CT <= kChains.
template <class T>
struct BigMean {
  static constexpr int QW = T::TC / 64;  // column wavefronts
  // LDS stride of a chain's G and cache rows in floats: four more than a row,
  // so the two or three chains of a 16-lane row group fall on different banks
  static constexpr int GS = T::TC + 4;
  // chains whose G and cache rows fit the operand buffers beside the partials
  static constexpr int kFit = (int)((2 * sizeof(typename T::Lds) - QW * bf16b::TR * 3 * sizeof(double)) /
                                    (2 * sizeof(float) * GS));
  static constexpr int kChains = kFit < 56 ? kFit : 56;
};

// Within a 16-lane row of the accumulator layout lane l holds tile row
// 16 rb + l % 16: the row below is lane l + 1 (DPP row_shl:1), and for lane 15
// it is lane 0 of the next block (DPP row_shr:15 of that block's values).
__device__ __forceinline__ float next_row1(float cur, float nxt) {
  const int fix = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, nxt), 0x11f, 0xf, 0xf, false);
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(fix, __builtin_bit_cast(int, cur), 0x101,
                                                               0xf, 0xf, false));
}
__device__ __forceinline__ float4 next_row(float4 cur, float4 nxt) {
  return make_float4(next_row1(cur.x, nxt.x), next_row1(cur.y, nxt.y), next_row1(cur.z, nxt.z),
                     next_row1(cur.w, nxt.w));
}

// Lane l receives lane l ^ 8's value (DPP row_ror:8 inside each 16-lane row).
__device__ __forceinline__ float xchg8_1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xf,
                                                               0xf, false));
}
__device__ __forceinline__ float4 xchg8(float4 v) {
  return make_float4(xchg8_1(v.x), xchg8_1(v.y), xchg8_1(v.z), xchg8_1(v.w));
}

__device__ __forceinline__ int big_tile_order(int nrt, int nct, int& rt) {
  // each XCD takes a contiguous range of column tiles (its slice of mu^T stays
  // in its L2) and walks the row tiles fastest inside it
  const int lin = xcd_tile(nrt * nct);
  rt = lin % nrt;
  return lin / nrt;
}

template <class T>
__global__ __launch_bounds__(T::kThreads, T::TC == 128 ? 2 : 1) void gmm_mean_lr_bf16_big_kernel(
    int R, int M, int d, int K1, int CT, const uint16_t* __restrict__ P,
    const uint16_t* __restrict__ muT, const float* __restrict__ X, const float* __restrict__ rowc,
    const float* __restrict__ SV, const int32_t* __restrict__ cstep,
    const float4* __restrict__ coef, float* __restrict__ mq, double* __restrict__ lrp,
    const uint32_t* __restrict__ rnd, uint64_t seed, const int* gate, int chain0) {
  using bf16b::CB;
  using bf16b::RB;
  using bf16b::TR;
  constexpr int TC = T::TC, QW = BigMean<T>::QW, NCH = BigMean<T>::kChains, GS = BigMean<T>::GS;
  if (gate && *gate == 0) return;
  __shared__ typename T::Lds sm[2];
  __shared__ float rc[3 * TR];
  __shared__ float cscale[NCH];
  __shared__ uint32_t crnd[NCH];
  const int B = R / K1;
  const int nrt = (B + CT - 1) / CT, nct = d / TC;
  int rt;
  const int ct = big_tile_order(nrt, nct, rt);
  const int b_first = rt * CT;
  const int nchain = min(CT, B - b_first);
  const int r0 = b_first * K1, rows = nchain * K1, c0 = ct * TC;
  for (int e = threadIdx.x; e < 3 * TR; e += T::kThreads)
    rc[e] = e < 3 * rows ? rowc[3 * (int64_t)r0 + e] : 0.f;
  if ((int)threadIdx.x < nchain) {
    crnd[threadIdx.x] = rnd[b_first + threadIdx.x];
    cscale[threadIdx.x] = coef[cstep[b_first + threadIdx.x]].w;  // 1 / c2 at the cache step
  }
  bf16b::f32x4 acc[RB][CB];
  bf16b::zero(acc);
  T::run(sm, buf_view(muT + (int64_t)c0 * M, (int64_t)TC * M * 2), M,
         buf_view(P + (int64_t)r0 * M, (int64_t)rows * M * 2), M, 0, M, acc);
  const __amdgpu_buffer_rsrc_t vx = buf_view(X + (int64_t)r0 * d, (int64_t)min(R - r0, rows + 1) * d * 4);
  const __amdgpu_buffer_rsrc_t vq = buf_view(mq + (int64_t)r0 * d, (int64_t)rows * d * 4);
  const __amdgpu_buffer_rsrc_t vs = buf_view(SV + (int64_t)b_first * d, (int64_t)nchain * d * 4);
  // HBM accesses of the epilogue cover whole 128-byte lines: lane l moves 16
  // bytes of row 8 h + l % 8 of a row block at column 16 ((l / 8) % 2) + 4
  // (l / 16) of a pair of column blocks, 8 rows x 128 bytes per instruction.
  // Lanes l and l ^ 8 then swap one value per pair (xchg8) to reach the
  // accumulator layout (row l % 16, four columns of each block), and back for
  // the stores of m^q.
  const int lane = threadIdx.x & 63, b3 = (lane >> 3) & 1;
  const int row7 = T::out_row(0) - (lane & 15) + (lane & 7);
  const int colp = c0 + T::out_col(0) - 4 * ((lane >> 4) & 3) + 16 * b3 + 4 * ((lane >> 4) & 3);
  auto load_x = [&](int rb, float4 (&raw)[CB]) {
#pragma unroll
    for (int pr = 0; pr < CB / 2; ++pr) {
      raw[2 * pr] = buf_ld4(vx, (uint32_t)(((row7 + 16 * rb) * d + colp + 32 * pr) * 4));
      raw[2 * pr + 1] = buf_ld4(vx, (uint32_t)(((row7 + 16 * rb + 8) * d + colp + 32 * pr) * 4));
    }
  };
  auto to_acc_layout = [&](const float4 (&raw)[CB], float4 (&xv)[CB]) {
#pragma unroll
    for (int pr = 0; pr < CB / 2; ++pr) {
      const float4 lo = raw[2 * pr], hi = raw[2 * pr + 1];
      const float4 recv = xchg8(b3 ? lo : hi);
      xv[2 * pr] = b3 ? recv : lo;
      xv[2 * pr + 1] = b3 ? hi : recv;
    }
  };
  // x is prefetched two row blocks ahead (the first ones before G is drawn)
  float4 xraw[RB][CB], xr[RB][CB];
  load_x(0, xraw[0]);
  load_x(1, xraw[1]);
  // G of the tile's chains and columns (four normals per Philox block) and the
  // chains' cache rows, into the (now free) operand buffers: gz, svs
  // [chain][column], GS floats per chain; then the per-row partial sums of
  // each column wavefront
  float* gz = reinterpret_cast<float*>(&sm[0]);
  float* svs = gz + NCH * GS;
  double* part = reinterpret_cast<double*>(svs + NCH * GS);
  for (int e = threadIdx.x; e < nchain * (TC / 4); e += T::kThreads) {
    const int cl = e / (TC / 4), g4 = e % (TC / 4);
    const float4 z = normals4(philox((uint32_t)((c0 >> 2) + g4), (uint32_t)(chain0 + b_first + cl), crnd[cl],
                                     TAG_RESID << 24, seed));
    *reinterpret_cast<float4*>(&gz[cl * GS + 4 * g4]) = z;
    *reinterpret_cast<float4*>(&svs[cl * GS + 4 * g4]) = buf_ld4(vs, (uint32_t)((cl * d + c0 + 4 * g4) * 4));
  }
  __syncthreads();
  const int wc = T::col_wave(), sub = (threadIdx.x >> 4) & 3;
  to_acc_layout(xraw[0], xr[0]);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (rb + 2 < RB) load_x(rb + 2, xraw[rb + 2]);
    if (rb + 1 < RB) to_acc_layout(xraw[rb + 1], xr[rb + 1]);
    const float4 (&xa)[CB] = xr[rb];
    const int lr = T::out_row(rb);  // tile row
    // rows past the tile's chains read zeros and store nothing (buffer views)
    const int b = min(lr / K1, NCH - 1), j = lr - (lr / K1) * K1;
    const bool keep = lr < rows && j < K1 - 1;
    const float c1 = rc[3 * min(lr, TR - 1)], c2 = rc[3 * min(lr, TR - 1) + 1],
                rho = rc[3 * min(lr, TR - 1) + 2];
    const float c2s = c2 * cscale[b];
    double a2 = 0.0, az = 0.0, ag = 0.0;
#pragma unroll
    for (int pr = 0; pr < CB / 2; ++pr) {
      float4 qs[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int cb = 2 * pr + h;
        const int tcol = T::out_col(cb);
        // the next draft of each row is the next row's x: lane l + 1 of the
        // same 16-lane row (DPP row shift), and for lane 15 row 0 of the next
        // block (lane 0 of its 16-lane row); past the wavefront's last block a
        // load
        const float4 y = rb + 1 < RB ? next_row(xa[cb], xr[rb + 1 < RB ? rb + 1 : rb][cb])
                                     : buf_ld4(vx, (uint32_t)(((lr + 1) * d + c0 + tcol) * 4));
        const bf16b::f32x4 o = acc[rb][cb];
        const float4 x = xa[cb];
        const float4 sv = *reinterpret_cast<const float4*>(&svs[b * GS + tcol]);
        const float4 qv = make_float4(c1 * x.x + c2 * (o[0] - rho * x.x), c1 * x.y + c2 * (o[1] - rho * x.y),
                                      c1 * x.z + c2 * (o[2] - rho * x.z), c1 * x.w + c2 * (o[3] - rho * x.w));
        qs[h] = qv;
        const float4 gv = *reinterpret_cast<const float4*>(&gz[b * GS + tcol]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pe = draft_mean(c1, comp(x, e), c2s, comp(sv, e));  // m^p
          const double dd = (double)pe - (double)comp(qv, e);
          const double zz = (double)comp(y, e) - (double)pe;
          a2 = fma(dd, dd, a2);
          az = fma(zz, dd, az);
          ag = fma((double)comp(gv, e), dd, ag);
        }
      }
      // m^q of the pair back to whole-line rows (the inverse swap), with
      // non-temporal stores: the round reads back two of a chain's K + 1 rows
      const float4 recv = xchg8(b3 ? qs[0] : qs[1]);
      buf_st4_stream(vq, (uint32_t)(((row7 + 16 * rb) * d + colp + 32 * pr) * 4), b3 ? recv : qs[0]);
      buf_st4_stream(vq, (uint32_t)(((row7 + 16 * rb + 8) * d + colp + 32 * pr) * 4), b3 ? qs[1] : recv);
    }
    // the four lanes of the row (sub = 0..3), in a fixed order
    a2 += __shfl_xor(a2, 16);
    az += __shfl_xor(az, 16);
    ag += __shfl_xor(ag, 16);
    a2 += __shfl_xor(a2, 32);
    az += __shfl_xor(az, 32);
    ag += __shfl_xor(ag, 32);
    if (sub == 0) {
      double* o = part + ((int64_t)wc * TR + lr) * 3;
      o[0] = keep ? a2 : 0.0;
      o[1] = keep ? az : 0.0;
      o[2] = keep ? ag : 0.0;
    }
  }
  __syncthreads();
  // the column wavefronts of each row, in a fixed order
  for (int lr = threadIdx.x; lr < rows; lr += T::kThreads) {
    double t[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      double v = part[lr * 3 + q];
#pragma unroll
      for (int w = 1; w < QW; ++w) v += part[(w * TR + lr) * 3 + q];
      t[q] = v;
    }
    double* o = lrp + ((int64_t)(r0 + lr) * nct + ct) * 3;
    o[0] = t[0];
    o[1] = t[1];
    o[2] = t[2];
  }
}

// The tile of the sampler's bf16 mean GEMM: 288 x 256, one workgroup per
// compute unit.
using MeanTile = bf16b::Tile<256, 64>;

// Chains per tile of the chain-aligned mean GEMM, and whether it applies.
inline int big_chains(int K1) { return min(bf16b::TR / K1, BigMean<MeanTile>::kChains); }
// (for fewer than 512 components a tile's contraction is too short to pay for
// the one-workgroup-per-compute-unit epilogue: the 128 x 128 kernel, two per
// compute unit, is faster there)
inline bool big_mean_ok(const Target& t, int K1, bool vecd) {
  return vecd && t.d % MeanTile::TC == 0 && t.M % MeanTile::KC == 0 && t.M >= 512 && K1 <= bf16b::TR &&
         (int64_t)(bf16b::TR + 1) * t.d * 4 < ((int64_t)1 << 31) &&
         (int64_t)bf16b::TR * t.M * 2 < ((int64_t)1 << 31);
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
// Buffers for R rows; the split over d is chosen for plan_rows rows (0: R).
Plan make_plan(const Target& t, int R, int plan_rows = 0) {
  Plan p{};
  p.wide = t.d % KC == 0;
  const int tm = p.wide ? bf16w::WT : TM, tn = p.wide ? bf16w::WT : TN;
  const int slots = p.wide ? 256 : 512;
  const int Rp = plan_rows > 0 ? plan_rows : R;
  const int tiles = ((Rp + tm - 1) / tm) * ((t.M + tn - 1) / tn);
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

size_t target_ws_bytes_bf16(const Target& t, int rows, int plan_rows) {
  return make_plan(t, rows, plan_rows).total;
}

hipError_t target_mean_bf16_launch(const Target& t, int R, const float* x, int64_t ldx,
                                   const int32_t* step, float* mq, int64_t ldq, float* score,
                                   int64_t lds, void* ws, hipStream_t s, const int* gate,
                                   int plan_rows) {
  const Plan p = make_plan(t, R, plan_rows);
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
                                      uint64_t seed, void* ws, hipStream_t s, const int* gate,
                                      int plan_rows, int chain0) {
  const Plan p = make_plan(t, R, plan_rows);
  const Bufs w = carve(p, ws);
  const bool vecd = (t.d % 4 == 0) && aligned16(x) && aligned16(mq) && aligned16(sv);
  hipError_t e = logits_and_softmax(t, p, w, R, x, t.d, vecd, step, s, gate);
  if (e != hipSuccess) return e;
  // chain-aligned 288 x 256 tiles: whole column tiles of d, whole chunks of
  // M, aligned rows, 32-bit offsets inside a tile's views
  // the tile count of the partials (lr_tiles_bf16) assumes this kernel
  // whenever the shapes allow it: the sampler's workspace rows are aligned
  if (big_mean_ok(t, K1, t.d % 4 == 0)) {
    if (!vecd) return hipErrorInvalidValue;
    const int CT = big_chains(K1), B = R / K1;
    return launch_timed("gmm_mean_lr_bf16", gmm_mean_lr_bf16_big_kernel<MeanTile>,
                        dim3(((B + CT - 1) / CT) * (t.d / MeanTile::TC)), dim3(MeanTile::kThreads), s, R,
                        t.M, t.d, K1, CT, w.P, t.muT16, x, w.rowc, sv, cstep, t.coef, mq, lrp, rnd,
                        seed, gate, chain0);
  }
  dim3 g2((t.d + TN - 1) / TN, (R + TM - 1) / TM);
  // the buffer path: whole chunks of M, whole tiles of d, aligned rows, at
  // least eight rows per chain, 32-bit offsets inside a tile's views
  const bool vec = t.M % KC == 0 && t.d % TN == 0 && vecd && K1 >= 8 &&
                   (int64_t)(TM + 2) * t.d * 4 < ((int64_t)1 << 31);
  return launch_timed("gmm_mean_lr_bf16",
                      vec ? gmm_mean_lr_bf16_kernel<true> : gmm_mean_lr_bf16_kernel<false>, g2,
                      dim3(kThreads), s, R, t.M, t.d, K1, w.P, t.muT16, x, w.rowc, sv, cstep, t.coef,
                      mq, lrp, vecd, rnd, seed, gate, chain0);
}

int lr_tiles_bf16(const Target& t, int K1) {
  return big_mean_ok(t, K1, t.d % 4 == 0) ? t.d / MeanTile::TC : (t.d + TN - 1) / TN;
}

}  // namespace sd
