// Float32 contractions on the bf16 matrix cores (gfx950).
//
// Each float32 value is split exactly into three bf16 terms, v = hi + mid + lo
// (hi = bf16(v), mid = bf16(v - hi), lo = bf16(v - hi - mid), rounding to
// nearest even; both residuals are exact in float32, and the 24-bit mantissa
// fits the three 8-bit ones).  A product a.b is formed from the six terms
//   lo.hi + hi.lo + mid.mid + mid.hi + hi.mid + hi.hi
// (smallest first) on v_mfma_f32_16x16x32_bf16, whose bf16 x bf16 products are
// exact in its float32 accumulator.  The three dropped terms (mid.lo, lo.mid,
// lo.lo) are below 2^-23 |a||b| together, the size of one float32 rounding, so
// the result is float32-accurate at 6/16 of the float32 instruction's
// matrix-core time.
//
// Tile: 64 RB rows of A x 64 rows of B (the output's columns) per workgroup
// of four wavefronts; wavefront w owns RB blocks of 16 rows (rows 16 (RB w +
// r) .. + 15, r < RB) and all four 16-column blocks, so each B fragment read
// from LDS feeds RB row blocks.  A (float32) goes from memory straight into
// its wavefront's registers, lane l holding row 16 (RB w + r) + l % 16 and
// k = 8 (l / 16) .. + 7 of each 32-wide step, and is split there.  B comes pre-split (three
// bf16 planes in memory, row-major with the same leading dimension) and is
// staged through LDS, 64 k per chunk, three planes of 64 x 72 (row stride 144
// bytes: the 16 rows of one 16-lane read pass fall in distinct banks).
// Output block c of row block r of wavefront w: lane l holds rows
// 16 (RB w + r) + 4 (l / 16) + j (j < 4) of column 16 c + l % 16.
//
// The aligned path only: every row 16-byte aligned, k ranges whole chunks,
// rows past a matrix read as zero from the tile's buffer views.
#pragma once

#include "bufio.hpp"
#include "common.hpp"

namespace sd {
namespace split {

constexpr int TILE = 64, KC = 64;
constexpr int LDH = KC + 8;  // LDS row stride in bf16 elements
constexpr int kPlaneElems = TILE * LDH;
constexpr int kLdsBytes = 3 * kPlaneElems * 2;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct Acc {
  f32x4 c[4];
};

__device__ __forceinline__ void zero(Acc& a) {
#pragma unroll
  for (int b = 0; b < 4; ++b) a.c[b] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// The three bf16 terms of eight float32 values.
__device__ __forceinline__ void split8(const float4& u, const float4& v, bf16x8& hi, bf16x8& mid,
                                       bf16x8& lo) {
  const float x[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const __bf16 h = (__bf16)x[i];
    const float r = x[i] - (float)h;
    const __bf16 m = (__bf16)r;
    hi[i] = h;
    mid[i] = m;
    lo[i] = (__bf16)(r - (float)m);
  }
}

// B chunk in registers: plane p, rows t / 8 + 32 h (h < 2), k = 8 (t % 8) .. + 7.
struct BChunk {
  uint4 v[3][2];
};

// views[p]: the (at most 64) rows of plane p of the tile.
__device__ __forceinline__ void load_b(const __amdgpu_buffer_rsrc_t (&views)[3], int64_t ldb,
                                       int k0, BChunk& c) {
  const int t = threadIdx.x;
  const uint32_t base = (uint32_t)(((t >> 3) * (int)ldb + 8 * (t & 7)) * 2);
  const uint32_t hstep = (uint32_t)(32 * (int)ldb * 2);
  const int so = __builtin_amdgcn_readfirstlane(k0 * 2);
#pragma unroll
  for (int p = 0; p < 3; ++p)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      c.v[p][h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(views[p], base + h * hstep, so, 0));
}

__device__ __forceinline__ void store_b(uint16_t* lds, const BChunk& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int p = 0; p < 3; ++p)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      *reinterpret_cast<uint4*>(&lds[p * kPlaneElems + ((t >> 3) + 32 * h) * LDH + 8 * (t & 7)]) = c.v[p][h];
}

// A chunk of this lane's row: k = 32 s + 8 (l / 16) .. + 7 for s < 2.
struct AChunk {
  float4 v[2][2];
};

// view: the (at most 64 RB) rows of A of the tile; lane rows 16 (RB w + r) + l % 16.
template <int RB>
__device__ __forceinline__ void load_a(__amdgpu_buffer_rsrc_t view, int64_t lda, int k0, AChunk (&a)[RB]) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int so = __builtin_amdgcn_readfirstlane(k0 * 4);
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const uint32_t base = (uint32_t)(((16 * (RB * w + r) + (lane & 15)) * (int)lda + 8 * (lane >> 4)) * 4);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int q = 0; q < 2; ++q)
        a[r].v[s][q] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(view, base + (uint32_t)((32 * s + 4 * q) * 4), so, 0));
  }
}

// float64 sum of squares of the lane's A values of a chunk.
__device__ __forceinline__ double squares(const AChunk& a) {
  double t = 0.0;
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float4 v = a.v[s][q];
      t += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
    }
  return t;
}

__device__ __forceinline__ bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// The chunk's 2 steps x 4 column blocks x RB row blocks x 6 terms.
template <int RB>
__device__ __forceinline__ void mma_chunk(const uint16_t* lds, const AChunk (&a)[RB], Acc (&acc)[RB]) {
  const int lane = threadIdx.x & 63;
  const uint16_t* pb = lds + (lane & 15) * LDH + 8 * (lane >> 4);
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    bf16x8 ah[RB], am[RB], al[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) split8(a[r].v[s][0], a[r].v[s][1], ah[r], am[r], al[r]);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const uint16_t* q = pb + 16 * b * LDH + 32 * s;
      const bf16x8 bh = frag(q), bm = frag(q + kPlaneElems), bl = frag(q + 2 * kPlaneElems);
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        f32x4 c = acc[r].c[b];
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[r], bh, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[r], bl, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am[r], bm, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am[r], bh, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[r], bm, c, 0, 0, 0);
        acc[r].c[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[r], bh, c, 0, 0, 0);
      }
    }
  }
}

// Accumulate the tile over the chunks of k in [kbeg, kend) (whole chunks, at
// least one), starting from the first chunk already loaded into ra, rb (so a
// caller can issue other loads after them: the first wait then excludes
// those), the B planes staged through `lds` (kLdsBytes); with SQ also this
// lane's float64 squares of A.  Later chunks are loaded when they are due,
// not a chunk ahead: a prefetch register set would cost the occupancy that
// hides those loads behind the other workgroups' matrix work.  The caller's
// first use of lds afterwards must follow a barrier.
template <bool SQ, int RB>
__device__ __forceinline__ void tile_run(uint16_t* lds, __amdgpu_buffer_rsrc_t va, int64_t lda,
                                         const __amdgpu_buffer_rsrc_t (&vb)[3], int64_t ldb,
                                         int kbeg, int kend, AChunk (&ra)[RB], BChunk& rb,
                                         Acc (&acc)[RB], double (&sq)[RB]) {
  const int n = (kend - kbeg) / KC;
  store_b(lds, rb);
  __syncthreads();
  if constexpr (SQ) {
#pragma unroll
    for (int r = 0; r < RB; ++r) sq[r] += squares(ra[r]);
  }
  mma_chunk<RB>(lds, ra, acc);
  for (int c = 1; c < n; ++c) {
    load_b(vb, ldb, kbeg + c * KC, rb);
    load_a<RB>(va, lda, kbeg + c * KC, ra);
    __syncthreads();  // every wavefront is done with the previous chunk
    store_b(lds, rb);
    __syncthreads();
    if constexpr (SQ) {
#pragma unroll
      for (int r = 0; r < RB; ++r) sq[r] += squares(ra[r]);
    }
    mma_chunk<RB>(lds, ra, acc);
  }
}

// The (at most 64) rows r0.. of a row-major bf16 plane with leading dimension ld.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rows(const uint16_t* P, int64_t ld, int nrows,
                                                           int r0) {
  return buf_view(P + (int64_t)r0 * ld, (int64_t)max(0, min(nrows - r0, TILE)) * ld * 2);
}

// Row (inside the tile) of accumulator element j of row block r, and column
// of block b.
template <int RB>
__device__ __forceinline__ int out_row(int r, int j) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return 16 * (RB * w + r) + 4 * (lane >> 4) + j;
}
__device__ __forceinline__ int out_col(int b) { return 16 * b + (threadIdx.x & 15); }

// The three bf16 planes of a float32 matrix [rows][cols] (host, row-major),
// each [rows][cols]: the split above, evaluated on the host.
inline uint16_t bf16_bits_rne(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
inline float bf16_value(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}
inline void split_host(const float* src, size_t n, uint16_t* hi, uint16_t* mid, uint16_t* lo) {
  for (size_t i = 0; i < n; ++i) {
    const float v = src[i];
    const uint16_t h = bf16_bits_rne(v);
    const float r = v - bf16_value(h);
    const uint16_t m = bf16_bits_rne(r);
    hi[i] = h;
    mid[i] = m;
    lo[i] = bf16_bits_rne(r - bf16_value(m));
  }
}

}  // namespace split
}  // namespace sd
