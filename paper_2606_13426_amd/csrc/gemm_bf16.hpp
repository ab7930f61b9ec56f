// bf16 matrix-core tile for the Gaussian-mixture contractions (gfx950).
//
// C[128 x 128] += A[rows][k] B[cols][k]^T over a k range: A float32 (rounded
// to bf16 with round-to-nearest-even while it is staged) or bf16, B bf16,
// float32 accumulation on v_mfma_f32_32x32x16_bf16.  Four wavefronts in a
// 2 x 2 layout each own a 64 x 64 sub-tile (2 x 2 blocks of 32 x 32).  k is
// staged through LDS in chunks of 64; within a chunk, MFMA step s (< 4) takes
// k = 16 s + 8 h + (0..7) from lane half h of both operands, so a lane reads
// its eight values of a row as one 16-byte LDS load.  Chunks are pipelined
// through two LDS buffers and two register sets (see tile()).
#pragma once

#include "common.hpp"

namespace sd {
namespace bf16 {

constexpr int kThreads = 256;
constexpr int TM = 128, TN = 128, KC = 64;
constexpr int LDH = KC + 8;  // LDS row stride in bf16 elements (144 bytes)

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two float32 -> packed bf16 pair (round to nearest even; one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 r;
  r[0] = (__bf16)lo;
  r[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, r);
}
__device__ __forceinline__ uint16_t to_bf16(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

struct OperandLds {
  uint16_t a[TM * LDH];
  uint16_t b[TN * LDH];
};

// One chunk of an operand in registers.  float32 A: 128 x 64 as eight float4
// per thread (rows t/16 + 16 h, columns 4 (t % 16)); bf16 operands: 128 x 64
// as four 16-byte vectors per thread (rows t/8 + 32 h, columns 8 (t % 8)).
template <class T>
struct Chunk;
template <>
struct Chunk<float> {
  float4 v[8];
};
template <>
struct Chunk<uint16_t> {
  uint4 v[4];
};

// Buffer view of the (at most TM) rows of one tile of a row-major matrix:
// reads at byte offsets past the rows that exist return zero in hardware.
// The host guarantees TM * ld * sizeof(T) < 2^31 for the VEC path.
constexpr uint32_t kBufferWord3 = 0x00020000;  // raw buffer, 32-bit dwords (gfx9 family)

// The base and size are wavefront-uniform; readfirstlane says so to the
// compiler, which otherwise wraps every load in a loop over distinct values.
template <class T>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_view(const T* A, int64_t ld, int nrows, int r0) {
  const int rows = max(0, min(nrows - r0, TM));
  const uint64_t base = reinterpret_cast<uint64_t>(A + (int64_t)r0 * ld);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)base);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
  const int bytes = __builtin_amdgcn_readfirstlane((int)((int64_t)rows * ld * (int64_t)sizeof(T)));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(((uint64_t)hi << 32) | lo),
                                           (short)0, bytes, (int)kBufferWord3);
}

// Rows r0.., columns k0.. (< kend) of a row-major matrix with row stride ld;
// out-of-range elements read as zero.  VEC: rows are 16-byte aligned and the
// k range is a whole number of chunks, so only rows can be out of range: one
// unconditional buffer load per 16-byte piece (rows past the end read zero
// from the view), which lets the compiler count the loads in flight.
// Otherwise element by element.
template <bool VEC>
__device__ __forceinline__ void load(const float* __restrict__ A, __amdgpu_buffer_rsrc_t view,
                                     int64_t ld, int nrows, int r0, int k0, int kend,
                                     Chunk<float>& c) {
  const int t = threadIdx.x;
  const int kc = k0 + 4 * (t & 15);
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    const int rr = (t >> 4) + 16 * h;
    if constexpr (VEC) {
      const uint32_t off = (uint32_t)((rr * (int)ld + kc) * 4);
      c.v[h] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(view, off, 0, 0));
    } else {
      const int r = r0 + rr;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r < nrows) {
        const float* p = A + (int64_t)r * ld + kc;
        if (kc < kend) v.x = p[0];
        if (kc + 1 < kend) v.y = p[1];
        if (kc + 2 < kend) v.z = p[2];
        if (kc + 3 < kend) v.w = p[3];
      }
      c.v[h] = v;
    }
  }
}

template <bool VEC>
__device__ __forceinline__ void load(const uint16_t* __restrict__ A, __amdgpu_buffer_rsrc_t view,
                                     int64_t ld, int nrows, int r0, int k0, int kend,
                                     Chunk<uint16_t>& c) {
  const int t = threadIdx.x;
  const int kc = k0 + 8 * (t & 7);
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int rr = (t >> 3) + 32 * h;
    if constexpr (VEC) {
      const uint32_t off = (uint32_t)((rr * (int)ld + kc) * 2);
      c.v[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(view, off, 0, 0));
    } else {
      const int r = r0 + rr;
      uint32_t w[4] = {0u, 0u, 0u, 0u};
      if (r < nrows) {
        const uint16_t* p = A + (int64_t)r * ld + kc;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (kc + e < kend) w[e >> 1] |= (uint32_t)p[e] << (16 * (e & 1));
      }
      c.v[h] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

__device__ __forceinline__ void store(uint16_t* lds, const Chunk<float>& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    const uint2 p = make_uint2(pack2(c.v[h].x, c.v[h].y), pack2(c.v[h].z, c.v[h].w));
    *reinterpret_cast<uint2*>(&lds[((t >> 4) + 16 * h) * LDH + 4 * (t & 15)]) = p;
  }
}

__device__ __forceinline__ void store(uint16_t* lds, const Chunk<uint16_t>& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 4; ++h)
    *reinterpret_cast<uint4*>(&lds[((t >> 3) + 32 * h) * LDH + 8 * (t & 7)]) = c.v[h];
}

// float64 sum of squares of the float32 values of a chunk, per loaded row.
__device__ __forceinline__ void add_squares(const Chunk<float>& c, double (&sq)[8]) {
#pragma unroll
  for (int h = 0; h < 8; ++h)
    sq[h] += (double)c.v[h].x * c.v[h].x + (double)c.v[h].y * c.v[h].y +
             (double)c.v[h].z * c.v[h].z + (double)c.v[h].w * c.v[h].w;
}

__device__ __forceinline__ bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// One chunk of 64 k on the matrix cores for this wavefront's 2 x 2 blocks.
__device__ __forceinline__ void mma_chunk(const OperandLds& sm, f32x16 (&acc)[2][2]) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wr = w >> 1, wc = w & 1;
  const int i = lane & 31, h = lane >> 5;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int ko = 16 * s + 8 * h;
    bf16x8 fa[2], fb[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      fa[q] = frag(&sm.a[(64 * wr + 32 * q + i) * LDH + ko]);
      fb[q] = frag(&sm.b[(64 * wc + 32 * q + i) * LDH + ko]);
    }
#pragma unroll
    for (int qa = 0; qa < 2; ++qa)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        acc[qa][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[qa], fb[qb], acc[qa][qb], 0, 0, 0);
  }
}

__device__ __forceinline__ void zero(f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int qa = 0; qa < 2; ++qa)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[qa][qb][v] = 0.f;
}

// Accumulate tile (r0, c0) of A[nra][.] B[nrb][.]^T over k in [kbeg, kend).
// With SQ (float32 A only) also the float64 squares of this thread's A rows.
// VEC: see load().
//
// Software pipeline: two LDS buffers and two register sets.  Step c multiplies
// the chunk in LDS buffer c % 2, then stores chunk c + 1 (fetched two steps
// earlier) into the other buffer and issues the global loads of chunk c + 3
// into the register set just freed; one barrier per step.  The matrix cores
// work on step c while chunk c + 1's loads complete, and two chunks are in
// flight per workgroup.  The steady state (more than four chunks) has no
// conditional loads, so the compiler's wait before each store counts exactly
// the newer loads; the last chunks and short ranges run without prefetch.
// The caller's first use of sm after this returns must follow a barrier.
template <bool SQ, bool VEC, class TA>
__device__ __forceinline__ void tile(OperandLds (&sm)[2], const TA* __restrict__ A, int64_t lda,
                                     int nra, const uint16_t* __restrict__ Bm, int64_t ldb, int nrb,
                                     int r0, int c0, int kbeg, int kend, f32x16 (&acc)[2][2],
                                     double (&sq)[8]) {
  const int n = (kend - kbeg + KC - 1) / KC;
  const __amdgpu_buffer_rsrc_t va = tile_view(A, lda, nra, r0);
  const __amdgpu_buffer_rsrc_t vb = tile_view(Bm, ldb, nrb, c0);
  Chunk<TA> ra0, ra1;
  Chunk<uint16_t> rb0, rb1;
  auto ld = [&](int c, Chunk<TA>& a, Chunk<uint16_t>& b) {
    load<VEC>(A, va, lda, nra, r0, kbeg + c * KC, kend, a);
    load<VEC>(Bm, vb, ldb, nrb, c0, kbeg + c * KC, kend, b);
  };
  auto st = [&](OperandLds& buf, const Chunk<TA>& a, const Chunk<uint16_t>& b) {
    store(buf.a, a);
    store(buf.b, b);
    if constexpr (SQ) add_squares(a, sq);
  };
  if (n > 4) {
    ld(0, ra0, rb0);
    ld(1, ra1, rb1);
    st(sm[0], ra0, rb0);
    ld(2, ra0, rb0);
    __syncthreads();
    int c = 0;
    for (; c + 4 < n; c += 2) {
      mma_chunk(sm[0], acc);
      st(sm[1], ra1, rb1);
      ld(c + 3, ra1, rb1);
      __syncthreads();
      mma_chunk(sm[1], acc);
      st(sm[0], ra0, rb0);
      ld(c + 4, ra0, rb0);
      __syncthreads();
    }
    // chunk c is in buffer 0, c + 1 in (ra1, rb1), c + 2 in (ra0, rb0); 3 or 4 remain
    mma_chunk(sm[0], acc);
    st(sm[1], ra1, rb1);
    const bool four = c + 3 < n;
    if (four) ld(c + 3, ra1, rb1);
    __syncthreads();
    mma_chunk(sm[1], acc);
    st(sm[0], ra0, rb0);
    __syncthreads();
    mma_chunk(sm[0], acc);
    if (four) {
      st(sm[1], ra1, rb1);
      __syncthreads();
      mma_chunk(sm[1], acc);
    }
    __syncthreads();
    return;
  }
  // up to four chunks: the same pipeline, unrolled (uniform branches on n)
  if (n <= 0) return;
  ld(0, ra0, rb0);
  if (n > 1) ld(1, ra1, rb1);
  st(sm[0], ra0, rb0);
  __syncthreads();
  if (n > 2) ld(2, ra0, rb0);
  mma_chunk(sm[0], acc);
  if (n > 1) {
    st(sm[1], ra1, rb1);
    __syncthreads();  // also: chunk 0's reads of buffer 0 are done
    if (n > 3) ld(3, ra1, rb1);
    mma_chunk(sm[1], acc);
  }
  if (n > 2) {
    st(sm[0], ra0, rb0);
    __syncthreads();  // also: chunk 1's reads of buffer 1 are done
    mma_chunk(sm[0], acc);
  }
  if (n > 3) {
    st(sm[1], ra1, rb1);
    __syncthreads();
    mma_chunk(sm[1], acc);
  }
  __syncthreads();
}

// Row of accumulator element v of block qa, and column of block qb, of this
// lane inside the 128 x 128 tile.
__device__ __forceinline__ int out_row(int qa, int v) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return 64 * (w >> 1) + 32 * qa + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}
__device__ __forceinline__ int out_col(int qb) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return 64 * (w & 1) + 32 * qb + (lane & 31);
}

}  // namespace bf16
}  // namespace sd
