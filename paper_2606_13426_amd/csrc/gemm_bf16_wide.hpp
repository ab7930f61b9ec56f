// Wide bf16 matrix-core tile for the large Gaussian-mixture contractions
// (gfx950): C[256 x 256] += A[rows][k] B[cols][k]^T over a k range, A float32
// (rounded to bf16 with round-to-nearest-even while it is staged) or bf16,
// B bf16, float32 accumulation on v_mfma_f32_32x32x16_bf16.
//
// One workgroup of eight wavefronts per compute unit, two per SIMD: in a
// 2 x 4 layout each owns a 128 x 64 sub-tile (4 x 2 blocks of 32 x 32, 128
// accumulators), so one wavefront's matrix work covers the other's LDS
// reads.  Per 64-wide k chunk a wavefront issues 32 MFMAs against 24 16-byte
// LDS reads, and the workgroup fetches 96 KB (float32 A) from L2 -- half the
// L2 bytes per flop of two 128 x 128 workgroups.
//
// Pipeline: two LDS buffers and one register set.  Step c multiplies the
// chunk in buffer c % 2; halfway through it stores chunk c + 1 (fetched one
// step earlier) into the other buffer and issues the global loads of chunk
// c + 2; one barrier per step.  Only one chunk's loads are ever in flight,
// so each store waits for all outstanding loads (vmcnt(0) is exact).
//
// The aligned (buffer) path only: every row of A and B is 16-byte aligned,
// the k range is a whole number of chunks, and a tile's rows fit 32-bit byte
// offsets; rows past a matrix read as zero from the tile's buffer view.
#pragma once

#include "bufio.hpp"
#include "common.hpp"

namespace sd {
namespace bf16w {

constexpr int kThreads = 512;
constexpr int WT = 256, KC = 64;
constexpr int LDH = KC + 8;  // LDS row stride in bf16 elements (144 bytes)

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

struct OperandLds {
  uint16_t a[WT * LDH];
  uint16_t b[WT * LDH];
};
static_assert(2 * sizeof(OperandLds) <= 160 * 1024, "two operand buffers must fit the LDS");

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 r;
  r[0] = (__bf16)lo;
  r[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, r);
}

// One chunk of an operand in registers.  float32 A: 256 x 64 as eight float4
// per thread (rows t/16 + 32 h, columns 4 (t % 16)); bf16: 256 x 64 as four
// 16-byte vectors per thread (rows t/8 + 64 h, columns 8 (t % 8)).
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

// The view of the (at most WT) rows r0.. of a row-major matrix.
template <class T>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_view(const T* A, int64_t ld, int nrows, int r0) {
  return buf_view(A + (int64_t)r0 * ld, (int64_t)max(0, min(nrows - r0, WT)) * ld * (int64_t)sizeof(T));
}

// Chunk at column k0 (uniform: passed as the load's scalar offset; the row
// part of every offset is per lane, so rows past the view read zero).
__device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t view, int64_t ld, int k0, Chunk<float>& c) {
  const int t = threadIdx.x;
  const uint32_t base = (uint32_t)(((t >> 4) * (int)ld + 4 * (t & 15)) * 4);
  const uint32_t hstep = (uint32_t)(32 * (int)ld * 4);
  const int so = __builtin_amdgcn_readfirstlane(k0 * 4);
#pragma unroll
  for (int h = 0; h < 8; ++h)
    c.v[h] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(view, base + h * hstep, so, 0));
}

__device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t view, int64_t ld, int k0, Chunk<uint16_t>& c) {
  const int t = threadIdx.x;
  const uint32_t base = (uint32_t)(((t >> 3) * (int)ld + 8 * (t & 7)) * 2);
  const uint32_t hstep = (uint32_t)(64 * (int)ld * 2);
  const int so = __builtin_amdgcn_readfirstlane(k0 * 2);
#pragma unroll
  for (int h = 0; h < 4; ++h)
    c.v[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(view, base + h * hstep, so, 0));
}

__device__ __forceinline__ void store(uint16_t* lds, const Chunk<float>& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    const uint2 p = make_uint2(pack2(c.v[h].x, c.v[h].y), pack2(c.v[h].z, c.v[h].w));
    *reinterpret_cast<uint2*>(&lds[((t >> 4) + 32 * h) * LDH + 4 * (t & 15)]) = p;
  }
}

__device__ __forceinline__ void store(uint16_t* lds, const Chunk<uint16_t>& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 4; ++h)
    *reinterpret_cast<uint4*>(&lds[((t >> 3) + 64 * h) * LDH + 8 * (t & 7)]) = c.v[h];
}

// Sum of squares of the float32 values of a chunk for the loaded rows h
// whose bit is set in mask (wavefront-uniform): the four values of a row
// summed in float32, the chunk partial added in float64.  The float32 partial
// is within a few ulp (about 2e-7 relative) of the exact one, far inside the
// bf16 rounding of the same values in the contraction.
__device__ __forceinline__ void add_squares(const Chunk<float>& c, double (&sq)[8], uint32_t mask) {
#pragma unroll
  for (int h = 0; h < 8; ++h) {
    if (!(mask >> h & 1u)) continue;
    const float4 v = c.v[h];
    sq[h] += (double)(v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w);
  }
}

__device__ __forceinline__ bf16x8 frag(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// MFMA steps s0 .. s0 + ns - 1 (16 k each) of the chunk in sm for this
// wavefront's 4 x 2 blocks: lane half h supplies k = 16 s + 8 h + (0..7) of
// row lane % 32 of each block, one 16-byte LDS read per operand block.
__device__ __forceinline__ void mma_steps(const OperandLds& sm, f32x16 (&acc)[4][2], int s0, int ns) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wr = w >> 2, wc = w & 3;
  const int i = lane & 31, h = lane >> 5;
  const uint16_t* pa = &sm.a[(128 * wr + i) * LDH + 8 * h];
  const uint16_t* pb = &sm.b[(64 * wc + i) * LDH + 8 * h];
#pragma unroll
  for (int s = s0; s < s0 + ns; ++s) {
    bf16x8 fa[4], fb[2];
#pragma unroll
    for (int q = 0; q < 4; ++q) fa[q] = frag(pa + 32 * q * LDH + 16 * s);
#pragma unroll
    for (int q = 0; q < 2; ++q) fb[q] = frag(pb + 32 * q * LDH + 16 * s);
#pragma unroll
    for (int qa = 0; qa < 4; ++qa)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        acc[qa][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[qa], fb[qb], acc[qa][qb], 0, 0, 0);
  }
}

__device__ __forceinline__ void zero(f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int qa = 0; qa < 4; ++qa)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[qa][qb][v] = 0.f;
}

// Accumulate the tile of the views va (A rows) and vb (B rows) over the
// chunks of k in [kbeg, kend) (a whole number of chunks).  With SQ (float32 A
// only) also the squares of this thread's A rows h selected by sqmask (a
// runtime mask rather than a second instantiation: one copy of the loop keeps
// the register allocation and schedule of the plain tile).  The caller's
// first use of sm after this returns must follow a barrier.
template <bool SQ, class TA>
__device__ __forceinline__ void tile(OperandLds (&sm)[2], __amdgpu_buffer_rsrc_t va, int64_t lda,
                                     __amdgpu_buffer_rsrc_t vb, int64_t ldb, int kbeg, int kend,
                                     f32x16 (&acc)[4][2], double (&sq)[8], uint32_t sqmask) {
  const int n = (kend - kbeg) / KC;
  if (n <= 0) return;
  Chunk<TA> ra;
  Chunk<uint16_t> rb;
  auto ld = [&](int c) {
    load(va, lda, kbeg + c * KC, ra);
    load(vb, ldb, kbeg + c * KC, rb);
  };
  auto st = [&](OperandLds& buf) {
    store(buf.a, ra);
    store(buf.b, rb);
    if constexpr (SQ) add_squares(ra, sq, sqmask);
  };
  ld(0);
  st(sm[0]);
  if (n > 1) ld(1);
  __syncthreads();
  for (int c = 0; c < n; ++c) {
    OperandLds& cur = sm[c & 1];
    mma_steps(cur, acc, 0, 2);
    if (c + 1 < n) {
      st(sm[(c + 1) & 1]);
      if (c + 2 < n) ld(c + 2);
    }
    mma_steps(cur, acc, 2, 2);
    __syncthreads();
  }
}

// Row of accumulator element v of block qa, and column of block qb, of this
// lane inside the 256 x 256 tile.
__device__ __forceinline__ int out_row(int qa, int v) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return 128 * (w >> 2) + 32 * qa + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}
__device__ __forceinline__ int out_col(int qb) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return 64 * (w & 3) + 32 * qb + (lane & 31);
}

}  // namespace bf16w
}  // namespace sd
