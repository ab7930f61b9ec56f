// Large bf16 matrix-core tiles for the Gaussian-mixture contractions (gfx950):
// C[rows][cols] += R[rows][k] Q[cols][k]^T over k, with tiles of TR = 288
// rows by TC (128 or 256) columns, both operands bf16 with float32
// accumulation on v_mfma_f32_16x16x32_bf16.
//
// The matrix instruction multiplies a 16 x 32 block of Q (its "A" operand:
// lane l holds column-side row l % 16, k = 8 (l / 16) + 0..7) by a 32 x 16
// block of R (its "B" operand, the same lane pattern over rows), so lane l's
// four accumulators of a block are FOUR CONSECUTIVE COLUMNS 4 (l / 16) + 0..3
// of the tile row l % 16: the epilogue reads and writes each row segment as
// one 16-byte access without staging the tile through LDS.
//
// Each wavefront owns 144 rows x 64 columns, 9 x 4 blocks of 16 x 16 (144
// accumulators); a tile has two row halves and TC / 64 column quarters, i.e.
// 2 TC / 64 wavefronts.  Per 32-k step a wavefront reads 4 + 9 16-byte
// fragments from LDS for 36 matrix instructions, so LDS reads stay below the
// matrix rate.  A tile moves (288 + TC) x 2 bytes of operands per k for
// 2 x 288 x TC flops: 136 flops per byte at TC = 256, 89 at TC = 128.  The
// 288 x 256 tile (eight wavefronts, 64-wide k chunks) takes a whole compute
// unit's LDS and most of its registers.  (Measured on the latent-sized mean
// GEMM: 70 us for the contraction alone against 83 us for 288 x 128 tiles
// with 32-wide chunks, two workgroups per compute unit, and 96 us for the
// 128 x 128 tile of gemm_bf16.hpp.)
//
// Pipeline: two LDS buffers of KC-wide k chunks and one register set; step c
// multiplies buffer c % 2, stores chunk c + 1 (loaded one step earlier) into
// the other buffer halfway through, then issues the loads of chunk c + 2.
// The aligned path only: rows 16-byte aligned, k a whole number of chunks,
// operand views whose byte offsets fit 32 bits; rows past a view read zero.
#pragma once

#include "bufio.hpp"
#include "common.hpp"

namespace sd {
namespace bf16b {

constexpr int TR = 288;
constexpr int RB = 9, CB = 4;  // 16 x 16 blocks per wavefront (rows, columns)

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <int TC_, int KC_>
struct Tile {
  static constexpr int TC = TC_, KC = KC_;
  static constexpr int kThreads = 2 * TC;           // 2 x (TC / 64) wavefronts
  static constexpr int LDH = KC + 8;                // LDS row stride in bf16 elements
  static constexpr int SEG = KC / 8;                // 16-byte pieces per row and chunk
  static constexpr int NQ = TC * SEG / kThreads;    // column-side pieces per thread
  static constexpr int NR = TR * SEG / kThreads;    // row-side pieces per thread (whole)
  static constexpr int NR_EXTRA = TR * SEG - NR * kThreads;  // pieces of the first threads
  static_assert(NQ * kThreads == TC * SEG, "column side splits evenly");
  static_assert(NR_EXTRA % 64 == 0 && NR_EXTRA < kThreads, "the extra pieces fill whole wavefronts");

  struct Lds {
    uint16_t q[TC * LDH];  // column side
    uint16_t r[TR * LDH];  // row side
  };

  struct Chunk {
    uint4 q[NQ];
    uint4 r[NR + (NR_EXTRA > 0 ? 1 : 0)];
  };

  // piece p = t + kThreads h of a side: row p / SEG, 16-byte segment p % SEG
  static __device__ __forceinline__ uint32_t piece_off(int p, int ld) {
    return (uint32_t)(((p / SEG) * ld + 8 * (p % SEG)) * 2);
  }
  static __device__ __forceinline__ int piece_lds(int p) { return (p / SEG) * LDH + 8 * (p % SEG); }

  static __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t vq, int ldq, __amdgpu_buffer_rsrc_t vr,
                                              int ldr, int k0, Chunk& c) {
    const int t = threadIdx.x;
    const int so = __builtin_amdgcn_readfirstlane(k0 * 2);
#pragma unroll
    for (int h = 0; h < NQ; ++h)
      c.q[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vq, piece_off(t + kThreads * h, ldq), so, 0));
#pragma unroll
    for (int h = 0; h < NR; ++h)
      c.r[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vr, piece_off(t + kThreads * h, ldr), so, 0));
    if (NR_EXTRA > 0 && t < NR_EXTRA)
      c.r[NR] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vr, piece_off(t + kThreads * NR, ldr), so, 0));
  }

  static __device__ __forceinline__ void store(Lds& sm, const Chunk& c) {
    const int t = threadIdx.x;
#pragma unroll
    for (int h = 0; h < NQ; ++h) *reinterpret_cast<uint4*>(&sm.q[piece_lds(t + kThreads * h)]) = c.q[h];
#pragma unroll
    for (int h = 0; h < NR; ++h) *reinterpret_cast<uint4*>(&sm.r[piece_lds(t + kThreads * h)]) = c.r[h];
    if (NR_EXTRA > 0 && t < NR_EXTRA) *reinterpret_cast<uint4*>(&sm.r[piece_lds(t + kThreads * NR)]) = c.r[NR];
  }

  static __device__ __forceinline__ bf16x8 frag(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
  }

  // The 32-k step s of the chunk in sm for this wavefront's 9 x 4 blocks.
  static __device__ __forceinline__ void mma_step(const Lds& sm, f32x4 (&acc)[RB][CB], int s) {
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    constexpr int QW = TC / 64;  // column quarters
    const int ko = 32 * s + 8 * (lane >> 4);
    const uint16_t* pq = &sm.q[(64 * (w % QW) + (lane & 15)) * LDH + ko];
    const uint16_t* pr = &sm.r[(144 * (w / QW) + (lane & 15)) * LDH + ko];
    bf16x8 fq[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) fq[cb] = frag(pq + 16 * cb * LDH);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const bf16x8 fr = frag(pr + 16 * rb * LDH);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fq[cb], fr, acc[rb][cb], 0, 0, 0);
    }
  }

  // Accumulate the tile of the views vq (column side, ldq elements per row)
  // and vr (row side) over the chunks of k in [kbeg, kend) (a whole number of
  // chunks).  The caller's first use of sm after this returns must follow a
  // barrier.
  static __device__ __forceinline__ void run(Lds (&sm)[2], __amdgpu_buffer_rsrc_t vq, int ldq,
                                             __amdgpu_buffer_rsrc_t vr, int ldr, int kbeg, int kend,
                                             f32x4 (&acc)[RB][CB]) {
    const int n = (kend - kbeg) / KC;
    if (n <= 0) return;
    Chunk rg;
    load(vq, ldq, vr, ldr, kbeg, rg);
    store(sm[0], rg);
    if (n > 1) load(vq, ldq, vr, ldr, kbeg + KC, rg);
    __syncthreads();
    for (int c = 0; c < n; ++c) {
      const Lds& cur = sm[c & 1];
      constexpr int half = KC / 64 > 0 ? KC / 64 : 1;  // 32-k steps before the store
#pragma unroll
      for (int s = 0; s < half; ++s) mma_step(cur, acc, s);
      if (c + 1 < n) {
        store(sm[(c + 1) & 1], rg);
        if (c + 2 < n) load(vq, ldq, vr, ldr, kbeg + (c + 2) * KC, rg);
      }
#pragma unroll
      for (int s = half; s < KC / 32; ++s) mma_step(cur, acc, s);
      __syncthreads();
    }
  }

  // Tile row of this lane's accumulators of row block rb, and the first of
  // the four tile columns of column block cb.
  static __device__ __forceinline__ int out_row(int rb) {
    return 144 * ((threadIdx.x >> 6) / (TC / 64)) + 16 * rb + (threadIdx.x & 15);
  }
  static __device__ __forceinline__ int out_col(int cb) {
    return 64 * ((threadIdx.x >> 6) % (TC / 64)) + 16 * cb + 4 * ((threadIdx.x >> 4) & 3);
  }
  static __device__ __forceinline__ int col_wave() { return (threadIdx.x >> 6) % (TC / 64); }
};

__device__ __forceinline__ void zero(f32x4 (&acc)[RB][CB]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};
}

}  // namespace bf16b
}  // namespace sd
