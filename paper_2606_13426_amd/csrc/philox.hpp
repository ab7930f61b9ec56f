// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) and the draws built on it.
//
// A round maps counter (c0,c1,c2,c3) and key (k0,k1) to
//   (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)),
// M0 = 0xD2511F53, M1 = 0xCD9E8D57, and the key is bumped by the Weyl
// constants (0x9E3779B9, 0xBB67AE85) between rounds.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

enum : uint32_t {
  TAG_INIT = 1,
  TAG_DRAFT = 2,
  TAG_COIN = 3,
  TAG_USAMPLE = 4,
  TAG_RESID = 5,
  TAG_TARGET = 6
};

__device__ __forceinline__ uint4 philox(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                        uint64_t seed) {
  uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // one 32x32 -> 64-bit product per multiplier (a single v_mad_u64_u32)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

__device__ __forceinline__ uint32_t pick(const uint4& w, int i) {
  return i == 0 ? w.x : i == 1 ? w.y : i == 2 ? w.z : w.w;
}

// 24-bit uniform in (0, 1), exact in float64.
__device__ __forceinline__ double uniform64(uint32_t w) {
  return ((double)(w >> 8) + 0.5) * 0x1p-24;
}

// -2 ln u for the 24-bit uniform u = (m + 0.5) 2^-24 of word w, in float32
// without losing the small-radius tail.  For u < 1/2, u is exact in float32.
// For u >= 1/2, t = 1 - u = (2^24 - 1 - m + 0.5) 2^-24 is exact, w = fl(1 - t)
// and ln u = ln w + (u - w)/w with u - w = -((w - 1) + t) exact, so one logf
// serves both halves (no divergent branch).  The correction is below one ulp
// of ln w, so the hardware reciprocal (about 1 ulp) is exact enough for it.
__device__ __forceinline__ float neg2log_u24(uint32_t w) {
  const uint32_t m = w >> 8;
  const bool hi = m >= (1u << 23);
  const float t = ((float)((1u << 24) - 1u - m) + 0.5f) * 0x1p-24f;
  const float wv = hi ? 1.0f - t : ((float)m + 0.5f) * 0x1p-24f;
  const float corr = hi ? -((wv - 1.0f) + t) * __builtin_amdgcn_rcpf(wv) : 0.0f;
  return -2.0f * (logf(wv) + corr);
}

// Box-Muller on (w0, w1) and (w2, w3): radius sqrt(-2 ln u_a), angle 2 pi u_b.
// The hardware sine and cosine take their argument in revolutions, so they
// evaluate sin(2 pi u_b), cos(2 pi u_b) directly on u_b in (0, 1); the radius
// uses the hardware square root (about 1 ulp; the argument is a normal
// float32 of at most 2 ln 2^25, so no range scaling is needed).
__device__ __forceinline__ float4 normals4(uint4 w) {
  const float ra = __builtin_amdgcn_sqrtf(neg2log_u24(w.x));
  const float rc = __builtin_amdgcn_sqrtf(neg2log_u24(w.z));
  const float ub = ((float)(w.y >> 8) + 0.5f) * 0x1p-24f;
  const float ud = ((float)(w.w >> 8) + 0.5f) * 0x1p-24f;
  return make_float4(ra * __builtin_amdgcn_cosf(ub), ra * __builtin_amdgcn_sinf(ub),
                     rc * __builtin_amdgcn_cosf(ud), rc * __builtin_amdgcn_sinf(ud));
}

__device__ __forceinline__ float get4(const float4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

}  // namespace sd
