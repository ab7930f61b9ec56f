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
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
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

// Box-Muller on (w0, w1) and (w2, w3).  The radius is computed from the exact
// float64 uniform (its float32 rounding would map 1 - 2^-25 to 1 and lose the
// small-radius tail); the angle 2 pi u uses sincospi in float32.
__device__ __forceinline__ float4 normals4(uint4 w) {
  const float ra = sqrtf((float)(-2.0 * log(uniform64(w.x))));
  const float rc = sqrtf((float)(-2.0 * log(uniform64(w.z))));
  float sa, ca, sc, cc;
  sincospif(((float)(w.y >> 8) + 0.5f) * 0x1p-23f, &sa, &ca);
  sincospif(((float)(w.w >> 8) + 0.5f) * 0x1p-23f, &sc, &cc);
  return make_float4(ra * ca, ra * sa, rc * cc, rc * sc);
}

__device__ __forceinline__ float get4(const float4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

}  // namespace sd
