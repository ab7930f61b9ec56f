// Four-coordinate row access and the Free-Drafter recursion, shared by the
// standalone draft kernel and the sampler's fused advance kernel.
#pragma once

#include "common.hpp"
#include "philox.hpp"

namespace sd {

__device__ __forceinline__ void load4(const float* p, int cnt, bool vec, float (&v)[4]) {
  if (vec) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = c < cnt ? p[c] : 0.0f;
  }
}

// stream: a non-temporal store of an aligned vector (see stream_rows).
__device__ __forceinline__ void store4(float* p, int cnt, bool vec, const float (&v)[4],
                                      bool stream = false) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  if (vec && stream) {
    const f32x4 t = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(t, reinterpret_cast<f32x4*>(p));
  } else if (vec) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (c < cnt) p[c] = v[c];
  }
}

// Per-step (c1, c2, sigma, 1/c2): from the target's float32 table when given,
// else evaluated from the schedule in float64 and rounded.
__device__ __forceinline__ float4 step_coef(const Sched& sc, const float4* __restrict__ coef, int n) {
  if (coef) return coef[n];
  const double c2 = sched_c2(sc, n);
  return make_float4((float)sched_c1(sc, n), (float)c2, (float)sched_sigma(sc, n), (float)(1.0 / c2));
}

// The Free Drafter's mean m^p = c1_n yhat + c2s sv with c2s = c2_n / c2_c and
// sv = c2_c S_c, in one fixed sequence of float32 operations (the product,
// then one fused multiply-add), so that every kernel that needs m^p recomputes
// the same bits as the draft that produced yhat.
__device__ __forceinline__ float draft_mean(float c1, float y, float c2s, float sv) {
  return __fmaf_rn(c1, y, c2s * sv);
}

// Draft rows 1..K of one chain for coordinates e0..e0+3 (group g), starting
// at yhat_0 = yv (already stored as row 0 by the caller) and step k with
// K_b = kb valid drafts (Sec. 3.3):
//   m^p_{i-1} = c1_n yhat_{i-1} + c2_n S_c,  yhat_i = m^p_{i-1} + sigma_n xi_i,
// where c2_n S_c = (c2_n * scale) * sv; rows past K_b repeat the last draft
// and mean so that every row the target call reads is finite.  mb may be
// null (the sampler recomputes m^p where it needs it, see draft_mean).
// stream: the rows are written with non-temporal stores (stream_rows).
__device__ __forceinline__ void draft_rows(const Sched& sc, const float4* __restrict__ coef, int K,
                                           int k, int kb, uint32_t chain, uint32_t rnd,
                                           uint64_t seed, int g, float (&yv)[4],
                                           const float (&sv)[4], float scale, float* xb,
                                           int64_t xr, float* mb, int64_t mr, int cnt, bool vec,
                                           bool stream) {
  float m[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = 1; i <= kb; ++i) {
    const int n = k + i - 1;
    const float4 cf = step_coef(sc, coef, n);
    const float c2 = cf.y * scale;
    const float4 z = normals4(philox((uint32_t)g, chain, rnd, (TAG_DRAFT << 24) | (uint32_t)i, seed));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      m[c] = draft_mean(cf.x, yv[c], c2, sv[c]);
      yv[c] = m[c] + cf.z * get4(z, c);
    }
    if (mb) store4(mb + (int64_t)(i - 1) * mr, cnt, vec, m, stream);
    store4(xb + (int64_t)i * xr, cnt, vec, yv, stream);
  }
  for (int i = kb + 1; i <= K; ++i) {
    if (mb) store4(mb + (int64_t)(i - 1) * mr, cnt, vec, m, stream);
    store4(xb + (int64_t)i * xr, cnt, vec, yv, stream);
  }
}

}  // namespace sd
