// Calibration of the bf16 matrix cores: a loop of v_mfma_f32_32x32x16_bf16 on
// register operands, with no memory traffic inside it, to measure the rate
// this GPU sustains (its clock under full matrix load) beside the published
// dense peak.  Each wavefront keeps four independent accumulators so that
// consecutive instructions do not wait on each other's results.
#include "common.hpp"

namespace sd {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kChains = 4;

__global__ __launch_bounds__(kThreads) void mfma_loop_kernel(int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(lane + i));
    b[i] = (__bf16)(0.002f * (float)(lane - i));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  // one value per wavefront keeps the loop live
  if (lane == 0) out[blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)] = s;
}

}  // namespace

hipError_t mfma_loop_launch(int blocks, int iters, float* out, hipStream_t s) {
  return launch_timed("mfma_loop", mfma_loop_kernel, dim3(blocks), dim3(kThreads), s, iters, out);
}

}  // namespace sd
