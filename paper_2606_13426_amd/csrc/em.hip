// The plain Euler-Maruyama chain Y_{n+1} = m^q_n(Y_n) + sigma_n xi_n of the
// VP-SDE (Sec. 2): the non-speculative sampler that speculative sampling must
// reproduce in law and whose target calls it saves.  A step is one target call
// on the B states followed by this elementwise kernel, which adds the noise
// (TARGET stream of chain b, round n, slot 1) and sets the next call's step.
#include "common.hpp"
#include "philox.hpp"
#include "rows.hpp"

namespace sd {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void em_noise_kernel(int d, int n, float sigma_n,
                                                            uint64_t seed,
                                                            const float* __restrict__ mq,
                                                            float* __restrict__ y,
                                                            int32_t* __restrict__ step,
                                                            bool vec_ok) {
  const int b = blockIdx.y;
  const int g = blockIdx.x * kThreads + threadIdx.x;
  if (g == 0) step[b] = n + 1;
  const int e0 = 4 * g;
  if (e0 >= d) return;
  const int cnt = min(4, d - e0);
  const bool vec = vec_ok && cnt == 4;
  float q[4], v[4];
  load4(mq + (int64_t)b * d + e0, cnt, vec, q);
  const float4 z = normals4(philox((uint32_t)g, (uint32_t)b, (uint32_t)n, (TAG_TARGET << 24) | 1u, seed));
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = q[c] + sigma_n * get4(z, c);
  store4(y + (int64_t)b * d + e0, cnt, vec, v);
}

}  // namespace

hipError_t em_noise_launch(int B, int d, int n, float sigma_n, uint64_t seed, const float* mq,
                           float* y, int32_t* step, hipStream_t s) {
  const int ng = (d + 3) / 4;
  dim3 grid((ng + kThreads - 1) / kThreads, B);
  const bool vec = (d % 4 == 0) && aligned16(mq) && aligned16(y);
  return timed("em_noise", s, [&] {
    em_noise_kernel<<<grid, kThreads, 0, s>>>(d, n, sigma_n, seed, mq, y, step, vec);
  });
}

}  // namespace sd
