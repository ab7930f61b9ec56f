// Raw buffer views for the GEMM kernels' aligned paths: loads past a view's
// end return zero and stores past it are dropped by the hardware, so tile
// edges need no branches and every load is issued unconditionally (which lets
// the compiler wait for exactly the loads it needs: the hardware counts
// outstanding loads in issue order).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

constexpr uint32_t kBufferWord3 = 0x00020000;  // raw buffer, 32-bit dwords (gfx9 family)

// A view of `bytes` bytes at p (bytes < 2^31).  The base and size are
// wavefront-uniform; readfirstlane says so, or the compiler would wrap every
// access in a loop over distinct descriptors.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_view(const void* p, int64_t bytes) {
  const uint64_t base = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)base);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(base >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)(bytes < 0 ? 0 : bytes));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(((uint64_t)hi << 32) | lo),
                                           (short)0, n, (int)kBufferWord3);
}

__device__ __forceinline__ float4 buf_ld4(__amdgpu_buffer_rsrc_t v, uint32_t off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(v, off, 0, 0));
}

__device__ __forceinline__ uint4 buf_ld16(__amdgpu_buffer_rsrc_t v, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(v, off, 0, 0));
}

__device__ __forceinline__ void buf_st4(__amdgpu_buffer_rsrc_t v, uint32_t off, float4 x) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), v, off, 0, 0);
}

// A non-temporal (streaming) store (cache policy bit 1, NT on gfx950): for
// outputs of which the next kernels read back only a small part, so that
// they do not displace the lines that are read again from the caches.
__device__ __forceinline__ void buf_st4_stream(__amdgpu_buffer_rsrc_t v, uint32_t off, float4 x) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), v, off, 0, 2);
}

}  // namespace sd
