// Deterministic sums of per-row values over the 16 lanes of a column group.
#pragma once

#include <hip/hip_runtime.h>

namespace sd {

// Each of the 16 lanes (lane index cg in the group) holds NR per-row partial
// sums (NR = 4 or 8) of the same NR rows.  Butterfly reduce-scatter: the
// exchanges at distance 8, 4 (and 2 for NR = 8) halve the rows a lane keeps,
// the remaining exchanges complete the sum, so lane cg ends with the total of
// row row_of<NR>(cg) over all 16 lanes (lanes that differ only in the low
// bits hold the same row).  Fixed order, hence deterministic.
template <int NR>
__device__ __forceinline__ int row_of(int cg) {
  return NR == 8 ? 4 * ((cg >> 3) & 1) + 2 * ((cg >> 2) & 1) + ((cg >> 1) & 1)
                 : 2 * ((cg >> 3) & 1) + ((cg >> 2) & 1);
}

template <int NR>
__device__ __forceinline__ double reduce_rows16(const double (&v)[NR], int cg) {
  static_assert(NR == 4 || NR == 8, "4 or 8 rows per lane");
  constexpr int H = NR / 2;
  const bool b3 = cg & 8, b2 = cg & 4, b1 = cg & 2;
  double w[H];
#pragma unroll
  for (int i = 0; i < H; ++i) {
    const double send = b3 ? v[i] : v[i + H];
    w[i] = (b3 ? v[i + H] : v[i]) + __shfl_xor(send, 8);
  }
  constexpr int Q = H / 2;
  double u[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const double send = b2 ? w[i] : w[i + Q];
    u[i] = (b2 ? w[i + Q] : w[i]) + __shfl_xor(send, 4);
  }
  double z;
  if constexpr (NR == 8) {
    z = (b1 ? u[1] : u[0]) + __shfl_xor(b1 ? u[0] : u[1], 2);
  } else {
    z = u[0] + __shfl_xor(u[0], 2);
  }
  return z + __shfl_xor(z, 1);
}

}  // namespace sd
