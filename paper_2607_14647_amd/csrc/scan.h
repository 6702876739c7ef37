// Workgroup-wide exclusive prefix sum (wave shuffles, then one pass over wave totals).
#pragma once
#include <hip/hip_runtime.h>

namespace dcut {

// blockDim.x must be a multiple of 64 and at most 1024.  `s_wave` holds 17
// entries of LDS.  Returns the exclusive prefix of `v`; *total gets the sum.
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T *s_wave, T *total) {
  const int lane = threadIdx.x & 63;
  const int wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  T x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    T y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) s_wave[wid] = x;
  __syncthreads();
  if (wid == 0) {
    T w = lane < nw ? s_wave[lane] : T(0);
    T z = w;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      T y = __shfl_up(z, off, 64);
      if (lane >= off) z += y;
    }
    if (lane < nw) s_wave[lane] = z - w;
    if (lane == nw - 1) s_wave[16] = z;
  }
  __syncthreads();
  T res = x - v + s_wave[wid];
  *total = s_wave[16];
  __syncthreads();
  return res;
}

}  // namespace dcut
