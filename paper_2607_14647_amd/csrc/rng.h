// Device helpers shared by the sampling kernels: the order-preserving float
// key, the Philox4x32-10 counter-based generator and the Gumbel transform.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dcut {

// Order-preserving map of a float to an unsigned key (larger float, larger key;
// -inf maps above 0, so a key of 0 means "no candidate").
__device__ __forceinline__ uint32_t orderable(float v) {
  uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// The same key without a select: the sign smeared by an arithmetic shift,
// with the top bit set, flips the magnitude bits of negative values only.
__device__ __forceinline__ uint32_t order_key(float v) {
  const uint32_t u = __float_as_uint(v);
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

// Philox4x32 with ten rounds (Salmon, Moraes, Dror, Shaw, SC 2011): each round
// multiplies words 0 and 2 by the two Philox constants and mixes the high and
// low halves with words 1 and 3 and the key; the key advances by the two Weyl
// constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
  }
  return c;
}

// Standard Gumbel variate -ln(-ln u) for u = (w + 0.5) / 2^32, with the
// hardware base-2 logarithm (v_log_f32, about one ulp).  t = -ln u comes from u
// itself when u < 1/2; otherwise from x = 1 - u (exact in float): by the series
// x + x^2/2 + x^3/3 + x^4/4 when x < 1/32 (relative error below x^4/5 < 2^-22),
// else as -ln(1 - x) with 1 - x rounded (relative error below 2^-24 / x <=
// 2^-19).  t so keeps its relative accuracy as u approaches 1, where the
// largest variates come from.  Both branches share one logarithm and are
// selected per lane, so lanes never diverge, and nothing divides.
__device__ __forceinline__ float gumbel_of(uint32_t w) {
  constexpr float LN2 = 0.6931471805599453f;
  const bool lo = w < 0x80000000u;
  const float u = ((float)w + 0.5f) * 0x1p-32f;
  const float x = ((float)(0xffffffffu - w) + 0.5f) * 0x1p-32f;
  const float l = __log2f(lo ? u : 1.0f - x) * LN2;    // one logarithm for either branch
  const float s = x * (1.0f + x * (0.5f + x * (1.0f / 3.0f + x * 0.25f)));
  const float t = (lo || x >= 0x1p-5f) ? -l : s;
  return -__log2f(t) * LN2;
}

// Uniform on (0, 1) from one Philox output word: (w + 0.5) / 2^32 in float64.
__device__ __forceinline__ double uniform01(uint32_t w) { return ((double)w + 0.5) * 0x1p-32; }

}  // namespace dcut
