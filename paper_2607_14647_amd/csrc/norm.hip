// Row RMSNorm: h = x / sqrt(mean(x^2) + eps) * gain, float32 in, bf16 out.
//
// One 256-thread workgroup per packed row, rows at or beyond K* exit.  The
// same pass optionally gathers the input from the embedding table (the first
// norm of the layer), keeps a float32 copy of the residual, writes the
// row's RoPE (cos, sin) table and clears the row's argmax key.  The sum of
// squares is reduced in a fixed order, so the result is deterministic.
//
// The first norm of a layer also builds the attention work order in one extra
// workgroup ahead of the rows (attn_plan.h): it needs only the batch layout,
// which is known at the start of the layer, and running beside the rows it
// costs no launch of its own.
#include "attn_plan.h"
#include "dcut_internal.h"

namespace dcut {

namespace {

__global__ void __launch_bounds__(256)
k_rmsnorm(const float *__restrict__ x_in, const uint16_t *__restrict__ embed,
          const int32_t *__restrict__ tok, int vocab, const uint16_t *__restrict__ gain, float eps,
          int H, const int32_t *__restrict__ m_count, float *__restrict__ x_copy,
          uint16_t *__restrict__ h_out, const int32_t *__restrict__ pos, int head_dim, float theta,
          float2 *__restrict__ rope_cs, unsigned long long *__restrict__ amax_init,
          int32_t *__restrict__ dev_err, AttnArgs plan) {
  __shared__ float s_red[4];
  extern __shared__ __align__(16) int plan_lds[];
  // the plan workgroup is dispatched first: it takes longer than a row
  if (plan.plan && blockIdx.x == 0) {
    attn_plan_block<256>(plan, plan_lds);
    return;
  }
  const int t = blockIdx.x - (plan.plan ? 1 : 0);
  if (t >= *m_count) return;
  const int tid = threadIdx.x;

  const float *xr = nullptr;
  const uint16_t *er = nullptr;
  if (x_in) {
    xr = x_in + (size_t)t * H;
  } else {
    int tk = tok[t];
    if (tk < 0 || tk >= vocab) {
      if (tid == 0 && dev_err) atomicOr(dev_err, DCUT_DERR_TOKEN);
      tk = 0;
    }
    er = embed + (size_t)tk * H;
  }
  // each thread owns 8-element groups g = tid, tid + 256, ...
  const int ng = H / 8;
  float ss = 0.0f;
  if (ng <= 4 * 256) {
    // the row in registers: every load issued at once, the row read once, and the
    // same sum of squares (groups ascending, elements ascending) as the loop below
    float v[4][8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gi = tid + 256 * q;
      if (gi >= ng) break;
      if (xr) {
        const float4 a = *(const float4 *)(xr + gi * 8), b = *(const float4 *)(xr + gi * 8 + 4);
        v[q][0] = a.x; v[q][1] = a.y; v[q][2] = a.z; v[q][3] = a.w;
        v[q][4] = b.x; v[q][5] = b.y; v[q][6] = b.z; v[q][7] = b.w;
      } else {
        uint4 u = *(const uint4 *)(er + gi * 8);
        const uint16_t *e = (const uint16_t *)&u;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[q][j] = bf2f(e[j]);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gi = tid + 256 * q;
      if (gi >= ng) break;
      if (x_copy && x_copy != x_in) {
        float *dst = x_copy + (size_t)t * H + gi * 8;
        *(float4 *)dst = make_float4(v[q][0], v[q][1], v[q][2], v[q][3]);
        *(float4 *)(dst + 4) = make_float4(v[q][4], v[q][5], v[q][6], v[q][7]);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) ss += v[q][j] * v[q][j];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    if ((tid & 63) == 0) s_red[tid >> 6] = ss;
    __syncthreads();
    const float tot = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
    const float r = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int gi = tid + 256 * q;
      if (gi >= ng) break;
      uint4 gv = *(const uint4 *)(gain + gi * 8);
      const uint16_t *gg = (const uint16_t *)&gv;
      uint4 o;
      uint32_t *ow = (uint32_t *)&o;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        ow[j] = pack_bf2(v[q][2 * j] * r * bf2f(gg[2 * j]), v[q][2 * j + 1] * r * bf2f(gg[2 * j + 1]));
      *(uint4 *)(h_out + (size_t)t * H + gi * 8) = o;
    }
  } else {
    for (int gi = tid; gi < ng; gi += 256) {
      float v[8];
      if (xr) {
        float4 a = *(const float4 *)(xr + gi * 8);
        float4 b = *(const float4 *)(xr + gi * 8 + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
      } else {
        uint4 u = *(const uint4 *)(er + gi * 8);
        const uint16_t *e = (const uint16_t *)&u;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = bf2f(e[j]);
      }
      if (x_copy && x_copy != x_in) {
        float *dst = x_copy + (size_t)t * H + gi * 8;
        *(float4 *)dst = make_float4(v[0], v[1], v[2], v[3]);
        *(float4 *)(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) ss += v[j] * v[j];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
    if ((tid & 63) == 0) s_red[tid >> 6] = ss;
    __syncthreads();
    const float tot = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
    const float r = 1.0f / sqrtf(tot / (float)H + eps);
    for (int gi = tid; gi < ng; gi += 256) {
      float v[8];
      if (xr) {
        float4 a = *(const float4 *)(xr + gi * 8);
        float4 b = *(const float4 *)(xr + gi * 8 + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
      } else {
        uint4 u = *(const uint4 *)(er + gi * 8);
        const uint16_t *e = (const uint16_t *)&u;
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = bf2f(e[j]);
      }
      uint4 gv = *(const uint4 *)(gain + gi * 8);
      const uint16_t *gg = (const uint16_t *)&gv;
      uint4 o;
      uint32_t *ow = (uint32_t *)&o;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        ow[j] = pack_bf2(v[2 * j] * r * bf2f(gg[2 * j]), v[2 * j + 1] * r * bf2f(gg[2 * j + 1]));
      *(uint4 *)(h_out + (size_t)t * H + gi * 8) = o;
    }
  }
  if (rope_cs) {
    const int half = head_dim >> 1;
    const double p = (double)pos[t];
    for (int j = tid; j < half; j += 256) {
      double inv = exp2(-(2.0 * j / head_dim) * log2((double)theta));
      double ang = p * inv;
      rope_cs[(size_t)t * half + j] = make_float2((float)cos(ang), (float)sin(ang));
    }
  }
  if (amax_init && tid == 0) amax_init[t] = 0ull;
}

// Split-K residual add and the following RMSNorm in one pass over the row.
__global__ void __launch_bounds__(256)
k_reduce_rmsnorm(const float *__restrict__ part, int splits, int M_max, int H,
                 const int32_t *__restrict__ m_count, float *__restrict__ x, const uint16_t *__restrict__ gain,
                 float eps, uint16_t *__restrict__ h_out) {
  __shared__ float s_red[4];
  const int t = blockIdx.x;
  if (t >= *m_count) return;
  const int tid = threadIdx.x;
  const int ng = H / 8;
  float v[4][8];                         // this thread's 8-element groups g = tid + 256 q
  float ss = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int gi = tid + 256 * q;
    if (gi >= ng) break;
    float *xr = x + (size_t)t * H + gi * 8;
    const float4 xa = *(const float4 *)xr, xb = *(const float4 *)(xr + 4);
    const f4x2 sum = sum_splits<f4x2>(splits, [&](int sp) {
      const float *ps = part + ((size_t)sp * M_max + t) * H + gi * 8;
      return f4x2{*(const float4 *)ps, *(const float4 *)(ps + 4)};
    });
    float4 a = sum.a, b = sum.b;
    a.x += xa.x; a.y += xa.y; a.z += xa.z; a.w += xa.w;
    b.x += xb.x; b.y += xb.y; b.z += xb.z; b.w += xb.w;
    *(float4 *)xr = a;
    *(float4 *)(xr + 4) = b;
    v[q][0] = a.x; v[q][1] = a.y; v[q][2] = a.z; v[q][3] = a.w;
    v[q][4] = b.x; v[q][5] = b.y; v[q][6] = b.z; v[q][7] = b.w;
#pragma unroll
    for (int j = 0; j < 8; ++j) ss += v[q][j] * v[q][j];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off, 64);
  if ((tid & 63) == 0) s_red[tid >> 6] = ss;
  __syncthreads();
  const float tot = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
  const float r = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int gi = tid + 256 * q;
    if (gi >= ng) break;
    uint4 gv = *(const uint4 *)(gain + gi * 8);
    const uint16_t *gg = (const uint16_t *)&gv;
    uint4 o;
    uint32_t *ow = (uint32_t *)&o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      ow[j] = pack_bf2(v[q][2 * j] * r * bf2f(gg[2 * j]), v[q][2 * j + 1] * r * bf2f(gg[2 * j + 1]));
    *(uint4 *)(h_out + (size_t)t * H + gi * 8) = o;
  }
}

}  // namespace

int reduce_rmsnorm_launch(int kid, const float *part, int splits, int M_max, int H, const int32_t *m_count,
                          float *x, const uint16_t *gain, float eps, uint16_t *h_out, hipStream_t s) {
  if (H % 8 || H > 8 * 256 * 4 || splits < 1) return DCUT_EINVAL;
  return launch(kid, k_reduce_rmsnorm, dim3(M_max), dim3(256), 0, s, part, splits, M_max, H, m_count, x, gain,
                eps, h_out);
}

int rmsnorm_launch(int kid, const float *x_in, const uint16_t *embed, const int32_t *tok, int vocab,
                   const uint16_t *gain, float eps, int H, int M_max, const int32_t *m_count,
                   float *x_copy, uint16_t *h_out, const int32_t *pos, int head_dim, float theta,
                   float2 *rope_cs, unsigned long long *amax_init, int32_t *dev_err, const AttnArgs *plan,
                   hipStream_t s) {
  AttnArgs p = {};
  size_t lds = 0;
  if (plan && plan->plan) {
    if (plan->B > PLAN_MAX_B) return DCUT_EINVAL;
    p = *plan;
    lds = attn_plan_lds_bytes(p.B, 256);
  }
  return launch(kid, k_rmsnorm, dim3(M_max + (p.plan ? 1 : 0)), dim3(256), lds, s, x_in, embed, tok, vocab, gain,
                eps, H, m_count, x_copy, h_out, pos, head_dim, theta, rope_cs, amax_init, dev_err, p);
}

}  // namespace dcut
