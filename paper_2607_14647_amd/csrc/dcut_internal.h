// Internal helpers shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

#include "dcut.h"

namespace dcut {

// ---------------------------------------------------------------- bf16 / vector types
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bf16 bits, round to nearest even (finite inputs; NaN kept quiet)
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// ---------------------------------------------------------------- profiling hook
struct ProfileHook {
  int kernel;
  hipEvent_t start, stop;
};
ProfileHook &profile_hook();

// Allow `kernel` to use `bytes` of dynamic LDS (needed above 64 KB); done once per kernel.
template <typename Kernel>
inline void allow_lds(Kernel kernel, size_t bytes) {
  if (bytes > 65536) hipFuncSetAttribute((const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

// Launch `kernel`, recording the armed profiling events around it when `kid` is armed.
template <typename Kernel, typename... Args>
inline int launch(int kid, Kernel kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t s,
                  Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return DCUT_OK;
  allow_lds(kernel, shmem);
  ProfileHook &h = profile_hook();
  if (kid != DCUT_KERNEL_NONE && h.kernel == kid) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, h.start, h.stop, 0, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
  return hipGetLastError() == hipSuccess ? DCUT_OK : DCUT_EHIP;
}

#define DCUT_TRY(expr)              \
  do {                              \
    int _st = (expr);               \
    if (_st != DCUT_OK) return _st; \
  } while (0)

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Validation shared by the entry points.
inline bool batch_ok(int B, int D) {
  return B >= 1 && B <= DCUT_MAX_BATCH && D >= 0 && D + 1 <= DCUT_MAX_BLOCK &&
         (long long)B * (D + 1) <= DCUT_MAX_ROWS;
}

// ---------------------------------------------------------------- GEMM interface
// C[M][N] = A[M][K] * W[N][K]^T in bf16 with float32 accumulation, for the rows
// m < M_dev = *m_count (device), launched for M_max rows.
enum EpiKind {
  EPI_STORE_BF16 = 0,   // out_bf16[m][n]
  EPI_RESID_F32 = 1,    // out_f32[m][n] += acc   (residual add, in place)
  EPI_SWIGLU = 2,       // W rows interleaved by tile: out_bf16[m][j] = SiLU(gate) * up
  EPI_QKV_ROPE = 3,     // RoPE + scatter q to out_bf16, k/v into the cache
  EPI_ARGMAX = 4        // per-row max/argmax merged with 64-bit atomics
};

struct GemmArgs {
  const uint16_t *A;     // [M][K] bf16, row stride lda
  const uint16_t *W;     // [N][K] bf16, row stride ldw
  int M_max, N, K, lda, ldw;
  const int32_t *m_count;  // device row count (K*), read by every workgroup
  // epilogue operands
  uint16_t *out_bf16;
  float *out_f32;
  int ldo;
  int swiglu_inter;        // EPI_SWIGLU: gate/up split point in W rows
  // EPI_QKV_ROPE
  const int32_t *packed_pos, *packed_req, *ctx_len;
  const float2 *rope_cs;   // [M_max][head_dim/2] (cos, sin)
  uint16_t *kv_k, *kv_v;
  const int64_t *kv_base;
  const int32_t *kv_cap;
  int n_q, n_kv, head_dim;
  // EPI_ARGMAX
  unsigned long long *amax_keys;  // [M_max]
  float *logits;                  // optional [M][N] float32
  long long ld_logits;
};

int gemm_launch(int kid, EpiKind epi, const GemmArgs &a, hipStream_t s);

// ---------------------------------------------------------------- other launchers
int rmsnorm_launch(int kid, const float *x_in, const uint16_t *embed, const int32_t *tok, int vocab,
                   const uint16_t *gain, float eps, int H, int M_max, const int32_t *m_count,
                   float *x_copy, uint16_t *h_out, const int32_t *pos, int head_dim, float theta,
                   float2 *rope_cs, unsigned long long *amax_init, int32_t *dev_err, hipStream_t s);

struct AttnArgs {
  const uint16_t *q;        // [M][n_q][hd] bf16 (after RoPE)
  const uint16_t *kv_k, *kv_v;
  const int64_t *kv_base;
  const int32_t *kv_cap;
  const int32_t *cu, *ctx_len;
  int B, D, n_q, n_kv, head_dim, chunk, max_chunks;
  float *part;              // [M_max][n_q][max_chunks][hd + 2]
  uint16_t *out;            // [M][n_q][hd] bf16
  int32_t *dev_err;
};
int attention_launch(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves,
                     hipStream_t s);

}  // namespace dcut
