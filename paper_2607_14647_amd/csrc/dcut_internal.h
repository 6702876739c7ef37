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

// Cache-policy bits of a vector memory instruction (the last operand of the
// buffer-load builtins): nt marks a load as streaming (non-temporal).
constexpr int CPOL_NT = 2;

// RoPE (rotate-half) of the pair (x1, x2) = dimensions (j, j + hd/2) of one row,
// cs = (cos, sin) of the row's position and frequency j.
__device__ __forceinline__ float2 rope_pair(float x1, float x2, float2 cs) {
  return make_float2(x1 * cs.x - x2 * cs.y, x2 * cs.x + x1 * cs.y);
}

// Split-K partial sums in split order, with the loads of four splits issued
// together (one memory round trip per four splits).  load(s) returns split s;
// indices past the last split re-read it, and the adds are selects rather than
// branches, so the compiler keeps each batch of loads together.
struct f4x2 {
  float4 a, b;
};
__device__ __forceinline__ float2 add_if(bool use, float2 x, float2 y) {
  return make_float2(use ? x.x + y.x : x.x, use ? x.y + y.y : x.y);
}
__device__ __forceinline__ float4 add_if(bool use, float4 x, float4 y) {
  return make_float4(use ? x.x + y.x : x.x, use ? x.y + y.y : x.y, use ? x.z + y.z : x.z,
                     use ? x.w + y.w : x.w);
}
__device__ __forceinline__ f4x2 add_if(bool use, f4x2 x, f4x2 y) {
  return f4x2{add_if(use, x.a, y.a), add_if(use, x.b, y.b)};
}
template <typename T, typename Load>
__device__ __forceinline__ T sum_splits(int splits, Load load) {
  T v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) v[u] = load(u < splits ? u : splits - 1);
  T acc = v[0];
#pragma unroll
  for (int u = 1; u < 4; ++u) acc = add_if(u < splits, acc, v[u]);
  for (int s0 = 4; s0 < splits; s0 += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = load(s0 + u < splits ? s0 + u : splits - 1);
#pragma unroll
    for (int u = 0; u < 4; ++u) acc = add_if(s0 + u < splits, acc, v[u]);
  }
  return acc;
}

// ---------------------------------------------------------------- profiling hook
struct ProfileHook {
  int kernel;
  hipEvent_t start, stop;
};
ProfileHook &profile_hook();

// Allow `kernel` to use `bytes` of dynamic LDS (needed above 64 KB).  The
// attribute is set once per kernel and size for each host thread (a small
// per-thread table of what it set; setting it again from another thread is
// harmless).
template <typename Kernel>
inline void allow_lds(Kernel kernel, size_t bytes) {
  if (bytes <= 65536) return;
  static thread_local const void *done_fn[64];
  static thread_local size_t done_bytes[64];
  static thread_local int n_done = 0;
  const void *f = (const void *)kernel;
  const int n = n_done < 64 ? n_done : 64;
  for (int j = 0; j < n; ++j)
    if (done_fn[j] == f && done_bytes[j] >= bytes) return;
  if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) == hipSuccess && n_done < 64) {
    done_fn[n_done] = f;
    done_bytes[n_done] = bytes;
    ++n_done;
  }
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
  EPI_ARGMAX = 4,       // per-row max/argmax: one u64 key per row and wave column range
  EPI_STORE_F32 = 5,    // out_f32[m][n] = acc
  EPI_SAMPLE = 6        // as EPI_ARGMAX on acc * inv_temp + Gumbel noise (temperature sampling)
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
  int n_req;                      // requests in the batch: rows whose packed_req is outside [0, n_req) are skipped
  // EPI_ARGMAX
  unsigned long long *amax_keys;  // [M_max][amax_slots]: per-row maxima of column ranges
  int amax_slots;                 // row stride of amax_keys, at least both gemm_argmax_slots() counts
  // EPI_SAMPLE: noise of column c at row t is keyed by (seed, row_req[t], row_pos[t], c)
  float inv_temp;
  uint32_t seed_lo, seed_hi;
  const int32_t *row_req, *row_pos;
  float2 *lse_part;               // EPI_SAMPLE, optional [M_max][amax_slots]: per column range
                                  // (max x, sum exp(x - max)) of x = acc * inv_temp
  float *logits;                  // optional [M][N] float32
  long long ld_logits;
  // split-K (EPI_RESID_F32 / EPI_STORE_F32): partial tiles [splits][M_max][N] float32
  int splits;
  float *split_part;
  int defer_reduce;               // with splits > 1: leave the partials for the caller to add
  // grouped mode (MoE experts): row tiles come from a device list of
  // (expert, first row, end row); W advances by w_stride elements per expert;
  // A rows are gathered through a_rows when it is not null.
  const int32_t *tiles;
  const int32_t *n_tiles;
  int m_tiles;              // grid rows of tiles (upper bound of *n_tiles)
  long long w_stride;
  const int32_t *a_rows;
  int a_extent;             // rows in the A buffer (0: M_max)
};

int gemm_launch(int kid, EpiKind epi, const GemmArgs &a, hipStream_t s);
// number of per-row partial argmax keys EPI_ARGMAX writes for this shape (at most 2 * ceil(N / 128))
// The LM-head GEMM with the argmax epilogue takes its tile on the device from
// the live row count M: 128 x 256 tiles with a four-slice W ring when the last
// 256-row tile would be at most half full, 256 x 256 tiles otherwise.  Both
// give bitwise the same results.
__host__ __device__ inline bool lm_head_mid_tile(int M) { return M > 0 && M % 256 != 0 && M % 256 <= 128; }
// Partial-key slots per row the argmax/sample GEMM writes: *big when the live
// rows take the 256 x 256 tile, *mid when they take the 128 x 256 one (equal
// when the launch makes no such choice).  The row stride must hold the larger.
void gemm_argmax_slots(const GemmArgs &a, EpiKind epi, int *big, int *mid);
// split-K factor for a residual GEMM of this shape (a function of the shapes and the CU count,
// never of K*)
int gemm_splits(int M_max, int N, int K);
// Whether the GEMM kernel's 32-bit buffer offsets reach every operand element:
// a_rows rows of A at stride lda (what one task addresses: a row tile of at
// most 256 rows, or all of A when rows are gathered) and w_rows rows of W at
// stride ldw (the span of one column tile: 256 rows, or the SwiGLU split point
// plus 256 since a tile pairs gate and up rows).  Operands of any total size
// pass as long as these spans stay below 2 GiB.
inline bool gemm_span_ok(long long a_rows, long long lda, long long w_rows, long long ldw) {
  const long long lim = 0x7fffffffLL - 256;
  return a_rows * lda * 2 < lim && w_rows * ldw * 2 < lim;
}

// ---------------------------------------------------------------- other launchers
// x[m] += sum of the split-K partials part[s][m] (in split order), then
// h[m] = RMSNorm(x[m]) * gain: the residual add of a split-K GEMM fused with the
// norm that reads its result.  One workgroup per live row; H % 8 == 0, H <= 8192.
int reduce_rmsnorm_launch(int kid, const float *part, int splits, int M_max, int H, const int32_t *m_count,
                          float *x, const uint16_t *gain, float eps, uint16_t *h_out, hipStream_t s);
struct AttnArgs;
// Row RMSNorm over the live rows (see norm.hip).  With `plan` (nullable; B <=
// 1024 and plan->plan set) one extra workgroup also writes that attention
// call's work order.
int rmsnorm_launch(int kid, const float *x_in, const uint16_t *embed, const int32_t *tok, int vocab,
                   const uint16_t *gain, float eps, int H, int M_max, const int32_t *m_count,
                   float *x_copy, uint16_t *h_out, const int32_t *pos, int head_dim, float theta,
                   float2 *rope_cs, unsigned long long *amax_init, int32_t *dev_err, const AttnArgs *plan,
                   hipStream_t s);

// Routed MoE MLP over the rows of h (bf16, [M_max][H]); adds into x_out.
struct MoeArgs {
  const uint16_t *h;
  const uint16_t *w_router, *w_gate_up, *w_down;
  int H, E, top_k, inter, M_max;
  const int32_t *m_count;
  float *x_out;
  void *ws;                 // moe_ws_bytes() bytes
};
size_t moe_ws_bytes(int M_max, int H, int E, int top_k, int inter);
bool moe_supported(int M_max, int H, int E, int top_k);
int moe_launch(const MoeArgs &m, hipStream_t s);

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
  int32_t *plan;            // work-order scratch of attn_plan_bytes(B, n_kv, max_chunks), or null
};
// Bytes of the attention work-order plan (0: the batch is too large to plan and
// the items run in chunk-slowest order).
size_t attn_plan_bytes(int B, int n_kv, int max_chunks);
int attention_launch(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves,
                     hipStream_t s);

}  // namespace dcut
