// dcut_lm_head_argmax: final RMSNorm, LM-head GEMM with a fused row argmax.
// dcut_lm_head_sample: the same with temperature sampling (Gumbel-max) fused in,
// optionally also writing the logits and each row's log-partition function
// (what rejection-sampling verification needs).
//
// The GEMM epilogue reduces each row's column ranges of the vocabulary (64 or
// 128 columns, by tile shape) to one 64-bit key each (order-preserving logit
// bits << 32 | ~column) and stores them; a second pass takes the maximum key
// of every row.  The full logits are
// never written, no atomics contend on a row, the result does not depend on
// workgroup order, and the lowest column wins exact ties.
#include <atomic>
#include <mutex>

#include "dcut_internal.h"

namespace dcut {

// Scratch of the LM-head call: the normalised rows, the partial keys and (for a
// sampling call that returns the log-partition) the partial (max, sum) pairs.
static size_t lmhead_need(int H, int V, int B, int D, bool with_lse) {
  const size_t M = (size_t)B * (D + 1);
  const size_t slots = 4 * (((size_t)V + 255) / 256);   // row stride of the partial keys (64 columns each)
  return align256(M * H * 2) + (with_lse ? 2 : 1) * align256(M * slots * sizeof(unsigned long long));
}

size_t lmhead_ws_bytes(int H, int V, int B, int D) { return lmhead_need(H, V, B, D, true); }

namespace {

// One workgroup per row: the maximum of the row's partial keys, decoded; with
// `lse`, also ln sum_c exp(logits[c] * inv_temp) merged from the row's
// per-range (max, rescaled sum) pairs.
__device__ __forceinline__ void lse_merge(float &m, float &s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == -__builtin_inff()) return;      // both empty
  s = s * __expf(m - M) + s2 * __expf(m2 - M);
  m = M;
}

__global__ void __launch_bounds__(256)
k_argmax_final(const unsigned long long *__restrict__ keys, const float2 *__restrict__ part, int slots_big,
               int slots_mid, int stride, const int32_t *__restrict__ m_count, int M_max,
               int32_t *__restrict__ argmax, float *__restrict__ max_logit, float *__restrict__ lse) {
  __shared__ unsigned long long s_max[4];
  __shared__ float s_m[4], s_s[4];
  const int t = blockIdx.x;
  const int M = *m_count;
  if (t >= M_max || t >= M) return;
  const int slots = lm_head_mid_tile(M) ? slots_mid : slots_big;   // the GEMM's own tile choice
  const int tid = threadIdx.x, lane = tid & 63;
  const unsigned long long *row = keys + (size_t)t * stride;
  unsigned long long k = 0ull;
  float m = -__builtin_inff(), sum = 0.0f;
  // four slots per thread per memory round trip (one round trip for up to 1024
  // slots), merged in the order s = tid, tid + 256, ...
  for (int s0 = tid; s0 < slots; s0 += 1024) {
    unsigned long long v[4];
    float2 p[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = s0 + 256 * u;
      v[u] = s < slots ? row[s] : 0ull;
      if (lse) p[u] = s < slots ? part[(size_t)t * stride + s] : make_float2(0.0f, 0.0f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      k = v[u] > k ? v[u] : k;
      if (lse && s0 + 256 * u < slots) lse_merge(m, sum, p[u].x, p[u].y);
    }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned long long o = __shfl_xor(k, off, 64);
    k = o > k ? o : k;
    if (lse) {
      const float m2 = __shfl_xor(m, off, 64), s2 = __shfl_xor(sum, off, 64);
      lse_merge(m, sum, m2, s2);
    }
  }
  if (lane == 0) {
    s_max[tid >> 6] = k;
    s_m[tid >> 6] = m;
    s_s[tid >> 6] = sum;
  }
  __syncthreads();
  if (tid != 0) return;
  for (int w = 1; w < 4; ++w) {
    k = s_max[w] > k ? s_max[w] : k;
    lse_merge(m, sum, s_m[w], s_s[w]);
  }
  argmax[t] = (int32_t)(0xffffffffu - (uint32_t)(k & 0xffffffffu));
  if (max_logit) {
    uint32_t u = (uint32_t)(k >> 32);
    u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
    max_logit[t] = __uint_as_float(u);
  }
  if (lse) lse[t] = m + __logf(sum);
}

}  // namespace
}  // namespace dcut

using namespace dcut;

// Final norm, LM-head GEMM with the argmax (epi EPI_ARGMAX) or sampling
// (EPI_SAMPLE) epilogue, then the per-row merge of the partial keys.
static int lm_head_run(EpiKind epi, int H, int V, int B, int D, const int32_t *cu, const float *x,
                       const dcut_bf16 *final_norm, float eps, const dcut_bf16 *w_lm, const int32_t *row_req,
                       const int32_t *row_pos, float inv_temp, uint64_t seed, int32_t *token, float *max_score,
                       float *logits, float *lse, void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!batch_ok(B, D) || H <= 0 || H % 8 || V <= 0) return DCUT_EINVAL;
  if (!cu || !x || !final_norm || !w_lm || !token || !(eps >= 0.0f)) return DCUT_EINVAL;
  if (!gemm_span_ok(256, H, 256, H)) return DCUT_EUNSUPPORTED;   // any V: W is addressed per column tile
  const size_t need = lmhead_need(H, V, B, D, lse != nullptr);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 255)) return DCUT_EWORKSPACE;
  const int M = B * (D + 1);
  uint16_t *f = (uint16_t *)ws;
  const int slots = 4 * ((V + 255) / 256);   // row stride; holds either of the gemm_argmax_slots() counts
  unsigned long long *keys = (unsigned long long *)((char *)ws + align256((size_t)M * H * 2));
  float2 *part = (float2 *)((char *)keys + align256((size_t)M * slots * sizeof(unsigned long long)));
  const int32_t *Kstar = cu + B;
  DCUT_TRY(rmsnorm_launch(DCUT_KERNEL_NORM, x, nullptr, nullptr, 0, final_norm, eps, H, M, Kstar,
                          nullptr, f, nullptr, 0, 0.0f, nullptr, nullptr, nullptr, nullptr, stream));
  GemmArgs g = {};
  g.A = f; g.lda = H; g.K = H; g.M_max = M; g.m_count = Kstar;
  g.W = w_lm; g.ldw = H; g.N = V;
  g.amax_keys = keys; g.amax_slots = slots; g.logits = logits; g.ld_logits = V;
  g.row_req = row_req; g.row_pos = row_pos; g.inv_temp = inv_temp;
  g.lse_part = lse ? part : nullptr;
  g.seed_lo = (uint32_t)seed; g.seed_hi = (uint32_t)(seed >> 32);
  int used_big, used_mid;
  gemm_argmax_slots(g, epi, &used_big, &used_mid);
  DCUT_TRY(gemm_launch(DCUT_KERNEL_LM_HEAD, epi, g, stream));
  return launch(DCUT_KERNEL_ARGMAX_FINAL, k_argmax_final, dim3(M), dim3(256), 0, stream,
                (const unsigned long long *)keys, (const float2 *)part, used_big, used_mid, slots, Kstar, M,
                token, max_score, lse);
}

extern "C" int dcut_lm_head_argmax(int H, int V, int B, int D, const int32_t *cu, const float *x,
                                   const dcut_bf16 *final_norm, float eps, const dcut_bf16 *w_lm,
                                   int32_t *argmax, float *max_logit, float *logits, void *ws,
                                   size_t ws_bytes, hipStream_t stream) {
  return lm_head_run(EPI_ARGMAX, H, V, B, D, cu, x, final_norm, eps, w_lm, nullptr, nullptr, 0.0f, 0, argmax,
                     max_logit, logits, nullptr, ws, ws_bytes, stream);
}

extern "C" int dcut_lm_head_sample(int H, int V, int B, int D, const int32_t *cu, const int32_t *packed_req,
                                   const int32_t *packed_pos, const float *x, const dcut_bf16 *final_norm,
                                   float eps, const dcut_bf16 *w_lm, float temperature, uint64_t seed,
                                   int32_t *token, float *max_score, float *logits, float *lse, void *ws,
                                   size_t ws_bytes, hipStream_t stream) {
  if (!packed_req || !packed_pos || !(temperature > 0.0f) || !(temperature < __builtin_inff()))
    return DCUT_EINVAL;
  return lm_head_run(EPI_SAMPLE, H, V, B, D, cu, x, final_norm, eps, w_lm, packed_req, packed_pos,
                     1.0f / temperature, seed, token, max_score, logits, lse, ws, ws_bytes, stream);
}

// ---------------------------------------------------------------- allocation-free variant
// The greedy LM head with its scratch in a file-scope device array instead of
// a caller workspace.  Each device the library runs on holds its own copy of
// the array (for the life of the process); host code reaches it only through
// the address hipGetSymbolAddress returns on that device, fetched once per
// device on the first call made with that device current.
namespace {
constexpr size_t LM_STATIC_SCRATCH = (size_t)32 << 20;
constexpr int MAX_DEVICES = 64;
__device__ __align__(256) unsigned char scratch[LM_STATIC_SCRATCH];
std::atomic<void *> scratch_addr[MAX_DEVICES];
std::mutex scratch_mutex;

int scratch_of_current_device(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DCUT_EHIP;
  if (dev < 0 || dev >= MAX_DEVICES) return DCUT_EUNSUPPORTED;
  void *p = scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(scratch_mutex);
    p = scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DCUT_EHIP;
      scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return DCUT_OK;
}
}  // namespace

extern "C" size_t dcut_lm_head_static_scratch_bytes(void) { return LM_STATIC_SCRATCH; }

extern "C" int dcut_lm_head_argmax_static(int H, int V, int B, int D, const int32_t *cu, const float *x,
                                          const dcut_bf16 *final_norm, float eps, const dcut_bf16 *w_lm,
                                          int32_t *argmax, float *max_logit, float *logits, hipStream_t stream) {
  if (!batch_ok(B, D) || H <= 0 || H % 8 || V <= 0) return DCUT_EINVAL;
  if (!cu || !x || !final_norm || !w_lm || !argmax || !(eps >= 0.0f)) return DCUT_EINVAL;
  if (!gemm_span_ok(256, H, 256, H) || lmhead_need(H, V, B, D, false) > LM_STATIC_SCRATCH) return DCUT_EUNSUPPORTED;
  void *ws = nullptr;
  DCUT_TRY(scratch_of_current_device(&ws));
  return lm_head_run(EPI_ARGMAX, H, V, B, D, cu, x, final_norm, eps, w_lm, nullptr, nullptr, 0.0f, 0, argmax,
                     max_logit, logits, nullptr, ws, LM_STATIC_SCRATCH, stream);
}
