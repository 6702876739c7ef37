// Greedy target-only acceptance (Sec. 3.2: sequential acceptance; App. A) and
// rejection-sampling acceptance (App. B).
//
// Greedy: one workgroup.  Every (request, depth) pair is compared at once; the
// first mismatch of each request (an LDS minimum) gives its accepted length.
#include "dcut_internal.h"
#include "rng.h"
#include "scan.h"

namespace dcut {

__global__ void __launch_bounds__(1024)
k_accept(int B, int D, const int32_t *__restrict__ draft, const int32_t *__restrict__ keep_len,
         const int32_t *__restrict__ cu, const int32_t *__restrict__ argmax,
         int32_t *__restrict__ accept_len, int32_t *__restrict__ next_tok,
         int32_t *__restrict__ total, int32_t *__restrict__ ctx_len_inout) {
  __shared__ int s_wave[17];
  __shared__ int s_n[DCUT_MAX_BATCH], s_base[DCUT_MAX_BATCH], s_first[DCUT_MAX_BATCH];
  const int D1 = D + 1;
  const int rows = B * D1;
  for (int i = threadIdx.x; i < B; i += blockDim.x) {
    int n = keep_len[i] - 1;
    n = n < 0 ? 0 : (n > D ? D : n);
    int base = cu[i];
    base = base < 0 ? 0 : (base > rows - 1 - n ? rows - 1 - n : base);   // stay in bounds
    s_n[i] = n;
    s_base[i] = base;
    s_first[i] = n;                     // no mismatch among the n checked drafts
  }
  __syncthreads();
  // draft j+1 of request i is checked against the greedy token of row base + j
  for (int idx = threadIdx.x; idx < B * D; idx += blockDim.x) {
    const int i = idx / D, j = idx - i * D;
    if (j < s_n[i] && draft[(size_t)i * D1 + j + 1] != argmax[s_base[i] + j]) atomicMin(&s_first[i], j);
  }
  __syncthreads();
  int local = 0;
  for (int i = threadIdx.x; i < B; i += blockDim.x) {
    const int a = s_first[i];
    const int base = s_base[i];
    accept_len[i] = a;
    next_tok[i] = argmax[base + a];
    local += a + 1;
    if (ctx_len_inout) ctx_len_inout[i] += a + 1;
  }
  int sum;
  block_exclusive_scan(local, s_wave, &sum);
  if (threadIdx.x == 0) total[0] = sum;
}

}  // namespace dcut

using namespace dcut;

extern "C" int dcut_accept(int B, int D, const int32_t *draft, const int32_t *keep_len,
                           const int32_t *cu, const int32_t *argmax, int32_t *accept_len,
                           int32_t *next_tok, int32_t *total, int32_t *ctx_len_inout,
                           hipStream_t stream) {
  if (!batch_ok(B, D)) return DCUT_EINVAL;
  if (!draft || !keep_len || !cu || !argmax || !accept_len || !next_tok || !total) return DCUT_EINVAL;
  return launch(DCUT_KERNEL_ACCEPT, k_accept, dim3(1), dim3(1024), 0, stream, B, D, draft, keep_len,
                cu, argmax, accept_len, next_tok, total, ctx_len_inout);
}

// ---------------------------------------------------------------------------
// Rejection-sampling acceptance (App. B, distributional correctness).
//
// Draft z_{i,j} is verified at row r = cu_i + j - 1 against the target
// distribution p_r = softmax(logits_r / T): it is accepted when
// u_r q_{i,j}(z) < p_r(z) (probability min(1, p/q)), u_r a Philox4x32-10
// uniform of the row.  At the first rejection the committed token is drawn
// from (p_r - q_{i,j})_+ by the Gumbel-max rule with the row's own noise; when
// every kept draft is accepted it is the target's sample at the last kept row.
// Three launches: the decisions (one workgroup, every kept draft tested at
// once), the residual draws over the vocabulary (one workgroup per request and
// column chunk), and the merge.
namespace dcut {

constexpr int RS_CHUNK = 2048;     // vocabulary columns per residual workgroup

size_t accept_rs_ws_bytes(int V, int B) {
  const size_t nch = ((size_t)V + RS_CHUNK - 1) / RS_CHUNK;
  return align256((size_t)B * 2 * sizeof(int32_t)) + align256((size_t)B * nch * sizeof(unsigned long long));
}

namespace {

__device__ __forceinline__ void block_bounds(int i, int B, int D, const int32_t *keep_len, const int32_t *cu,
                                             int &n, int &base) {
  const int rows = B * (D + 1);
  n = keep_len[i] - 1;
  n = n < 0 ? 0 : (n > D ? D : n);
  base = cu[i];
  base = base < 0 ? 0 : (base > rows - 1 - n ? rows - 1 - n : base);   // stay in bounds
}

// Every (request, depth) test at once; the first failing depth of each request
// (an LDS minimum) is where its verification stops.
__global__ void __launch_bounds__(1024)
k_rs_decide(int B, int D, int V, float inv_temp, uint32_t seed_lo, uint32_t seed_hi,
            const int32_t *__restrict__ draft, const float *__restrict__ q,
            const int32_t *__restrict__ keep_len, const int32_t *__restrict__ cu,
            const int32_t *__restrict__ packed_pos, const float *__restrict__ logits,
            const float *__restrict__ lse, int32_t *__restrict__ rej_row, int32_t *__restrict__ acc,
            int32_t *__restrict__ dev_err) {
  __shared__ int s_n[DCUT_MAX_BATCH], s_base[DCUT_MAX_BATCH], s_first[DCUT_MAX_BATCH];
  __shared__ int s_err;
  if (threadIdx.x == 0) s_err = 0;
  for (int i = threadIdx.x; i < B; i += blockDim.x) {
    int n, base;
    block_bounds(i, B, D, keep_len, cu, n, base);
    s_n[i] = n;
    s_base[i] = base;
    s_first[i] = n;                    // no failure among the n kept drafts
  }
  __syncthreads();
  // draft j = d + 1 of request i is tested at row base + d
  for (int idx = threadIdx.x; idx < B * D; idx += blockDim.x) {
    const int i = idx / D, d = idx - i * D;
    if (d >= s_n[i]) continue;
    const int r = s_base[i] + d;
    const int z = draft[(size_t)i * (D + 1) + d + 1];
    bool pass = false;
    if (z < 0 || z >= V) {               // an invalid draft is never accepted
      s_err = 1;
    } else {
      const double p = exp((double)(logits[(size_t)r * V + z] * inv_temp) - (double)lse[r]);
      const double qz = (double)q[((size_t)i * D + d) * V + z];
      const uint4 w = philox4x32_10(make_uint4(0u, (uint32_t)packed_pos[r], (uint32_t)i, 1u), seed_lo, seed_hi);
      pass = uniform01(w.x) * qz < p;
    }
    if (!pass) atomicMin(&s_first[i], d);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < B; i += blockDim.x) {
    const int a = s_first[i];
    rej_row[i] = a < s_n[i] ? s_base[i] + a : -1;
    acc[i] = a;
  }
  if (threadIdx.x == 0 && s_err && dev_err) atomicOr(dev_err, DCUT_DERR_TOKEN);
}

// Residual draw of a rejecting row over one chunk of the vocabulary: the
// largest key of ln((p_c - q_c)_+) + G_c (lowest column on ties); 0 if no
// column of the chunk has p_c > q_c.  Each thread takes one Philox call per
// 128-column block, which covers its four columns c, c + 32, c + 64, c + 96.
__global__ void __launch_bounds__(256)
k_rs_residual(int D, int V, int nch, float inv_temp, uint32_t seed_lo, uint32_t seed_hi,
              const float *__restrict__ q, const int32_t *__restrict__ packed_pos,
              const float *__restrict__ logits, const float *__restrict__ lse,
              const int32_t *__restrict__ rej_row, const int32_t *__restrict__ acc,
              unsigned long long *__restrict__ keys) {
  __shared__ unsigned long long s_key[4];
  const int i = blockIdx.y;
  const int r = rej_row[i];
  if (r < 0) return;                      // the whole workgroup leaves together
  const int a = acc[i];
  const float *lr = logits + (size_t)r * V;
  const float *qr = q + ((size_t)i * D + a) * V;
  const float lz = lse[r];
  const uint32_t pos = (uint32_t)packed_pos[r];
  const int c0 = blockIdx.x * RS_CHUNK;
  unsigned long long best = 0ull;
  for (int t = threadIdx.x; t < RS_CHUNK / 4; t += blockDim.x) {
    const int blk = t >> 5, l = t & 31;
    const int cb = c0 + blk * 128 + l;    // column of word 0
    if (cb >= V) break;                   // t only grows, and so does cb
    const uint4 w = philox4x32_10(make_uint4((uint32_t)(32 * (cb >> 7) + l), pos, (uint32_t)i, 0u), seed_lo, seed_hi);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = cb + 32 * k;
      if (c < V) {
        const float d = __expf(lr[c] * inv_temp - lz) - qr[c];
        if (d > 0.0f) {
          const uint32_t wk = k == 0 ? w.x : k == 1 ? w.y : k == 2 ? w.z : w.w;
          const unsigned long long key = ((unsigned long long)orderable(__logf(d) + gumbel_of(wk)) << 32) |
                                         (0xffffffffu - (uint32_t)c);
          best = key > best ? key : best;
        }
      }
    }
  }
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned long long o = __shfl_xor(best, off, 64);
    best = o > best ? o : best;
  }
  if ((threadIdx.x & 63) == 0) s_key[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) best = s_key[w] > best ? s_key[w] : best;
    keys[(size_t)i * nch + blockIdx.x] = best;
  }
}

// Committed token, accepted length and totals: one wave per request merges
// the residual keys of its chunks.
__global__ void __launch_bounds__(1024)
k_rs_finish(int B, int D, int nch, const int32_t *__restrict__ keep_len, const int32_t *__restrict__ cu,
            const int32_t *__restrict__ token, const int32_t *__restrict__ rej_row,
            const int32_t *__restrict__ acc, const unsigned long long *__restrict__ keys,
            int32_t *__restrict__ accept_len, int32_t *__restrict__ next_tok, int32_t *__restrict__ total,
            int32_t *__restrict__ ctx_len_inout) {
  __shared__ int s_wave[17];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int local = 0;
  for (int i = wv; i < B; i += nw) {
    const int a = acc[i], r = rej_row[i];
    unsigned long long k = 0ull;
    if (r >= 0)
      for (int c = lane; c < nch; c += 64) {
        const unsigned long long v = keys[(size_t)i * nch + c];
        k = v > k ? v : k;
      }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const unsigned long long o = __shfl_xor(k, off, 64);
      k = o > k ? o : k;
    }
    if (lane == 0) {
      int n, base;
      block_bounds(i, B, D, keep_len, cu, n, base);
      int t;
      if (r >= 0) t = k ? (int32_t)(0xffffffffu - (uint32_t)(k & 0xffffffffu)) : token[r];   // empty residual: p
      else t = token[base + a];
      accept_len[i] = a;
      next_tok[i] = t;
      local += a + 1;
      if (ctx_len_inout) ctx_len_inout[i] += a + 1;
    }
  }
  int sum;
  block_exclusive_scan(local, s_wave, &sum);
  if (threadIdx.x == 0) total[0] = sum;
}

}  // namespace
}  // namespace dcut

extern "C" int dcut_accept_rs(int B, int D, int V, float temperature, uint64_t seed, const int32_t *draft,
                              const float *q, const int32_t *keep_len, const int32_t *cu,
                              const int32_t *packed_pos, const float *logits, const float *lse,
                              const int32_t *token, int32_t *accept_len, int32_t *next_tok, int32_t *total,
                              int32_t *ctx_len_inout, void *ws, size_t ws_bytes, int32_t *dev_err,
                              hipStream_t stream) {
  if (!batch_ok(B, D) || V <= 0) return DCUT_EINVAL;
  if (!(temperature > 0.0f) || !(temperature < __builtin_inff())) return DCUT_EINVAL;
  if (!draft || (!q && D > 0) || !keep_len || !cu || !packed_pos || !logits || !lse || !token || !accept_len ||
      !next_tok || !total)
    return DCUT_EINVAL;
  if (!ws || ws_bytes < accept_rs_ws_bytes(V, B) || ((uintptr_t)ws & 255)) return DCUT_EWORKSPACE;
  const int nch = (V + RS_CHUNK - 1) / RS_CHUNK;
  int32_t *rej_row = (int32_t *)ws;
  int32_t *acc = rej_row + B;
  unsigned long long *keys = (unsigned long long *)((char *)ws + align256((size_t)B * 2 * sizeof(int32_t)));
  const float inv_temp = 1.0f / temperature;
  const uint32_t lo = (uint32_t)seed, hi = (uint32_t)(seed >> 32);
  DCUT_TRY(launch(DCUT_KERNEL_RS_DECIDE, k_rs_decide, dim3(1), dim3(1024), 0, stream, B, D, V,
                  inv_temp, lo, hi, draft, q, keep_len, cu, packed_pos, logits, lse, rej_row, acc, dev_err));
  if (D > 0)
    DCUT_TRY(launch(DCUT_KERNEL_RS_RESIDUAL, k_rs_residual, dim3(nch, B), dim3(256), 0, stream, D, V, nch,
                    inv_temp, lo, hi, q, packed_pos, logits, lse, (const int32_t *)rej_row,
                    (const int32_t *)acc, keys));
  return launch(DCUT_KERNEL_RS_FINISH, k_rs_finish, dim3(1), dim3(1024), 0, stream, B, D, nch, keep_len, cu,
                token, (const int32_t *)rej_row, (const int32_t *)acc, (const unsigned long long *)keys,
                accept_len, next_tok, total, ctx_len_inout);
}
