// Greedy target-only acceptance (Sec. 3.2: sequential acceptance; App. A).
//
// One workgroup.  Every (request, depth) pair is compared at once; the first
// mismatch of each request (an LDS minimum) gives its accepted length.
#include "dcut_internal.h"
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
