// Cross-request selection (scores, ranking, budget choice, keep depths) and packing.
//
// Sec. 3.2 Eq. dcut-prefix-score, Sec. 3.3 Eq. dcut-objective, Alg. 1 and the
// packing of App. C; for rejection-sampling verification (App. B) the same
// kernel ranks the shifted scores of Eq. dcut-shifted-score and chooses the
// budget causally: by the early-stopping scan, or as a budget fixed beforehand.
// One 1024-thread workgroup does it all, packing included: the whole problem is
// at most 8192 positions (64 KB of sort keys in LDS), so a single workgroup
// avoids any grid-wide synchronisation and launch round trips.
//
// Bit-exactness: each request's scores are one sequential float32 product per
// depth (denormals kept, no contraction); ranking uses the unique 64-bit key
// (score bits, 63 - depth, 65535 - request), so any correct sort gives the same
// order; benefits are integer sums of trunc(s * 2^40); the budget objective is
// one float64 division.  The outputs are therefore identical on any hardware.
#include "dcut_internal.h"
#include "scan.h"

namespace dcut {

enum SelectMode { SEL_BUCKETS = 0, SEL_SCAN = 1, SEL_FIXED = 2, SEL_HISTORY = 3 };

struct SelectParams {
  int B, D, R;
  int shift;      // 1: rank the shifted scores s~_{i,k} = s_{i,k-1} (s~_{i,1} = 1)
  int mode;       // SelectMode
  int budgets[DCUT_MAX_CANDIDATES];
  double costs[DCUT_MAX_CANDIDATES];
};

__device__ __forceinline__ unsigned long long rank_key(float s, int k, int i) {
  return ((unsigned long long)__float_as_uint(s) << 32) |
         ((unsigned long long)(63 - k) << 16) | (unsigned long long)(65535 - i);
}

// trunc(s * 2^40) for the score held in a key's upper half
__device__ __forceinline__ unsigned long long key_units(unsigned long long key) {
  float s = __uint_as_float((uint32_t)(key >> 32));
  return (unsigned long long)((double)s * 1099511627776.0);
}

__device__ __forceinline__ bool conf_bad(float c) { return !(c >= 0.0f && c <= 1.0f) || signbit(c); }

#pragma clang fp contract(off)
// Step cost at an arbitrary verification size K for the causal scan: linear
// between consecutive budgets (K_r, C_r), the end costs outside them, and the
// last of several equal budgets at that K.  Same float64 operations, in the
// same order, on every platform.  The candidates sit in LDS (bud, cst); r is
// found by binary search over the non-decreasing budgets.
__device__ double cost_at(const int *bud, const double *cst, int R, int K) {
  int lo = 0, hi = R;                 // r = (number of budgets <= K) - 1
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (bud[mid] <= K) lo = mid + 1;
    else hi = mid;
  }
  const int r = lo - 1;
  if (r < 0) return cst[0];
  if (r == R - 1) return cst[R - 1];
  const int ka = bud[r], kb = bud[r + 1];
  const double ca = cst[r], cb = cst[r + 1];
  return ca + ((cb - ca) * (double)(K - ka)) / (double)(kb - ka);
}

// objective of Eq. dcut-objective for the exact fixed-point benefit P
__device__ __forceinline__ double objective(unsigned long long P, double cost) {
  return ((double)P * 0x1p-40) / cost;
}

__global__ void __launch_bounds__(1024)
k_select(SelectParams p, const float *__restrict__ conf, const int32_t *__restrict__ draft,
         const int32_t *__restrict__ ctx_len, int32_t *__restrict__ keep_len, int32_t *__restrict__ cu,
         int32_t *__restrict__ ptok, int32_t *__restrict__ ppos, int32_t *__restrict__ preq,
         int32_t *__restrict__ choice, unsigned long long *__restrict__ benefit,
         int32_t *__restrict__ dev_err, int32_t *__restrict__ k_state) {
  extern __shared__ unsigned long long smem[];
  __shared__ unsigned long long s_wave[17];
  __shared__ unsigned long long s_ben[DCUT_MAX_CANDIDATES];
  __shared__ double s_cost[DCUT_MAX_CANDIDATES], s_obj[DCUT_MAX_CANDIDATES];
  __shared__ int s_bud[DCUT_MAX_CANDIDATES];
  __shared__ unsigned long long s_tau;
  __shared__ int s_err, s_stop;

  const int tid = threadIdx.x;
  const int D = p.D, D1 = p.D + 1, B = p.B;
  const int N = B * D1;
  int NP = 64;
  while (NP < N) NP <<= 1;
  unsigned long long *keys = smem;          // [NP]
  int *s_kl = (int *)smem;                  // [B], then s_cu [B+1]: the key area (and the prefix
                                            // sums after it) once both are dead
  int *s_cu = s_kl + B;
  float *s_conf = (float *)(smem + NP + blockDim.x);   // [B * D], staged once (coalesced)
  if (tid == 0) {
    s_err = 0;
    s_stop = N;
  }
  for (int j = tid; j < B * D; j += blockDim.x) s_conf[j] = conf[j];
  if (tid < p.R) {
    s_bud[tid] = p.budgets[tid];
    s_cost[tid] = p.costs[tid];
  }
  __syncthreads();

  // 1. scores and keys, one thread per request, sequential in depth
  for (int i = tid; i < B; i += blockDim.x) {
    float s = 1.0f;
    keys[i * D1] = rank_key(s, 0, i);
    for (int k = 1; k <= D; ++k) {
      float c = s_conf[i * D + (k - 1)];
      if (conf_bad(c)) {
        s_err = 1;
        c = 0.0f;
      }
      const float prev = s;          // the shifted score of depth k: the product up to k - 1
      s = s * c;
      keys[i * D1 + k] = rank_key(p.shift ? prev : s, k, i);
    }
  }
  for (int j = N + tid; j < NP; j += blockDim.x) keys[j] = 0ull;   // sorts last

  // 2. sort, descending.  Each wave sorts 64-key runs in registers (a bitonic
  // network over cross-lane shuffles, no barrier); then runs are merged
  // pairwise: a key's place in the merged run is its index in its own run plus
  // the number of keys ahead of it in the other run (a binary search; equal
  // keys, which only the zero padding has, go left run first).
  __syncthreads();
  {
    const int lane = tid & 63, wv = tid >> 6, nwv = blockDim.x >> 6;
    for (int run = wv; run < NP / 64; run += nwv) {
      unsigned long long x = keys[run * 64 + lane];
#pragma unroll
      for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
          const unsigned long long y = __shfl_xor(x, stride, 64);
          // the lower lane of a pair keeps the larger key in a descending run
          const bool take_max = ((lane & stride) == 0) == ((lane & size) == 0);
          x = take_max ? (x > y ? x : y) : (x < y ? x : y);
        }
      keys[run * 64 + lane] = x;
    }
    const int EM = NP > (int)blockDim.x ? NP / (int)blockDim.x : 1;   // keys per thread, <= 8
    for (int width = 64; width < NP; width <<= 1) {
      __syncthreads();
      unsigned long long mine[8];
      int dest[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (e >= EM) break;
        const int idx = tid + e * (int)blockDim.x;
        dest[e] = -1;
        if (idx >= NP) continue;
        const unsigned long long x = keys[idx];
        const int base = idx & ~(2 * width - 1);
        const bool left = idx - base < width;
        const int own = idx - base - (left ? 0 : width);
        const unsigned long long *other = keys + base + (left ? width : 0);
        int lo = 0, hi = width;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          const unsigned long long o = other[mid];
          if (left ? (o > x) : (o >= x)) lo = mid + 1;
          else hi = mid;
        }
        mine[e] = x;
        dest[e] = base + own + lo;
      }
      __syncthreads();
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (e >= EM) break;
        if (dest[e] >= 0) keys[dest[e]] = mine[e];
      }
    }
  }
  __syncthreads();

  // 3. exact prefix sums of the fixed-point scores in rank order
  const int E = NP > (int)blockDim.x ? NP / (int)blockDim.x : 1;   // ranks per thread
  unsigned long long local = 0;
  for (int m = tid * E; m < tid * E + E; ++m)
    if (m < N) local += key_units(keys[m]);
  unsigned long long total;
  unsigned long long pre = block_exclusive_scan(local, s_wave, &total);
  unsigned long long *s_pre = smem + NP;    // [blockDim.x]
  s_pre[tid] = pre;
  __syncthreads();
  if (tid < p.R) {
    int K = p.budgets[tid];
    int t = K / E, rem = K - t * E;
    unsigned long long P = (t < (int)blockDim.x) ? s_pre[t] : total;
    for (int m = t * E; m < t * E + rem; ++m) P += key_units(keys[m]);
    s_ben[tid] = P;
    s_obj[tid] = objective(P, s_cost[tid]);   // every candidate's objective at once
    if (benefit) benefit[tid] = P;
  }
  __syncthreads();

  // 4a. causal scan (App. B): the positions enter in rank order from K = B on,
  // and the scan stops at the first K whose next position does not strictly
  // raise the objective.  Every thread tests the sizes of its own ranks.
  if (p.mode == SEL_SCAN) {
    unsigned long long P = s_pre[tid];          // benefit of the first tid * E ranks
    int stop = N;
    for (int m = tid * E; m < tid * E + E && m < N; ++m) {
      const unsigned long long P1 = P + key_units(keys[m]);
      if (m >= B && !(objective(P1, cost_at(s_bud, s_cost, p.R, m + 1)) >
                      objective(P, cost_at(s_bud, s_cost, p.R, m)))) {
        stop = m;
        break;
      }
      P = P1;
    }
    if (stop < N) atomicMin(&s_stop, stop);
  }
  __syncthreads();

  // 4b. budget choice: the first strict maximum of benefit * 2^-40 / cost over
  // the candidates, the fixed budget, the scan's stop, or the budget carried
  // over from the previous block (which then carries this block's choice on)
  if (tid == 0) {
    int best = 0, Kstar;
    int bucket = 0;                   // first strict maximum of the objective over the candidates
    double best_obj = -1.0;
    for (int r = 0; r < p.R; ++r) {
      const double obj = s_obj[r];
      if (obj > best_obj) {
        best_obj = obj;
        bucket = r;
      }
    }
    if (p.mode == SEL_BUCKETS) {
      best = bucket;
      Kstar = p.budgets[best];
    } else if (p.mode == SEL_FIXED) {
      Kstar = p.budgets[0];
    } else {
      if (p.mode == SEL_SCAN) {
        Kstar = s_stop;
      } else {
        const int k = k_state[0];
        Kstar = k < B ? B : (k > N ? N : k);
        k_state[0] = p.budgets[bucket];
      }
      best = -1;                      // the last candidate budget not above K*
      for (int r = 0; r < p.R; ++r)
        if (p.budgets[r] <= Kstar) best = r;
    }
    choice[0] = Kstar;
    choice[1] = best;
    s_tau = keys[Kstar - 1];          // the K*-th largest key
    if (s_err && dev_err) atomicOr(dev_err, DCUT_DERR_CONF);
  }
  __syncthreads();

  // 5. keep depths: a request keeps the depths whose key ranks within the top K*
  const unsigned long long tau = s_tau;
  for (int i = tid; i < B; i += blockDim.x) {
    float s = 1.0f;
    int n = 1;                        // the bonus key (s = 1, k = 0) always ranks first in its request
    for (int k = 1; k <= D; ++k) {
      float c = s_conf[i * D + (k - 1)];
      if (conf_bad(c)) c = 0.0f;
      const float prev = s;
      s = s * c;
      if (rank_key(p.shift ? prev : s, k, i) >= tau) n = k + 1;
      else break;
    }
    if (rank_key(1.0f, 0, i) < tau) n = 0;   // impossible when K* >= B; kept for safety
    keep_len[i] = n;
    s_kl[i] = n;
  }
  __syncthreads();

  // 6. packing (App. C): cu = exclusive scan of keep_len; row t = cu[i] + k
  // gets (z_{i,k}, L_i + k, i).  The sort keys are dead by now; their LDS holds
  // the offsets.
  const int per = (B + blockDim.x - 1) / blockDim.x;   // <= 4
  int v[4];
  int loc = 0;
  for (int j = 0; j < per; ++j) {
    const int i = tid * per + j;
    v[j] = i < B ? s_kl[i] : 0;
    loc += v[j];
  }
  int kept;
  int off = block_exclusive_scan(loc, (int *)s_wave, &kept);
  for (int j = 0; j < per; ++j) {
    const int i = tid * per + j;
    if (i < B) s_cu[i] = off;
    off += v[j];
  }
  if (tid == 0) s_cu[B] = kept;
  __syncthreads();
  for (int i = tid; i <= B; i += blockDim.x) cu[i] = s_cu[i];
  for (int idx = tid; idx < N; idx += blockDim.x) {
    const int i = idx / D1, k = idx - i * D1;
    if (k < s_cu[i + 1] - s_cu[i]) {
      const int t = s_cu[i] + k;
      ptok[t] = draft[idx];
      ppos[t] = ctx_len[i] + k;
      preq[t] = i;
    }
  }
}
#pragma clang fp contract(on)

}  // namespace dcut

using namespace dcut;

static int select_run(int B, int D, const float *conf, const int32_t *draft, const int32_t *ctx_len,
                      int shift, int mode, int R, const int32_t *budgets, const double *costs, int32_t *k_state,
                      int32_t *keep_len, int32_t *cu, int32_t *packed_tok, int32_t *packed_pos,
                      int32_t *packed_req, int32_t *choice, uint64_t *benefit, int32_t *dev_err,
                      hipStream_t stream) {
  if (!batch_ok(B, D)) return DCUT_EINVAL;
  if (R < 1 || R > DCUT_MAX_CANDIDATES || !budgets || !costs) return DCUT_EINVAL;
  if (mode == SEL_FIXED && R != 1) return DCUT_EINVAL;
  if (mode == SEL_HISTORY && !k_state) return DCUT_EINVAL;
  if (!conf && D > 0) return DCUT_EINVAL;
  if (!draft || !ctx_len || !keep_len || !cu || !packed_tok || !packed_pos || !packed_req || !choice)
    return DCUT_EINVAL;
  SelectParams p;
  p.B = B;
  p.D = D;
  p.R = R;
  p.shift = shift;
  p.mode = mode;
  for (int r = 0; r < R; ++r) {
    int K = budgets[r];
    double c = costs[r];
    if (K < B || K > B * (D + 1)) return DCUT_EINVAL;
    if (r > 0 && K < budgets[r - 1]) return DCUT_EINVAL;
    if (!(c > 0.0) || !(c < __builtin_inf())) return DCUT_EINVAL;
    p.budgets[r] = K;
    p.costs[r] = c;
  }
  int N = B * (D + 1), NP = 64;
  while (NP < N) NP <<= 1;
  size_t shmem = (size_t)(NP + 1024) * sizeof(unsigned long long) + (size_t)B * D * sizeof(float);
  return launch(DCUT_KERNEL_SELECT, k_select, dim3(1), dim3(1024), shmem, stream, p, conf, draft, ctx_len,
                keep_len, cu, packed_tok, packed_pos, packed_req, choice, (unsigned long long *)benefit, dev_err,
                k_state);
}

extern "C" int dcut_select(int B, int D, const float *conf, const int32_t *draft,
                           const int32_t *ctx_len, int R, const int32_t *budgets,
                           const double *costs, int32_t *keep_len, int32_t *cu,
                           int32_t *packed_tok, int32_t *packed_pos, int32_t *packed_req,
                           int32_t *choice, uint64_t *benefit, int32_t *dev_err,
                           hipStream_t stream) {
  return select_run(B, D, conf, draft, ctx_len, 0, SEL_BUCKETS, R, budgets, costs, nullptr, keep_len, cu,
                    packed_tok, packed_pos, packed_req, choice, benefit, dev_err, stream);
}

extern "C" int dcut_select_rs(int B, int D, const float *conf, const int32_t *draft,
                              const int32_t *ctx_len, int mode, int R, const int32_t *budgets,
                              const double *costs, int32_t *k_state, int32_t *keep_len, int32_t *cu,
                              int32_t *packed_tok, int32_t *packed_pos, int32_t *packed_req,
                              int32_t *choice, uint64_t *benefit, int32_t *dev_err,
                              hipStream_t stream) {
  int m;
  if (mode == DCUT_RS_SCAN) m = SEL_SCAN;
  else if (mode == DCUT_RS_FIXED) m = SEL_FIXED;
  else if (mode == DCUT_RS_HISTORY) m = SEL_HISTORY;
  else return DCUT_EINVAL;
  return select_run(B, D, conf, draft, ctx_len, 1, m, R, budgets, costs, k_state, keep_len, cu, packed_tok,
                    packed_pos, packed_req, choice, benefit, dev_err, stream);
}
