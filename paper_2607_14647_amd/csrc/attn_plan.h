// Attention work items and their longest-first order (device side).
//
// Work item = (request i, kv head g, chunk c) of the split-KV attention.  Chunk
// c covers cache keys [c*CH, min((c+1)*CH, L_i)); the last chunk also covers
// the block keys.  An item's work is its key count: a full chunk has CH keys,
// a request's last chunk L - (nc-1)*CH + d.
//
// Workgroups are dispatched in blockIdx order as slots free up, so ordering
// the live items by work length, longest first, makes the hardware dispatcher
// run a longest-processing-time-first schedule: the short ragged last chunks
// fill the gaps at the end instead of a long item starting last.  The order is
//   1. last chunks longer than CH, by length descending (ties: request index),
//   2. all full chunks, request by request, chunk then kv head,
//   3. the remaining last chunks, by length descending (ties: request index),
// kv head fastest within a request's last chunk.  Requests with no kept rows
// have no items.  One workgroup (attn_plan_block) ranks the requests and
// writes the item list and its length; attention workgroup b takes item b,
// and those past the end exit at once.  The results do not depend on the
// order: every item writes its own partial, merged in chunk order.
//
// Plan layout: int32 count at offset 0, items from byte PLAN_HEAD on, 8 int32
// each: {request, kv head, chunk, first packed row, kept rows, usable context,
// cap, 0}.
#pragma once
#include "dcut_internal.h"

namespace dcut {

constexpr int PLAN_MAX_B = 1024;      // sort keys hold 10 bits of request index
constexpr int PLAN_HEAD = 256;
constexpr int PLAN_MIN_ITEMS = 512;   // a grid this small runs in one round of slots

// Cached length used for request i (clamped so bad device data stays in bounds)
// and its number of chunks (at least one: the block keys).
__device__ __forceinline__ int usable_ctx(int L, int cap, int D) {
  int hi = cap - D - 1;
  if (L > hi) L = hi;
  return L < 0 ? 0 : L;
}
__device__ __forceinline__ int n_chunks(int L, int chunk, int MC) {
  int nc = L > 0 ? (L + chunk - 1) / chunk : 1;
  return nc > MC ? MC : nc;
}

// LDS of attn_plan_block for B requests and NT threads.
inline size_t attn_plan_lds_bytes(int B, int NT) {
  return (size_t)(((B + 3) & ~3) + 3 * (NT / 64)) * sizeof(int);
}

// The plan, built by one workgroup of NT threads (B <= PLAN_MAX_B); thread t
// owns requests t*R .. t*R+R-1, R = ceil(B / NT), and writes their items at
// the places the order gives them: its full chunks after the full chunks of
// the requests before it (a scan), its last chunk at its rank among the last
// chunks (a count of larger keys).  Also reports capacity faults of requests
// with kept rows.  `s` is attn_plan_lds_bytes(B, NT) of LDS.
template <int NT>
__device__ __forceinline__ void attn_plan_block(const AttnArgs &a, int *s) {
  constexpr int NW = NT / 64, RMAX = PLAN_MAX_B / NT;
  const int B = a.B, CH = a.chunk, MC = a.max_chunks, nkv = a.n_kv;
  const int B4 = (B + 3) & ~3;
  const int R = (B + NT - 1) / NT;
  int *s_ck = s, *s_w = s_ck + B4;
  const int t = threadIdx.x, w = t >> 6, ln = t & 63;
  int ck[RMAX], full[RMAX], t0s[RMAX], ds[RMAX], Ls[RMAX], caps[RMAX], lasts[RMAX];
  int sum = 0, nl = 0, nv = 0;
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    const int j = t * R + r;
    int key = -1;
    full[r] = t0s[r] = ds[r] = Ls[r] = caps[r] = lasts[r] = 0;
    if (r < R && j < B) {
      const int t0 = a.cu[j];
      const int d = a.cu[j + 1] - t0;
      const int L0 = a.ctx_len[j];
      const int cap = a.kv_cap[j];
      if (d > 0 && (L0 < 0 || L0 + a.D + 1 > cap) && a.dev_err) atomicOr(a.dev_err, DCUT_DERR_CAPACITY);
      const int L = usable_ctx(L0, cap, a.D);
      const int nc = n_chunks(L, CH, MC);
      if (d > 0) {
        key = min(L + d - (nc - 1) * CH, 1 << 20);   // only a cap beyond max_ctx makes it larger
        full[r] = nc - 1;
      }
      t0s[r] = t0; ds[r] = d; Ls[r] = L; caps[r] = cap; lasts[r] = nc - 1;
    }
    // sort key: length descending, then request index ascending (key <= 2^20,
    // B <= 1024), so a request's rank is the number of larger keys
    ck[r] = key > 0 ? (key << 10) | (1023 - j) : -1;
    if (r < R && j < B4) s_ck[j] = ck[r];
    sum += full[r];
    nl += key > CH;
    nv += key > 0;
  }
  int x = sum;                                    // inclusive scan within the wave
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (ln >= o) x += y;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    nl += __shfl_xor(nl, o);
    nv += __shfl_xor(nv, o);
  }
  if (ln == 63) s_w[w] = x;
  if (ln == 0) {
    s_w[NW + w] = nl;
    s_w[2 * NW + w] = nv;
  }
  __syncthreads();
  int before = 0, n_full = 0, n_long = 0, n_live = 0;
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    const int sv = s_w[v];
    before += v < w ? sv : 0;
    n_full += sv;
    n_long += s_w[NW + v];
    n_live += s_w[2 * NW + v];
  }
  const int e1 = n_long * nkv, e2 = e1 + n_full * nkv, e3 = e2 + (n_live - n_long) * nkv;
  int32_t *plan = a.plan;
  if (t == 0) plan[0] = e3;
  int4 *items = (int4 *)((char *)plan + PLAN_HEAD);
  int run = before + x - sum;                     // full chunks of the requests before mine
  const int4 *k4 = (const int4 *)s_ck;
#pragma unroll
  for (int r = 0; r < RMAX; ++r) {
    const int j = t * R + r;
    if (r >= R || j >= B) continue;
    const int pre = e1 + run * nkv;               // this request's first full-chunk item
    run += full[r];
    if (ck[r] < 0) continue;                      // no kept rows: no items
    int rank = 0;
#pragma unroll 4
    for (int k = 0; k < (B4 >> 2); ++k) {
      const int4 v = k4[k];
      rank += (v.x > ck[r]) + (v.y > ck[r]) + (v.z > ck[r]) + (v.w > ck[r]);
    }
    const int4 tail = make_int4(ds[r], Ls[r], caps[r], 0);
    for (int c = 0; c < full[r]; ++c)
      for (int g = 0; g < nkv; ++g) {
        const int p = pre + c * nkv + g;
        items[2 * p] = make_int4(j, g, c, t0s[r]);
        items[2 * p + 1] = tail;
      }
    // last chunks: the n_long longer than a chunk first, the others after the full chunks
    const int base = rank < n_long ? rank * nkv : e2 + (rank - n_long) * nkv;
    for (int g = 0; g < nkv; ++g) {
      items[2 * (base + g)] = make_int4(j, g, lasts[r], t0s[r]);
      items[2 * (base + g) + 1] = tail;
    }
  }
}

}  // namespace dcut
