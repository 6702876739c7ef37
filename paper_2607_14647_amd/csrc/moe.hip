// Routed MoE MLP over the packed rows: router, top-k, expert grouping, grouped
// SwiGLU expert GEMMs and a fixed-order weighted combine.
//
// out[t] += sum_{s < top_k} w[t][s] * down_e(SiLU(gate_e(h_t)) * up_e(h_t)),
// e = the s-th routed expert of row t; routing is softmax over the router
// logits, the top_k largest (ties to the lower expert id), weights
// renormalised over the chosen experts.
//
// Determinism and causality: a row's routing, its expert GEMM rows and its
// combine depend only on that row.  Grouping orders the assignments by
// (expert, row * top_k + slot), so each expert's rows appear in row order,
// and the combine adds the top_k expert outputs of a row in slot order.
#include "dcut_internal.h"
#include "scan.h"

namespace dcut {

namespace {

constexpr int TILE_M = 128;    // row tile of the grouped GEMMs (k_gemm<.., 2, 2>)
constexpr int MAX_ASSIGN = 32768;

struct MoeWs {
  size_t logits, split, ids, wts, row_of, inv, tiles, ntiles, mid, eo, total;
  int splits, max_tiles;
};

MoeWs moe_ws(int M, int H, int E, int k, int inter) {
  MoeWs w;
  size_t off = 0;
  const size_t A = (size_t)M * k;
  w.splits = gemm_splits(M, E, H);
  w.max_tiles = (int)((A + TILE_M - 1) / TILE_M) + E;
  w.logits = off; off = align256(off + (size_t)M * E * 4);
  w.split = off; off = align256(off + (w.splits > 1 ? (size_t)w.splits * M * E * 4 : 0));
  w.ids = off; off = align256(off + A * 4);
  w.wts = off; off = align256(off + A * 4);
  w.row_of = off; off = align256(off + A * 4);
  w.inv = off; off = align256(off + A * 4);
  w.tiles = off; off = align256(off + (size_t)w.max_tiles * 3 * 4);
  w.ntiles = off; off = align256(off + 4);
  w.mid = off; off = align256(off + A * inter * 2);
  w.eo = off; off = align256(off + A * H * 4);
  w.total = off;
  return w;
}

__device__ __forceinline__ uint32_t orderable(float v) {
  uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// One wave per row: top_k of the E router logits (largest first, ties to the
// lower id) and their softmax weights renormalised over the chosen experts.
__global__ void __launch_bounds__(256)
k_moe_route(const float *__restrict__ logits, int E, int k, int M_max, const int32_t *__restrict__ m_count,
            int32_t *__restrict__ ids, float *__restrict__ wts) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= M_max || t >= *m_count) return;
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int e = lane + 64 * j;
    v[j] = e < E ? logits[(size_t)t * E + e] : -__builtin_inff();
  }
  float top0 = 0.0f, denom = 0.0f, my_p = 0.0f;
  int my_e = 0;
  for (int s = 0; s < k; ++s) {
    unsigned long long best = 0ull;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int e = lane + 64 * j;
      if (e < E && v[j] != -__builtin_inff()) {
        unsigned long long key = ((unsigned long long)orderable(v[j]) << 32) | (0xffffffffu - (uint32_t)e);
        best = key > best ? key : best;
      }
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      unsigned long long o = __shfl_xor(best, off, 64);
      best = o > best ? o : best;
    }
    const int e = (int)(0xffffffffu - (uint32_t)(best & 0xffffffffu));
    float le = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane + 64 * j == e) {
        le = v[j];
        v[j] = -__builtin_inff();
      }
    le = __shfl(le, e & 63, 64);
    if (s == 0) top0 = le;
    const float p = __expf(le - top0);
    denom += p;
    if (lane == s) {
      my_p = p;
      my_e = e;
    }
  }
  if (lane < k) {
    ids[(size_t)t * k + lane] = my_e;
    wts[(size_t)t * k + lane] = my_p / denom;
  }
}

// One workgroup: a stable counting sort of the K* * k assignments j = row * k +
// slot by expert (each expert's assignments in increasing j, the order of the
// keys (expert, j)), then the gather rows, inverse positions and the (expert,
// first, end) row tiles.  Assignments go in chunks of one per thread; within a
// wave, the lanes holding the same expert are found with one ballot per bit of
// the expert id, and the per-wave counts of the chunk place each assignment
// after those of earlier waves and earlier chunks.
__global__ void __launch_bounds__(1024)
k_moe_group(const int32_t *__restrict__ ids, int E, int k, int M_max, const int32_t *__restrict__ m_count,
            int32_t *__restrict__ row_of, int32_t *__restrict__ inv, int32_t *__restrict__ tiles,
            int32_t *__restrict__ n_tiles) {
  __shared__ int s_base[256];           // per expert: count, then the next free position
  __shared__ int s_wcnt[16][256];       // per wave and expert: assignments of the current chunk
  __shared__ int s_wave[17];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, nw = blockDim.x >> 6;
  const int N = min(*m_count, M_max) * k;
  auto expert_of = [&](int j) {
    const int e = ids[j];
    return e < 0 ? 0 : (e >= E ? E - 1 : e);
  };
  for (int e = tid; e < 256; e += blockDim.x) s_base[e] = 0;
  for (int i = tid; i < 16 * 256; i += blockDim.x) (&s_wcnt[0][0])[i] = 0;
  __syncthreads();
  for (int j = tid; j < N; j += blockDim.x) atomicAdd(&s_base[expert_of(j)], 1);
  __syncthreads();
  // exclusive scans over experts: row offsets and tile offsets
  const int cnt = tid < E ? s_base[tid] : 0;
  const int ntl = (cnt + TILE_M - 1) / TILE_M;
  int tot_r, tot_t;
  const int off_r = block_exclusive_scan(cnt, s_wave, &tot_r);
  const int off_t = block_exclusive_scan(ntl, s_wave, &tot_t);
  if (tid < E) {
    for (int q = 0; q < ntl; ++q) {
      const int tt = off_t + q;
      tiles[3 * tt] = tid;
      tiles[3 * tt + 1] = off_r + q * TILE_M;
      tiles[3 * tt + 2] = off_r + cnt;
    }
    s_base[tid] = off_r;
  }
  if (tid == 0) n_tiles[0] = tot_t;
  __syncthreads();
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int c0 = 0; c0 < N; c0 += blockDim.x) {
    const int j = c0 + tid;
    const bool live = j < N;
    const int e = live ? expert_of(j) : 0;
    unsigned long long same = __ballot(live);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (e >> b) & 1;
      const unsigned long long m = __ballot(bit);
      same &= bit ? m : ~m;
    }
    const int wrank = __popcll(same & below);
    if (live && wrank == 0) s_wcnt[wv][e] = __popcll(same);
    __syncthreads();
    if (live) {
      int p = s_base[e] + wrank;
      for (int v = 0; v < wv; ++v) p += s_wcnt[v][e];
      row_of[p] = j / k;
      inv[j] = p;
    }
    __syncthreads();
    for (int e2 = tid; e2 < E; e2 += blockDim.x) {
      int add = 0;
      for (int v = 0; v < nw; ++v) {
        add += s_wcnt[v][e2];
        s_wcnt[v][e2] = 0;
      }
      s_base[e2] += add;
    }
    __syncthreads();
  }
}

// One workgroup per row: out[t] += sum_s w[t][s] * eo[inv[t*k + s]], slot order.
__global__ void __launch_bounds__(256)
k_moe_combine(const float *__restrict__ eo, const int32_t *__restrict__ inv, const float *__restrict__ wts,
              int H, int k, const int32_t *__restrict__ m_count, float *__restrict__ out) {
  const int t = blockIdx.x;
  if (t >= *m_count) return;
  for (int c = threadIdx.x * 4; c < H; c += 1024) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < k; ++s) {
      const float w = wts[(size_t)t * k + s];
      const float4 v = *(const float4 *)(eo + (size_t)inv[(size_t)t * k + s] * H + c);
      acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
    }
    float4 *o = (float4 *)(out + (size_t)t * H + c);
    float4 x = *o;
    x.x += acc.x; x.y += acc.y; x.z += acc.z; x.w += acc.w;
    *o = x;
  }
}

}  // namespace

size_t moe_ws_bytes(int M_max, int H, int E, int top_k, int inter) {
  return moe_ws(M_max, H, E, top_k, inter).total;
}

bool moe_supported(int M_max, int H, int E, int top_k) {
  return E >= 1 && E <= 256 && top_k >= 1 && top_k <= 64 && top_k <= E &&
         (long long)M_max * top_k <= MAX_ASSIGN && H % 4 == 0;
}

int moe_launch(const MoeArgs &m, hipStream_t s) {
  const MoeWs L = moe_ws(m.M_max, m.H, m.E, m.top_k, m.inter);
  char *b = (char *)m.ws;
  float *logits = (float *)(b + L.logits);
  int32_t *ids = (int32_t *)(b + L.ids);
  float *wts = (float *)(b + L.wts);
  int32_t *row_of = (int32_t *)(b + L.row_of);
  int32_t *inv = (int32_t *)(b + L.inv);
  int32_t *tiles = (int32_t *)(b + L.tiles);
  int32_t *ntiles = (int32_t *)(b + L.ntiles);
  uint16_t *mid = (uint16_t *)(b + L.mid);
  float *eo = (float *)(b + L.eo);
  const int M = m.M_max, A = m.M_max * m.top_k;

  GemmArgs r = {};
  r.A = m.h; r.lda = m.H; r.K = m.H; r.M_max = M; r.m_count = m.m_count;
  r.W = m.w_router; r.ldw = m.H; r.N = m.E;
  r.out_f32 = logits; r.ldo = m.E;
  r.splits = m.E % 4 == 0 ? L.splits : 1; r.split_part = (float *)(b + L.split);
  DCUT_TRY(gemm_launch(DCUT_KERNEL_MOE, EPI_STORE_F32, r, s));
  DCUT_TRY(launch(DCUT_KERNEL_MOE, k_moe_route, dim3((M + 3) / 4), dim3(256), 0, s, (const float *)logits,
                  m.E, m.top_k, M, m.m_count, ids, wts));
  DCUT_TRY(launch(DCUT_KERNEL_MOE, k_moe_group, dim3(1), dim3(1024), 0, s, (const int32_t *)ids,
                  m.E, m.top_k, M, m.m_count, row_of, inv, tiles, ntiles));
  // gathered rows of h through the grouped gate-up GEMM with the SwiGLU epilogue
  GemmArgs gu = {};
  gu.A = m.h; gu.lda = m.H; gu.K = m.H; gu.M_max = A; gu.m_count = m.m_count;
  gu.W = m.w_gate_up; gu.ldw = m.H; gu.N = 2 * m.inter; gu.swiglu_inter = m.inter;
  gu.out_bf16 = mid; gu.ldo = m.inter;
  gu.tiles = tiles; gu.n_tiles = ntiles; gu.m_tiles = L.max_tiles; gu.w_stride = (long long)2 * m.inter * m.H;
  gu.a_rows = row_of; gu.a_extent = M;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_GATE_UP, EPI_SWIGLU, gu, s));
  GemmArgs dn = {};
  dn.A = mid; dn.lda = m.inter; dn.K = m.inter; dn.M_max = A; dn.m_count = m.m_count;
  dn.W = m.w_down; dn.ldw = m.inter; dn.N = m.H;
  dn.out_f32 = eo; dn.ldo = m.H;
  dn.tiles = tiles; dn.n_tiles = ntiles; dn.m_tiles = L.max_tiles; dn.w_stride = (long long)m.H * m.inter;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_DOWN, EPI_STORE_F32, dn, s));
  return launch(DCUT_KERNEL_MOE, k_moe_combine, dim3(M), dim3(256), 0, s, (const float *)eo,
                (const int32_t *)inv, (const float *)wts, m.H, m.top_k, m.m_count, m.x_out);
}

}  // namespace dcut
