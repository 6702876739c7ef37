// Ragged causal GQA attention over per-request KV slabs, split over key chunks.
//
// App. C: every kept position is scored against its request's accepted prefix
// (cache slots 0..L_i-1) and, causally, against the kept block positions before
// it (slots L_i..L_i+k, appended by the QKV epilogue).
//
// Work item = (request i, kv head g, chunk c).  Chunk c covers cache keys
// [c*CH, min((c+1)*CH, L_i)); the last chunk also covers the block keys
// [L_i, L_i + d_i).  The chunking depends on L_i only, never on d_i, so a row's
// partial results are the same whichever later rows are kept.  All G = n_q/n_kv
// query heads of the group and all d_i kept rows (G*d_i <= 256 rows, 16 per
// wave) share each 64-key tile, so the cache is read from HBM exactly once.
//
// Per tile and wave (v_mfma_f32_16x16x32_bf16):
//   S^T[key][row] = K[key][:] . Q[row][:]   -> lane (row = lane%16) owns keys
//                                              4*(lane/16)+j of each 16-key block
//   online softmax per row (exp2 domain), row statistics stay lane-local
//   O^T[d][row]  += V^T[d][key] . P^T[key][row], with P taken straight from the
//                   S^T accumulators (the same key permutation is applied to the
//                   V^T operand), V staged transposed in LDS.
// Partial (o, m, l) per (row, head, chunk) are merged in chunk order by
// k_attn_combine; a request with a single chunk is finished in place.
#include "dcut_internal.h"

namespace dcut {

namespace {

constexpr int KT = 64;     // keys per tile

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

template <int HD, int NW>
__global__ void __launch_bounds__(NW * 64)
k_attn(AttnArgs a) {
  constexpr int LDKs = HD + 8;      // K tile row (bf16), 16-byte aligned rows
  constexpr int LDV = KT + 2;       // V^T tile row (bf16): an odd number of words
  constexpr int NS = HD / 32;       // k-steps of the QK product
  constexpr int NT = HD / 16;       // 16-row tiles of O^T
  constexpr int TOTCH = KT * (HD / 8);                 // 16-byte chunks per tile
  constexpr int NCH = (TOTCH + NW * 64 - 1) / (NW * 64);  // per thread
  __shared__ __align__(16) uint16_t Ks[KT * LDKs];
  __shared__ __align__(16) uint16_t Vt[HD * LDV];

  const int MC = a.max_chunks;
  const int idx = blockIdx.x;
  const int c = idx % MC;
  const int g = (idx / MC) % a.n_kv;
  const int i = idx / (MC * a.n_kv);
  if (i >= a.B) return;
  const int t0 = a.cu[i];
  const int d = a.cu[i + 1] - t0;
  const int L0 = a.ctx_len[i];
  const int cap = a.kv_cap[i];
  if (d <= 0) return;
  if (L0 < 0 || L0 + a.D + 1 > cap) {
    if (c == 0 && g == 0 && threadIdx.x == 0 && a.dev_err) atomicOr(a.dev_err, DCUT_DERR_CAPACITY);
  }
  const int L = usable_ctx(L0, cap, a.D);
  const int nc = n_chunks(L, a.chunk, MC);
  if (c >= nc) return;
  const int kstart = c * a.chunk;
  int kend = (c == nc - 1) ? L + d : min((c + 1) * a.chunk, L);
  if (kend > cap) kend = cap;

  const int G = a.n_q / a.n_kv;
  const int R = G * d;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp4 = lane >> 4;

  // this lane's query row
  const int rr = wave * 16 + l16;
  const bool row_ok = rr < R;
  const int hl = row_ok ? rr / d : 0;
  const int krow = row_ok ? rr - hl * d : 0;
  const int head = g * G + hl;
  const int t = t0 + krow;
  const int kmax = L + krow;          // last visible key position
  const bool wave_active = wave * 16 < R;

  bf16x8 qf[NS];
  {
    const uint16_t *qp = a.q + ((size_t)t * a.n_q + head) * HD + 8 * grp4;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      if (row_ok) qf[s] = *(const bf16x8 *)(qp + 32 * s);
      else {
        uint4 z = make_uint4(0, 0, 0, 0);
        qf[s] = *(bf16x8 *)&z;
      }
    }
  }

  floatx4 o[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) o[n] = {0.f, 0.f, 0.f, 0.f};
  float m_run = -__builtin_inff();
  float l_run = 0.0f;
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)

  const size_t slab = (size_t)a.kv_base[i] + (size_t)g * cap * HD;
  const uint16_t *kbase = a.kv_k + slab;
  const uint16_t *vbase = a.kv_v + slab;

  // chunk -> (key row, column): 8 lanes cover one key's 128 contiguous bytes
  int ckr[NCH], cc8[NCH];
  bool cok[NCH];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    int ch = tid + j * NW * 64;
    cok[j] = ch < TOTCH;
    int blk = ch >> 6, l = ch & 63;
    ckr[j] = (blk % (KT / 8)) * 8 + (l >> 3);
    cc8[j] = (blk / (KT / 8)) * 64 + (l & 7) * 8;
  }
  uint4 rk[NCH], rv[NCH];
  auto gload = [&](int p0) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      int p = p0 + ckr[j];
      if (cok[j] && p < kend) {
        rk[j] = *(const uint4 *)(kbase + (size_t)p * HD + cc8[j]);
        rv[j] = *(const uint4 *)(vbase + (size_t)p * HD + cc8[j]);
      } else {
        rk[j] = make_uint4(0, 0, 0, 0);
        rv[j] = make_uint4(0, 0, 0, 0);
      }
    }
  };

  const int ntiles = (kend - kstart + KT - 1) / KT;
  if (ntiles > 0) gload(kstart);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int p0 = kstart + tile * KT;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      if (!cok[j]) continue;
      *(uint4 *)(Ks + ckr[j] * LDKs + cc8[j]) = rk[j];
      const uint16_t *ve = (const uint16_t *)&rv[j];
#pragma unroll
      for (int e = 0; e < 8; ++e) Vt[(cc8[j] + e) * LDV + ckr[j]] = ve[e];
    }
    __syncthreads();
    if (tile + 1 < ntiles) gload(p0 + KT);
    if (!wave_active) continue;

    // S^T tiles: 4 blocks of 16 keys
    floatx4 s4[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s4[kb] = {0.f, 0.f, 0.f, 0.f};
      const uint16_t *kp = Ks + (kb * 16 + l16) * LDKs + 8 * grp4;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        bf16x8 kf = *(const bf16x8 *)(kp + 32 * s);
        s4[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[s], s4[kb], 0, 0, 0);
      }
    }
    // mask + scale, tile max
    float tmax = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int p = p0 + kb * 16 + 4 * grp4 + j;
        bool vis = row_ok && p < kend && p <= kmax;
        float v = vis ? s4[kb][j] * sl2 : -__builtin_inff();
        s4[kb][j] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    float alpha = 1.0f;
    if (m_new != -__builtin_inff()) alpha = exp2f(m_run - m_new);
    float psum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = s4[kb][j];
        float pv = (v == -__builtin_inff()) ? 0.0f : exp2f(v - m_new);
        s4[kb][j] = pv;
        psum += pv;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int n = 0; n < NT; ++n) o[n] *= alpha;

    // O^T += V^T P^T over two 32-key steps
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 pf;
      uint32_t *pw = (uint32_t *)&pf;
      pw[0] = pack_bf2(s4[2 * ks][0], s4[2 * ks][1]);
      pw[1] = pack_bf2(s4[2 * ks][2], s4[2 * ks][3]);
      pw[2] = pack_bf2(s4[2 * ks + 1][0], s4[2 * ks + 1][1]);
      pw[3] = pack_bf2(s4[2 * ks + 1][2], s4[2 * ks + 1][3]);
      const int key_a = 32 * ks + 4 * grp4;          // keys key_a..+3 and key_a+16..+3
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const uint32_t *vp = (const uint32_t *)(Vt + (n * 16 + l16) * LDV + key_a);
        bf16x8 vf;
        uint32_t *vw = (uint32_t *)&vf;
        vw[0] = vp[0];
        vw[1] = vp[1];
        vw[2] = vp[8];
        vw[3] = vp[9];
        o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[n], 0, 0, 0);
      }
    }
  }
  if (!row_ok) return;

  // lane holds O^T[16n + 4*grp4 + j][row]
  if (nc == 1) {
    const float inv = l_run > 0.0f ? 1.0f / l_run : 0.0f;
    uint16_t *op = a.out + ((size_t)t * a.n_q + head) * HD;
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int j = 0; j < 4; ++j) op[16 * n + 4 * grp4 + j] = f2bf(o[n][j] * inv);
  } else {
    float *pp = a.part + (((size_t)t * a.n_q + head) * MC + c) * (HD + 2);
#pragma unroll
    for (int n = 0; n < NT; ++n)
      *(float4 *)(pp + 16 * n + 4 * grp4) = make_float4(o[n][0], o[n][1], o[n][2], o[n][3]);
    if (grp4 == 0) {
      pp[HD] = m_run;
      pp[HD + 1] = l_run;
    }
  }
}

// One wave per (row, head): merge the chunk partials in chunk order.
template <int HD>
__global__ void __launch_bounds__(256)
k_attn_combine(AttnArgs a, const int32_t *__restrict__ packed_req, int rows_max) {
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int M = a.cu[a.B];
  const int t = wid / a.n_q, head = wid - t * a.n_q;
  if (t >= M || t >= rows_max) return;
  const int req = packed_req[t];
  if (req < 0 || req >= a.B) return;
  const int MC = a.max_chunks;
  const int L = usable_ctx(a.ctx_len[req], a.kv_cap[req], a.D);
  const int nc = n_chunks(L, a.chunk, MC);
  if (nc == 1) return;
  const float *pp = a.part + ((size_t)t * a.n_q + head) * MC * (HD + 2);
  float mx = -__builtin_inff();
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, pp[c * (HD + 2) + HD]);
  constexpr int PER = HD / 64;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  float lsum = 0.0f;
  for (int c = 0; c < nc; ++c) {
    const float *q = pp + c * (HD + 2);
    float mc = q[HD];
    float sc = (mc == -__builtin_inff()) ? 0.0f : exp2f(mc - mx);
    lsum += q[HD + 1] * sc;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += q[lane * PER + e] * sc;
  }
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
  uint16_t *op = a.out + ((size_t)t * a.n_q + head) * HD;
#pragma unroll
  for (int e = 0; e < PER; ++e) op[lane * PER + e] = f2bf(acc[e] * inv);
}

template <int HD>
int launch_hd(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves, hipStream_t s) {
  const dim3 grid(a.B * a.n_kv * a.max_chunks);
  if (waves <= 4) {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 4>, grid, dim3(256), 0, s, a));
  } else if (waves <= 8) {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 8>, grid, dim3(512), 0, s, a));
  } else {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 16>, grid, dim3(1024), 0, s, a));
  }
  int nw = rows_max * a.n_q;
  return launch(DCUT_KERNEL_ATTN_COMBINE, k_attn_combine<HD>, dim3((nw + 3) / 4), dim3(256), 0, s, a,
                packed_req, rows_max);
}

}  // namespace

int attention_launch(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves, hipStream_t s) {
  if (a.head_dim == 128) return launch_hd<128>(a, rows_max, packed_req, waves, s);
  if (a.head_dim == 64) return launch_hd<64>(a, rows_max, packed_req, waves, s);
  return DCUT_EUNSUPPORTED;
}

}  // namespace dcut
