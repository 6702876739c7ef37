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
// wave) share each 32-key tile, so the cache is read from HBM exactly once.
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
//
// Workgroup b takes item b of the longest-first work order (attn_plan.h),
// which the layer's first norm kernel builds in one extra workgroup; batches
// too large to plan and grids of one round of slots number the items
// arithmetically, chunk index slowest.
#include "attn_plan.h"
#include "dcut_internal.h"

namespace dcut {

namespace {

constexpr int KT = 32;     // keys per tile

typedef short short4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// Barrier of the LDS ring: each wave has waited (s_waitcnt vmcnt) for its own
// loads of the stage it reads next, so only the hardware barrier is needed; a
// memory fence here would drain every stage still in flight.  The empty asm
// statements keep the compiler from moving LDS accesses across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Transposing LDS reads (ds_read_b64_tr_b16), four columns x two key halves per
// call.  They are issued from one asm statement that also waits for them
// (lgkmcnt(0)), so the compiler only ever sees completed results; it cannot
// model these reads itself without also draining every LDS-DMA stage still in
// flight (vmcnt(0)).  The ring protocol (vmcnt wait + barrier) orders them
// after the DMA writes of the stage they read.
__device__ __forceinline__ void lds_read_tr16_x8(short4v (&r)[8], const uint32_t (&ad)[8]) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8\n\t"
      "ds_read_b64_tr_b16 %1, %9\n\t"
      "ds_read_b64_tr_b16 %2, %10\n\t"
      "ds_read_b64_tr_b16 %3, %11\n\t"
      "ds_read_b64_tr_b16 %4, %12\n\t"
      "ds_read_b64_tr_b16 %5, %13\n\t"
      "ds_read_b64_tr_b16 %6, %14\n\t"
      "ds_read_b64_tr_b16 %7, %15\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
      : "v"(ad[0]), "v"(ad[1]), "v"(ad[2]), "v"(ad[3]), "v"(ad[4]), "v"(ad[5]), "v"(ad[6]), "v"(ad[7])
      : "memory");
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void *base, int bytes) {
  const uintptr_t b = (uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const int n = __builtin_amdgcn_readfirstlane(bytes);
  return __builtin_amdgcn_make_buffer_rsrc((void *)(((uintptr_t)hi << 32) | lo), (short)0, n, 0x00020000);
}

// NSTAGE LDS ring stages: NSTAGE - 1 tiles in flight while one is used.  At
// most 168 registers (three waves per SIMD), so three 4-wave workgroups with
// 3-stage rings (48 KB of LDS each) share a CU.
template <int HD, int NW, int NSTAGE>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3)))
k_attn(AttnArgs a) {
  constexpr int ROWB = HD * 2;              // bytes per key row
  constexpr int CPR = ROWB / 16;            // 16-byte chunks per key row (8 or 16)
  constexpr int TILEB = KT * ROWB;          // bytes of one K (or V) tile
  constexpr int STAGEB = 2 * TILEB;         // K tile then V tile
  constexpr int RPI = 1024 / ROWB;          // key rows per 1 KB wave load
  constexpr int LPK = (TILEB / 1024 + NW - 1) / NW;      // wave loads per stage for K (and for V)
  constexpr int LPW = 2 * LPK;
  constexpr int NS = HD / 32;               // k-steps of the QK product
  constexpr int NT = HD / 16;               // 16-row tiles of O^T
  __shared__ __align__(16) unsigned char ring[NSTAGE * STAGEB];

  const int MC = a.max_chunks;
  const int tid = threadIdx.x, lane = tid & 63;
  int i, g, c, t0, d, L, cap;
  if (a.plan) {
    const int idx = blockIdx.x;
    const int n = a.plan[0];
    const int4 *it = (const int4 *)((const char *)a.plan + PLAN_HEAD) + 2 * idx;
    const int4 e0 = it[0], e1 = it[1];
    if (idx >= n) return;
    i = e0.x; g = e0.y; c = e0.z; t0 = e0.w;
    d = e1.x; L = e1.y; cap = e1.z;
  } else {
    // Chunk index slowest: the work items that exist for every request (the
    // first chunks) come first, so workgroups of chunks a request does not
    // have are dispatched last and exit without holding a slot among live ones.
    const int idx = blockIdx.x;
    c = idx / (a.B * a.n_kv);
    g = idx % a.n_kv;
    i = (idx / a.n_kv) % a.B;
    if (c >= MC) return;
    t0 = a.cu[i];
    d = a.cu[i + 1] - t0;
    const int L0 = a.ctx_len[i];
    cap = a.kv_cap[i];
    if (d <= 0) return;
    if (L0 < 0 || L0 + a.D + 1 > cap) {
      if (c == 0 && g == 0 && threadIdx.x == 0 && a.dev_err) atomicOr(a.dev_err, DCUT_DERR_CAPACITY);
    }
    L = usable_ctx(L0, cap, a.D);
    if (c >= n_chunks(L, a.chunk, MC)) return;
  }
  const int nc = n_chunks(L, a.chunk, MC);
  const int kstart = c * a.chunk;
  int kend = (c == nc - 1) ? L + d : min((c + 1) * a.chunk, L);
  if (kend > cap) kend = cap;

  const int G = a.n_q / a.n_kv;
  const int R = G * d;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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

  // K and V of (request i, kv head g) as buffers: out-of-range keys read as zeros
  const size_t slab = (size_t)a.kv_base[i] + (size_t)g * cap * HD;
  const int slab_bytes = cap * ROWB;
  const __amdgpu_buffer_rsrc_t rK = uniform_rsrc(a.kv_k + slab, slab_bytes);
  const __amdgpu_buffer_rsrc_t rV = uniform_rsrc(a.kv_v + slab, slab_bytes);
  // Tile layout in LDS: key row r at r * ROWB; its 16-byte chunk c holds the
  // row's global chunk c ^ (r % CPR), so 16 consecutive rows read at one column
  // land in different banks.  A wave load fills RPI rows (1 KB): lane l writes
  // row l / CPR, chunk l % CPR.
  const int lrow = lane / CPR, lchk = lane % CPR;
  auto issue = [&](int tile, int slot) {
    const int p0 = kstart + tile * KT;
    unsigned char *st = ring + slot * STAGEB;
#pragma unroll
    for (int j = 0; j < LPK; ++j) {
      const int q = wave + NW * j;                 // 1 KB block of the K (and V) tile
      if (q >= TILEB / 1024) continue;
      const int r = q * RPI + lrow;                // key row within the tile
      const int p = p0 + r;
      const unsigned off = p < kend ? (unsigned)(p * ROWB + 16 * (lchk ^ (r % CPR))) : 0x80000000u;
      // each key is read once: non-temporal loads (cache policy nt) keep the
      // stream from displacing reused lines in L2
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rK, (lds_void *)(st + q * 1024), 16, off, 0, 0, CPOL_NT);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rV, (lds_void *)(st + TILEB + q * 1024), 16, off, 0, 0, CPOL_NT);
    }
  };

  const int ntiles = (kend - kstart + KT - 1) / KT;
#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < ntiles) issue(s, s);
  constexpr int W0 = 0 | (7 << 4) | (15 << 8);
  constexpr int W1 = (LPW & 15) | ((LPW >> 4) << 14) | (7 << 4) | (15 << 8);
  constexpr int W2 = ((2 * LPW) & 15) | (((2 * LPW) >> 4) << 14) | (7 << 4) | (15 << 8);
  for (int tile = 0; tile < ntiles; ++tile) {
    const int pending = min(NSTAGE - 2, ntiles - 1 - tile);
    if (pending >= 2) __builtin_amdgcn_s_waitcnt(W2);
    else if (pending == 1) __builtin_amdgcn_s_waitcnt(W1);
    else __builtin_amdgcn_s_waitcnt(W0);
    ring_barrier();
    if (tile + NSTAGE - 1 < ntiles) issue(tile + NSTAGE - 1, (tile + NSTAGE - 1) % NSTAGE);
    if (!wave_active) continue;
    const int p0 = kstart + tile * KT;
    const unsigned char *Ks = ring + (tile % NSTAGE) * STAGEB;
    const unsigned char *Vs = Ks + TILEB;

    // S^T: KT/16 blocks of 16 keys; lane reads key row kb*16 + l16, global chunk 4s + grp4
    floatx4 s4[KT / 16];
#pragma unroll
    for (int kb = 0; kb < KT / 16; ++kb) {
      s4[kb] = {0.f, 0.f, 0.f, 0.f};
      const int r = kb * 16 + l16;
      const unsigned char *kp = Ks + r * ROWB;
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        bf16x8 kf = *(const bf16x8 *)(kp + 16 * ((4 * s + grp4) ^ (r % CPR)));
        s4[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[s], s4[kb], 0, 0, 0);
      }
    }
    // mask + scale, tile max
    float tmax = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < KT / 16; ++kb)
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
    for (int kb = 0; kb < KT / 16; ++kb)
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

    // O^T += V^T P^T per 32-key step.  P^T slots of this lane: keys 4*grp4+j of the
    // two 16-key blocks; the V^T fragment with the same keys comes from two
    // transposing reads: source lane s of a 16-lane group reads key row
    // k0 + s/4, columns 16n + 4(s%4)..+3, and lane d receives keys k0..k0+3 of
    // column 16n + d.
#pragma unroll
    for (int ks = 0; ks < KT / 32; ++ks) {
      bf16x8 pf;
      uint32_t *pw = (uint32_t *)&pf;
      pw[0] = pack_bf2(s4[2 * ks][0], s4[2 * ks][1]);
      pw[1] = pack_bf2(s4[2 * ks][2], s4[2 * ks][3]);
      pw[2] = pack_bf2(s4[2 * ks + 1][0], s4[2 * ks + 1][1]);
      pw[3] = pack_bf2(s4[2 * ks + 1][2], s4[2 * ks + 1][3]);
      const int r0 = 32 * ks + 4 * grp4 + (l16 >> 2);      // source key row, first half
      const int r1 = r0 + 16;
      const int csub = 4 * (l16 & 3);                       // element offset within 16 columns
      static_assert(NT % 4 == 0, "transposing reads come in groups of four columns");
#pragma unroll
      for (int n0 = 0; n0 < NT; n0 += 4) {
        uint32_t ad[8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int col = 16 * (n0 + u) + csub;              // first of 4 columns read
          const int gc = col >> 3, half = (col & 7) * 2;     // 16-byte chunk, byte offset in it
          ad[2 * u] = (uint32_t)(uintptr_t)(Vs + r0 * ROWB + 16 * (gc ^ (r0 % CPR)) + half);
          ad[2 * u + 1] = (uint32_t)(uintptr_t)(Vs + r1 * ROWB + 16 * (gc ^ (r1 % CPR)) + half);
        }
        short4v vr[8];
        lds_read_tr16_x8(vr, ad);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          bf16x8 vf;
          short4v *vw = (short4v *)&vf;
          vw[0] = vr[2 * u];
          vw[1] = vr[2 * u + 1];
          o[n0 + u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[n0 + u], 0, 0, 0);
        }
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
  // the loads of up to CG chunks are issued together (one memory latency per
  // group rather than per chunk); the sums still run in chunk order
  constexpr int CG = 8;
  constexpr int PER = HD / 64;
  const float *pl = pp + lane * PER;
  uint16_t *op = a.out + ((size_t)t * a.n_q + head) * HD;
  if (nc <= CG) {
    // every chunk's (max, sum, partial) in one memory round trip; the same
    // operations in the same order as the two-pass loop below
    float mv[CG], lv[CG], xv[CG][PER];
#pragma unroll
    for (int c = 0; c < CG; ++c) {
      mv[c] = c < nc ? pp[c * (HD + 2) + HD] : -__builtin_inff();
      lv[c] = c < nc ? pp[c * (HD + 2) + HD + 1] : 0.0f;
#pragma unroll
      for (int e = 0; e < PER; ++e) xv[c][e] = c < nc ? pl[c * (HD + 2) + e] : 0.0f;
    }
    float mx = -__builtin_inff();
#pragma unroll
    for (int c = 0; c < CG; ++c) mx = fmaxf(mx, mv[c]);
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
    float lsum = 0.0f;
#pragma unroll
    for (int c = 0; c < CG; ++c) {
      if (c < nc) {
        const float sc = (mv[c] == -__builtin_inff()) ? 0.0f : exp2f(mv[c] - mx);
        lsum += lv[c] * sc;
#pragma unroll
        for (int e = 0; e < PER; ++e) acc[e] += xv[c][e] * sc;
      }
    }
    const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
#pragma unroll
    for (int e = 0; e < PER; ++e) op[lane * PER + e] = f2bf(acc[e] * inv);
    return;
  }
  float mx = -__builtin_inff();
  for (int c0 = 0; c0 < nc; c0 += CG) {
    float mv[CG];
#pragma unroll
    for (int c = 0; c < CG; ++c) mv[c] = c0 + c < nc ? pp[(c0 + c) * (HD + 2) + HD] : -__builtin_inff();
#pragma unroll
    for (int c = 0; c < CG; ++c) mx = fmaxf(mx, mv[c]);
  }
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  float lsum = 0.0f;
  for (int c0 = 0; c0 < nc; c0 += CG) {
    float mv[CG], lv[CG], xv[CG][PER];
#pragma unroll
    for (int c = 0; c < CG; ++c) {
      if (c0 + c < nc) {
        const float *q = pp + (c0 + c) * (HD + 2);
        mv[c] = q[HD];
        lv[c] = q[HD + 1];
#pragma unroll
        for (int e = 0; e < PER; ++e) xv[c][e] = q[lane * PER + e];
      }
    }
#pragma unroll
    for (int c = 0; c < CG; ++c) {
      if (c0 + c < nc) {
        const float sc = (mv[c] == -__builtin_inff()) ? 0.0f : exp2f(mv[c] - mx);
        lsum += lv[c] * sc;
#pragma unroll
        for (int e = 0; e < PER; ++e) acc[e] += xv[c][e] * sc;
      }
    }
  }
  const float inv = lsum > 0.0f ? 1.0f / lsum : 0.0f;
#pragma unroll
  for (int e = 0; e < PER; ++e) op[lane * PER + e] = f2bf(acc[e] * inv);
}

template <int HD>
int launch_hd(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves, hipStream_t s) {
  // Up to 64 rows per item: 4 waves and a 3-stage ring, three workgroups per
  // CU, so one streams on while another starts or finishes an item.  Up to 128
  // or 256 rows: 8 or 16 waves and a 4-stage ring, two or one per CU (8 waves
  // measured faster than 4 at two workgroups per CU: the extra waves share
  // the tile loads).
  const dim3 grid(a.B * a.n_kv * a.max_chunks);
  if (waves <= 4) {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 4, 3>, grid, dim3(256), 0, s, a));
  } else if (waves <= 8) {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 8, 4>, grid, dim3(512), 0, s, a));
  } else {
    DCUT_TRY(launch(DCUT_KERNEL_ATTN, k_attn<HD, 16, 4>, grid, dim3(1024), 0, s, a));
  }
  int nw = rows_max * a.n_q;
  return launch(DCUT_KERNEL_ATTN_COMBINE, k_attn_combine<HD>, dim3((nw + 3) / 4), dim3(256), 0, s, a,
                packed_req, rows_max);
}

}  // namespace

size_t attn_plan_bytes(int B, int n_kv, int max_chunks) {
  // a grid that fits in one round of workgroup slots gains nothing from an order
  if (B > PLAN_MAX_B || (long long)B * n_kv * max_chunks <= PLAN_MIN_ITEMS) return 0;
  return PLAN_HEAD + (size_t)B * n_kv * max_chunks * 8 * sizeof(int32_t);
}

int attention_launch(const AttnArgs &a, int rows_max, const int32_t *packed_req, int waves, hipStream_t s) {
  if (a.plan && a.B > PLAN_MAX_B) return DCUT_EINVAL;
  if (a.head_dim == 128) return launch_hd<128>(a, rows_max, packed_req, waves, s);
  if (a.head_dim == 64) return launch_hd<64>(a, rows_max, packed_req, waves, s);
  return DCUT_EUNSUPPORTED;
}

}  // namespace dcut
