// bf16 NT GEMM on gfx950 MFMA with fused epilogues: C = A W^T, A [M][K], W [N][K].
//
// Block tile (2*WM*32) x (2*WN*32) x 64 with four waves in a 2 x 2 grid; every
// wave owns WM x WN tiles of v_mfma_f32_32x32x16_bf16 (float32 accumulators).
// Operands stream from memory straight into a double-buffered LDS ring (buffer
// loads with the LDS destination, XOR-swizzled 16-byte chunks, hardware zeros
// for rows and k beyond the operands), so the next k-slice is in flight while
// the current one is multiplied and no registers stage it.  64 KB of LDS per
// workgroup keeps two workgroups resident per CU; deeper rings and larger tiles
// measured slower on MI355X (fewer resident workgroups).  Residual
// GEMMs with few output tiles split K over gridDim.y (a factor fixed by the
// shape); k_splitk_reduce then adds the partial tiles in split order.
//
// Rows: the grid covers M_max rows; the live row count M (K*) is read on the
// device and whole row tiles beyond it exit at once.  The tile shape never
// depends on M and the k loop is the same for every row, so a row's result
// does not depend on which or how many other rows are present.
//
// Column groups: each 32-column MFMA tile loads a 32-row group of W chosen by
// the epilogue, so that values an epilogue combines sit in the same lane:
//   SWIGLU    groups (2p, 2p+1) = (gate rows, up rows) of the same 32 outputs;
//   QKV_ROPE  groups (2p, 2p+1) = the two halves (j, j + hd/2) of RoPE pairs.
// Tile order is XCD-major: consecutive workgroups of one XCD (the hardware
// deals workgroups round-robin over 8 XCDs) walk the row tiles of the same
// column tiles, so the W slice they share stays in that XCD's L2.

#include "dcut_internal.h"

namespace dcut {

namespace {

constexpr int TK = 64;
constexpr int NSTAGE = 2;     // LDS stages: one k-slice in flight while the other is multiplied

__device__ __forceinline__ uint32_t orderable(float v) {
  uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Workgroup barrier for the LDS ring: each wave has already waited (s_waitcnt
// vmcnt) for its own loads of the stage it is about to read, so no memory fence
// (which would drain every stage still in flight) is needed, only the hardware
// barrier; the empty asm statements keep the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// W row feeding logical tile column group `grp` (global, 32 columns each), plus
// the first output column of that group; returns -1 when the group is past N.
template <int EPI>
__device__ __forceinline__ int group_wrow(const GemmArgs &a, int grp) {
  if (EPI == EPI_SWIGLU) {
    int p = grp >> 1;                       // output block of 32 columns
    if (p * 32 >= a.swiglu_inter) return -1;
    return (grp & 1) ? a.swiglu_inter + p * 32 : p * 32;
  } else if (EPI == EPI_QKV_ROPE) {
    int hd = a.head_dim;
    int gph = hd / 32;                      // groups per head (2 or 4)
    int head = grp / gph, wg = grp - head * gph;
    int base;
    if (gph == 4) {
      const int perm[4] = {0, 64, 32, 96};
      base = perm[wg];
    } else {
      base = wg * 32;
    }
    int row = head * hd + base;
    return row < a.N ? row : -1;
  } else {
    int row = grp * 32;
    return row < a.N ? row : -1;
  }
}

template <int EPI, int WM, int WN>
__global__ void __launch_bounds__(256)
k_gemm(GemmArgs a) {
  constexpr int GM = 2, GN = 2, NWV = GM * GN;
  constexpr int TM = GM * WM * 32, TN = GN * WN * 32;
  extern __shared__ __align__(16) uint16_t lds[];   // [NSTAGE][TM*TK (A) + TN*TK (B)]

  int M = *a.m_count;
  const int nMT = a.m_tiles > 0 ? a.m_tiles : (a.M_max + TM - 1) / TM;
  const int total = gridDim.x;
  const int per = total >> 3;
  const int w = blockIdx.x;
  const int id = (w < per * 8) ? (w & 7) * per + (w >> 3) : w;
  const int mt = id % nMT, nt = id / nMT;
  int m0 = mt * TM;
  const uint16_t *Wb = a.W;
  if (a.tiles) {
    if (mt >= *a.n_tiles) return;
    const int e = a.tiles[3 * mt];
    m0 = a.tiles[3 * mt + 1];
    M = a.tiles[3 * mt + 2];
    Wb += (size_t)e * a.w_stride;
  }
  if (m0 >= M) return;
  const int grp0 = nt * (TN / 32);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / GN, wn = wave % GN;

  // Operand loads go straight from memory to LDS (buffer_load ... lds): each
  // wave instruction fills one 1 KB block = 8 rows x 64 k (128 B per row).
  // Block q holds rows 8q..8q+7; in row r the 16-byte chunk c holds global k
  // chunk c ^ (r & 7), so the MFMA fragment reads of 32 consecutive rows spread
  // over all LDS banks.  Out-of-range rows and k chunks get an offset past the
  // buffer end and read as zeros.
  const int a_rows_ext = a.a_extent > 0 ? a.a_extent : a.M_max;
  const long long a_bytes = (long long)a_rows_ext * a.lda * 2;
  const int w_rows_ext = (EPI == EPI_SWIGLU) ? 2 * a.swiglu_inter : a.N;
  const long long w_bytes = (long long)w_rows_ext * a.ldw * 2;
  const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.A, (short)0, (int)(a_bytes < 0x7fffffffLL ? a_bytes : 0x7fffffffLL), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsW = __builtin_amdgcn_make_buffer_rsrc(
      (void *)Wb, (short)0, (int)(w_bytes < 0x7fffffffLL ? w_bytes : 0x7fffffffLL), 0x00020000);
  constexpr unsigned OOB = 0x80000000u;
  constexpr int CPR = TK / 8, RPI = 64 / CPR;   // 16-byte chunks per row, rows per 1 KB wave load
  constexpr int AJ = TM / (NWV * RPI), BJ = TN / (NWV * RPI);     // load instructions per wave per stage
  const int lr = lane / CPR, lc = lane % CPR;
  unsigned aoff[AJ], boff[BJ];
  int akc[AJ], bkc[BJ];
#pragma unroll
  for (int j = 0; j < AJ; ++j) {
    const int r = RPI * (wave + NWV * j) + lr;
    akc[j] = 8 * (lc ^ (r % CPR));                 // first k of the chunk this lane fetches
    const int gm = m0 + r;
    unsigned off = OOB;
    if (gm < M) {
      const int src = a.a_rows ? a.a_rows[gm] : gm;
      off = (unsigned)(((long long)src * a.lda + akc[j]) * 2);
    }
    aoff[j] = off;
  }
#pragma unroll
  for (int j = 0; j < BJ; ++j) {
    const int r = RPI * (wave + NWV * j) + lr;
    bkc[j] = 8 * (lc ^ (r % CPR));
    const int grp = grp0 + (r >> 5);
    const int wr = group_wrow<EPI>(a, grp);
    bool ok = wr >= 0;
    if (EPI == EPI_SWIGLU) ok = ok && ((grp >> 1) * 32 + (r & 31)) < a.swiglu_inter;
    else ok = ok && wr + (r & 31) < a.N;
    boff[j] = ok ? (unsigned)(((long long)(wr + (r & 31)) * a.ldw + bkc[j]) * 2) : OOB;
  }
  constexpr int STAGE = (TM + TN) * TK;            // bf16 elements per stage
  auto issue = [&](int kt, int slot) {
    const int k0 = kt * TK;
    uint16_t *sa = lds + slot * STAGE;
    uint16_t *sb = sa + TM * TK;
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
      const unsigned off = (aoff[j] != OOB && k0 + akc[j] < a.K) ? aoff[j] + (unsigned)k0 * 2 : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (__attribute__((address_space(3))) void *)(sa + (wave + NWV * j) * 512),
                                               16, off, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const unsigned off = (boff[j] != OOB && k0 + bkc[j] < a.K) ? boff[j] + (unsigned)k0 * 2 : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (__attribute__((address_space(3))) void *)(sb + (wave + NWV * j) * 512),
                                               16, off, 0, 0, 0);
    }
  };

  floatx16 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int l32 = lane & 31, kh = lane >> 5;
  // fragment read offsets within a stage (row r: block r>>3, row r&7, chunk swizzled by r&7)
  int afrag[WM], bfrag[WN], arx[WM], brx[WN];
#pragma unroll
  for (int i = 0; i < WM; ++i) {
    const int r = wm * WM * 32 + i * 32 + l32;
    afrag[i] = r * TK;
    arx[i] = r % CPR;
  }
#pragma unroll
  for (int j = 0; j < WN; ++j) {
    const int r = wn * WN * 32 + j * 32 + l32;
    bfrag[j] = TM * TK + r * TK;
    brx[j] = r % CPR;
  }

  // this workgroup's k range (split-K over gridDim.y, fixed by the shape)
  const int nk_all = (a.K + TK - 1) / TK;
  const int per_split = (nk_all + (int)gridDim.y - 1) / (int)gridDim.y;
  const int kt0 = (int)blockIdx.y * per_split;
  const int nk = max(0, min(nk_all, kt0 + per_split) - kt0);
  // s_waitcnt immediates waiting for all but 0, 1 or 2 stages of AJ+BJ loads
  constexpr int LPS = AJ + BJ;
  constexpr int W0 = 0 | (7 << 4) | (15 << 8);
  constexpr int W1 = (LPS & 15) | ((LPS >> 4) << 14) | (7 << 4) | (15 << 8);
  constexpr int W2 = ((2 * LPS) & 15) | (((2 * LPS) >> 4) << 14) | (7 << 4) | (15 << 8);
#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < nk) issue(kt0 + s, s);
  for (int it = 0; it < nk; ++it) {
    const int pending = min(NSTAGE - 2, nk - 1 - it);
    if (pending >= 2) __builtin_amdgcn_s_waitcnt(W2);
    else if (pending == 1) __builtin_amdgcn_s_waitcnt(W1);
    else __builtin_amdgcn_s_waitcnt(W0);
    ring_barrier();
    if (it + NSTAGE - 1 < nk) issue(kt0 + it + NSTAGE - 1, (it + NSTAGE - 1) % NSTAGE);
    const uint16_t *st = lds + (it % NSTAGE) * STAGE;
#pragma unroll
    for (int ks = 0; ks < TK / 16; ++ks) {
      const int kc = 2 * ks + kh;
      bf16x8 af[WM], bf[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) af[i] = *(const bf16x8 *)(st + afrag[i] + 8 * (kc ^ arx[i]));
#pragma unroll
      for (int j = 0; j < WN; ++j) bf[j] = *(const bf16x8 *)(st + bfrag[j] + 8 * (kc ^ brx[j]));
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  }

  if (gridDim.y > 1) {
    // split-K partial tile; k_splitk_reduce applies the epilogue in split order
    float *part = a.split_part + (size_t)blockIdx.y * a.M_max * a.N;
    const int rb_ = m0 + wm * WM * 32 + 4 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        int col = (grp0 + wn * WN + j) * 32 + l32;
        if (col >= a.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int gm = rb_ + i * 32 + 8 * (r >> 2) + (r & 3);
          if (gm < M) part[(size_t)gm * a.N + col] = acc[i][j][r];
        }
      }
    return;
  }

  // ------------------------------------------------------------ epilogues
  // accumulator element r of a 32x32 tile: row 8*(r/4) + 4*(lane/32) + r%4, column lane%32
  const int rbase = m0 + wm * WM * 32 + 4 * (lane >> 5);
  if (EPI == EPI_STORE_BF16 || EPI == EPI_RESID_F32 || EPI == EPI_STORE_F32) {
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        int wr = group_wrow<EPI>(a, grp0 + wn * WN + j);
        if (wr < 0) continue;
        int col = wr + l32;
        if (col >= a.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int gm = rbase + i * 32 + 8 * (r >> 2) + (r & 3);
          if (gm >= M) continue;
          if (EPI == EPI_STORE_BF16) a.out_bf16[(size_t)gm * a.ldo + col] = f2bf(acc[i][j][r]);
          else if (EPI == EPI_STORE_F32) a.out_f32[(size_t)gm * a.ldo + col] = acc[i][j][r];
          else {
            float *o = a.out_f32 + (size_t)gm * a.ldo + col;
            *o = *o + acc[i][j][r];
          }
        }
      }
  } else if (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int p = 0; p < WN / 2; ++p) {
        int ob = ((grp0 + wn * WN + 2 * p) >> 1) * 32;
        int col = ob + l32;
        if (col >= a.swiglu_inter) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int gm = rbase + i * 32 + 8 * (r >> 2) + (r & 3);
          if (gm >= M) continue;
          float g = acc[i][2 * p][r], u = acc[i][2 * p + 1][r];
          a.out_bf16[(size_t)gm * a.ldo + col] = f2bf(silu(g) * u);
        }
      }
  } else if (EPI == EPI_QKV_ROPE) {
    const int hd = a.head_dim, half = hd >> 1, gph = hd / 32;
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int p = 0; p < WN / 2; ++p) {
        int grp = grp0 + wn * WN + 2 * p;
        int head = grp / gph;
        if (head >= a.n_q + 2 * a.n_kv) continue;
        int wr = group_wrow<EPI>(a, grp);
        int j = wr - head * hd + l32;       // dimension in the first half, < hd/2
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int gm = rbase + i * 32 + 8 * (r >> 2) + (r & 3);
          if (gm >= M) continue;
          float x1 = acc[i][2 * p][r], x2 = acc[i][2 * p + 1][r];
          float o1 = x1, o2 = x2;
          if (head < a.n_q + a.n_kv) {
            float2 cs = a.rope_cs[(size_t)gm * half + j];
            o1 = x1 * cs.x - x2 * cs.y;
            o2 = x2 * cs.x + x1 * cs.y;
          }
          if (head < a.n_q) {
            uint16_t *q = a.out_bf16 + (size_t)gm * a.ldo + head * hd;
            q[j] = f2bf(o1);
            q[j + half] = f2bf(o2);
          } else {
            int req = a.packed_req[gm];
            int slot = a.packed_pos[gm];
            int cap = a.kv_cap[req];
            if (slot < 0 || slot >= cap) continue;      // reported by the norm kernel
            int g = (head < a.n_q + a.n_kv) ? head - a.n_q : head - a.n_q - a.n_kv;
            uint16_t *dst = (head < a.n_q + a.n_kv ? a.kv_k : a.kv_v) + a.kv_base[req] +
                            ((size_t)g * cap + slot) * hd;
            dst[j] = f2bf(o1);
            dst[j + half] = f2bf(o2);
          }
        }
      }
  } else if (EPI == EPI_ARGMAX) {
#pragma unroll
    for (int i = 0; i < WM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int gm = rbase + i * 32 + 8 * (r >> 2) + (r & 3);
        unsigned long long best = 0ull;
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          int col = (grp0 + wn * WN + j) * 32 + l32;
          if (col < a.N) {
            float v = acc[i][j][r];
            unsigned long long key = ((unsigned long long)orderable(v) << 32) | (0xffffffffu - (uint32_t)col);
            best = key > best ? key : best;
            if (a.logits && gm < M) a.logits[(size_t)gm * a.ld_logits + col] = v;
          }
        }
#pragma unroll
        for (int off = 1; off < 32; off <<= 1) {
          unsigned long long o = __shfl_xor(best, off, 64);
          best = o > best ? o : best;
        }
        if (l32 == 0 && gm < M && best) atomicMax(a.amax_keys + gm, best);
      }
    }
  }
}

// out[m][n] (+)= sum over splits of part[s][m][n], in split order (rows m < K*).
__global__ void __launch_bounds__(256)
k_splitk_reduce(const float *__restrict__ part, int splits, int M_max, int N,
                const int32_t *__restrict__ m_count, float *__restrict__ out, int ldo, int accumulate) {
  const int m = blockIdx.y;
  if (m >= *m_count) return;
  const int n = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (n >= N) return;
  float4 acc = *(const float4 *)(part + (size_t)m * N + n);
  for (int s = 1; s < splits; ++s) {
    float4 v = *(const float4 *)(part + ((size_t)s * M_max + m) * N + n);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  float4 *o = (float4 *)(out + (size_t)m * ldo + n);
  if (accumulate) {
    float4 x = *o;
    acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
  }
  *o = acc;
}

template <int EPI, int WM, int WN>
int launch_tile(int kid, const GemmArgs &a, hipStream_t s) {
  constexpr int TM = 2 * WM * 32, TN = 2 * WN * 32;
  int ncols = (EPI == EPI_SWIGLU) ? 2 * a.swiglu_inter : a.N;
  int nMT = a.m_tiles > 0 ? a.m_tiles : (a.M_max + TM - 1) / TM;
  int nNT = (EPI == EPI_SWIGLU) ? (a.swiglu_inter + TN / 2 - 1) / (TN / 2) : (ncols + TN - 1) / TN;
  size_t shmem = (size_t)NSTAGE * (TM + TN) * TK * sizeof(uint16_t);
  const int splits = a.splits > 1 ? a.splits : 1;
  if (splits > 1) {
    if ((EPI != EPI_RESID_F32 && EPI != EPI_STORE_F32) || a.tiles || !a.split_part || a.N % 4 || a.ldo % 4)
      return DCUT_EINVAL;
    DCUT_TRY(launch(kid, k_gemm<EPI, WM, WN>, dim3(nMT * nNT, splits), dim3(256), shmem, s, a));
    return launch(DCUT_KERNEL_NONE, k_splitk_reduce, dim3((a.N + 1023) / 1024, a.M_max), dim3(256), 0, s,
                  (const float *)a.split_part, splits, a.M_max, a.N, a.m_count, a.out_f32, a.ldo,
                  EPI == EPI_RESID_F32 ? 1 : 0);
  }
  return launch(kid, k_gemm<EPI, WM, WN>, dim3(nMT * nNT), dim3(256), shmem, s, a);
}

}  // namespace

int gemm_splits(int M_max, int N, int K) {
  const int nMT = (M_max + 127) / 128, nNT = (N + 127) / 128;
  const int nk = (K + TK - 1) / TK;
  int sp = (1024 + nMT * nNT - 1) / (nMT * nNT);
  const int cap = nk / 8 > 1 ? nk / 8 : 1;      // keep at least 8 k-slices per split
  if (sp > cap) sp = cap;
  if (sp > 16) sp = 16;
  return sp < 1 ? 1 : sp;
}

int gemm_launch(int kid, EpiKind epi, const GemmArgs &a, hipStream_t s) {
  switch (epi) {
    case EPI_STORE_BF16: return launch_tile<EPI_STORE_BF16, 2, 2>(kid, a, s);
    case EPI_RESID_F32: return launch_tile<EPI_RESID_F32, 2, 2>(kid, a, s);
    case EPI_SWIGLU: return launch_tile<EPI_SWIGLU, 2, 2>(kid, a, s);
    case EPI_QKV_ROPE: return launch_tile<EPI_QKV_ROPE, 2, 2>(kid, a, s);
    case EPI_ARGMAX: return launch_tile<EPI_ARGMAX, 2, 2>(kid, a, s);
    case EPI_STORE_F32: return launch_tile<EPI_STORE_F32, 2, 2>(kid, a, s);
  }
  return DCUT_EINVAL;
}

}  // namespace dcut
