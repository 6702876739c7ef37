// bf16 NT GEMM on gfx950 MFMA with fused epilogues: C = A W^T, A [M][K], W [N][K].
//
// Block tile (GM*WM*32) x (GN*WN*32) x 64 with GM x GN waves; every wave owns
// WM x WN tiles of v_mfma_f32_32x32x16_bf16 (float32 accumulators).  Two
// shapes: 128 x 128 (4 waves of 64 x 64) and, for GEMMs with many column
// tiles, 256 x 256 (8 waves of 128 x 64), which halves the operand traffic
// from L2 per flop.  The choice depends on the shape only, never on K*.
// Operands go global -> registers -> LDS (double buffered, 16-byte padded rows),
// with the next k-slice loaded while the current one is multiplied.  Residual
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
constexpr int LDK = TK + 8;   // 144-byte LDS rows

__device__ __forceinline__ uint32_t orderable(float v) {
  uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }


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

template <int EPI, int GM, int GN, int WM, int WN>
__global__ void __launch_bounds__(GM * GN * 64)
k_gemm(GemmArgs a) {
  constexpr int NTH = GM * GN * 64;
  constexpr int TM = GM * WM * 32, TN = GN * WN * 32;
  extern __shared__ __align__(16) uint16_t lds[];   // [2][TM][LDK] (A) then [2][TN][LDK] (B)

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
  constexpr int ACH = TM * TK / 8 / NTH;    // 16-byte A chunks per thread
  constexpr int BCH = TN * TK / 8 / NTH;
  uint16_t *As = lds;                        // [2][TM][LDK]
  uint16_t *Bs = lds + 2 * TM * LDK;         // [2][TN][LDK]

  // per-thread load descriptors
  const uint16_t *aptr[ACH];
  bool aval[ACH];
  int arow[ACH], acol[ACH];
#pragma unroll
  for (int j = 0; j < ACH; ++j) {
    int c = tid + NTH * j;
    arow[j] = c >> 3;
    acol[j] = (c & 7) * 8;
    int gm = m0 + arow[j];
    aval[j] = gm < M;
    int src = aval[j] ? gm : 0;
    if (a.a_rows && aval[j]) src = a.a_rows[gm];
    aptr[j] = a.A + (size_t)src * a.lda + acol[j];
  }
  const uint16_t *bptr[BCH];
  bool bval[BCH];
  int brow[BCH], bcol[BCH];
#pragma unroll
  for (int j = 0; j < BCH; ++j) {
    int c = tid + NTH * j;
    brow[j] = c >> 3;
    bcol[j] = (c & 7) * 8;
    int wr = group_wrow<EPI>(a, grp0 + (brow[j] >> 5));
    int r = wr + (brow[j] & 31);
    bool ok = wr >= 0;
    if (EPI == EPI_SWIGLU) ok = ok && ((((grp0 + (brow[j] >> 5)) >> 1) * 32 + (brow[j] & 31)) < a.swiglu_inter);
    else ok = ok && r < a.N;
    bval[j] = ok;
    bptr[j] = Wb + (size_t)(ok ? r : 0) * a.ldw + bcol[j];
  }

  // the next k-slice is loaded into registers while the current one is multiplied
  uint4 ra[ACH], rb[BCH];
  auto gload = [&](int kt) {
    const int k0 = kt * TK;
#pragma unroll
    for (int j = 0; j < ACH; ++j) {
      const bool ok = aval[j] && k0 + acol[j] < a.K;
      const uint4 v = *(const uint4 *)(aptr[j] + (ok ? k0 : 0));
      ra[j] = ok ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < BCH; ++j) {
      const bool ok = bval[j] && k0 + bcol[j] < a.K;
      const uint4 v = *(const uint4 *)(bptr[j] + (ok ? k0 : 0));
      rb[j] = ok ? v : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
    uint16_t *as = As + buf * TM * LDK;
    uint16_t *bs = Bs + buf * TN * LDK;
#pragma unroll
    for (int j = 0; j < ACH; ++j) *(uint4 *)(as + arow[j] * LDK + acol[j]) = ra[j];
#pragma unroll
    for (int j = 0; j < BCH; ++j) *(uint4 *)(bs + brow[j] * LDK + bcol[j]) = rb[j];
  };

  floatx16 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int l32 = lane & 31, khalf = (lane >> 5) * 8;
  // this workgroup's k range (split-K over gridDim.y, fixed by the shape)
  const int nk_all = (a.K + TK - 1) / TK;
  const int per_split = (nk_all + (int)gridDim.y - 1) / (int)gridDim.y;
  const int kt0 = (int)blockIdx.y * per_split;
  const int nk = max(0, min(nk_all, kt0 + per_split) - kt0);
  if (nk > 0) {
    gload(kt0);
    lstore(0);
    __syncthreads();
  }
  for (int it = 0; it < nk; ++it) {
    const int buf = it & 1;
    if (it + 1 < nk) gload(kt0 + it + 1);
    const uint16_t *as = As + buf * TM * LDK + (wm * WM * 32 + l32) * LDK + khalf;
    const uint16_t *bs = Bs + buf * TN * LDK + (wn * WN * 32 + l32) * LDK + khalf;
#pragma unroll
    for (int ks = 0; ks < TK / 16; ++ks) {
      bf16x8 af[WM], bf[WN];
#pragma unroll
      for (int i = 0; i < WM; ++i) af[i] = *(const bf16x8 *)(as + i * 32 * LDK + ks * 16);
#pragma unroll
      for (int j = 0; j < WN; ++j) bf[j] = *(const bf16x8 *)(bs + j * 32 * LDK + ks * 16);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (it + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
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

template <int EPI, int GM, int GN, int WM, int WN>
int launch_tile(int kid, const GemmArgs &a, hipStream_t s) {
  constexpr int TM = GM * WM * 32, TN = GN * WN * 32;
  constexpr int NTH = GM * GN * 64;
  int ncols = (EPI == EPI_SWIGLU) ? 2 * a.swiglu_inter : a.N;
  int nMT = a.m_tiles > 0 ? a.m_tiles : (a.M_max + TM - 1) / TM;
  int nNT = (EPI == EPI_SWIGLU) ? (a.swiglu_inter + TN / 2 - 1) / (TN / 2) : (ncols + TN - 1) / TN;
  size_t shmem = (size_t)2 * (TM + TN) * LDK * sizeof(uint16_t);
  const int splits = a.splits > 1 ? a.splits : 1;
  if (splits > 1) {
    if ((EPI != EPI_RESID_F32 && EPI != EPI_STORE_F32) || a.tiles || !a.split_part || a.N % 4 || a.ldo % 4)
      return DCUT_EINVAL;
    DCUT_TRY(launch(kid, k_gemm<EPI, GM, GN, WM, WN>, dim3(nMT * nNT, splits), dim3(NTH), shmem, s, a));
    return launch(DCUT_KERNEL_NONE, k_splitk_reduce, dim3((a.N + 1023) / 1024, a.M_max), dim3(256), 0, s,
                  (const float *)a.split_part, splits, a.M_max, a.N, a.m_count, a.out_f32, a.ldo,
                  EPI == EPI_RESID_F32 ? 1 : 0);
  }
  return launch(kid, k_gemm<EPI, GM, GN, WM, WN>, dim3(nMT * nNT), dim3(NTH), shmem, s, a);
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

// 256 x 256 tiles when they still give at least one workgroup per CU, else 128 x 128.
// Measured on MI355X: with one 8-wave workgroup per CU the 256 x 256 tile exposes
// the global-load latency of every k-slice and runs slower than two 128 x 128
// workgroups per CU, so the large tile is disabled until its loads are pipelined
// deeper.
constexpr bool kBigTiles = false;
static bool use_big_tile(EpiKind epi, const GemmArgs &a) {
  if (!kBigTiles || a.tiles || a.splits > 1) return false;
  const int ncols = epi == EPI_SWIGLU ? 2 * a.swiglu_inter : a.N;
  const long long tiles = (long long)((a.M_max + 255) / 256) * ((ncols + 255) / 256);
  return tiles >= 256;
}

template <int EPI>
static int launch_epi(int kid, const GemmArgs &a, hipStream_t s, bool big) {
  return big ? launch_tile<EPI, 2, 4, 4, 2>(kid, a, s) : launch_tile<EPI, 2, 2, 2, 2>(kid, a, s);
}

int gemm_launch(int kid, EpiKind epi, const GemmArgs &a, hipStream_t s) {
  const bool big = use_big_tile(epi, a);
  switch (epi) {
    case EPI_STORE_BF16: return launch_epi<EPI_STORE_BF16>(kid, a, s, big);
    case EPI_RESID_F32: return launch_epi<EPI_RESID_F32>(kid, a, s, big);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(kid, a, s, big);
    case EPI_QKV_ROPE: return launch_epi<EPI_QKV_ROPE>(kid, a, s, big);
    case EPI_ARGMAX: return launch_epi<EPI_ARGMAX>(kid, a, s, big);
    case EPI_STORE_F32: return launch_epi<EPI_STORE_F32>(kid, a, s, big);
  }
  return DCUT_EINVAL;
}

}  // namespace dcut
