// bf16 NT GEMM on gfx950 MFMA with fused epilogues: C = A W^T, A [M][K], W [N][K].
//
// Two tile shapes share one kernel template (32x32x16 bf16 MFMA, float32
// accumulators, k-slices of 64):
//   Big   256 x 256, eight waves in a 4 x 2 grid, each wave 64 x 128;
//         160 KB of LDS, one workgroup per CU (dense GEMMs with many tiles);
//   Small 128 x 128, four waves in a 2 x 2 grid, each wave 64 x 64;
//         80 KB of LDS, two workgroups per CU (grouped MoE GEMMs, split-K).
// Operands stream from memory straight into LDS (buffer loads with the LDS
// destination, 128-byte rows of 64 k split in XOR-swizzled 16-byte chunks,
// hardware zeros for rows and k beyond the operands).  A and W have rings of
// their own: A (activations, mostly L2-resident) two stages, W (weights,
// streamed from HBM) three stages, so a W slice is requested two k-steps before
// it is multiplied.  Fragment reads of the next 16-k step are issued before the
// MFMAs of the current one.
//
// Scheduling: the grid is persistent (at most one wave of workgroups); every
// workgroup reads the live row count M (K*) on the device and walks only the
// tiles that exist, so rows beyond K* cost nothing.  Tasks (row tile, column
// tile, k split) are numbered with the row tile fastest and the split slowest
// and cut into eight contiguous ranges, one per XCD (the hardware deals
// workgroups round-robin over the eight XCDs): row tiles sharing a W slice run
// at the same time on the same L2, and an XCD reads the A columns of one or
// two splits only, not all of A.
//
// Determinism and causality: every output element is the same sequence of
// MFMA k-steps from k = 0 upwards whatever the tile shape; split-K partials are
// added in split order; the tile shape and split factor depend on M_max (the
// grid's row bound), never on M.  A row's bits therefore do not depend on which
// or how many other rows are present.
//
// Column groups: each 32-column MFMA tile loads a 32-row group of W chosen by
// the epilogue, so that values an epilogue combines sit in the same lane:
//   SWIGLU    groups (2p, 2p+1) = (gate rows, up rows) of the same 32 outputs;
//   QKV_ROPE  groups (2p, 2p+1) = the two halves (j, j + hd/2) of RoPE pairs.

#include <atomic>
#include <type_traits>

#include "dcut_internal.h"
#include "rng.h"

namespace dcut {

namespace {

constexpr int TK = 64;       // k per LDS stage: one 128-byte row per operand row
constexpr int CPR = TK / 8;  // 16-byte chunks per row
constexpr int RPI = 64 / CPR;  // rows per 1 KB wave load

template <int GM_, int GN_, int WM_, int WN_, int NA_ = 2, int NB_ = 3, bool SKEW_ = false>
struct Tile {
  static constexpr int GM = GM_, GN = GN_, WM = WM_, WN = WN_;
  static constexpr bool SKEW = SKEW_;   // second half of the waves two sub-steps behind (8-wave tiles)
  static constexpr int NWV = GM * GN, THREADS = 64 * NWV;
  static constexpr int TM = GM * WM * 32, TN = GN * WN * 32;
  // ring stages of A and W: slice it + NA - 1 of A and it + NB - 1 of W are
  // requested while slice it is multiplied
  static constexpr int NA = NA_, NB = NB_;
  static_assert(NA >= 2 && NB >= 2, "double buffering at least");
  static constexpr size_t LDS = (size_t)(NA * TM + NB * TN) * TK * sizeof(uint16_t);
  static_assert(LDS <= 163840, "the LDS of one CU");
  static constexpr int PER_CU = LDS > 81920 ? 1 : 2;
};
using Big = Tile<4, 2, 2, 4, 2, 3, true>;
using Mid = Tile<2, 4, 2, 2, 2, 3, true>;     // 128 x 256, eight waves in a 2 x 4 grid, 128 KB
using Small = Tile<2, 2, 2, 2>;
using MidDeep = Tile<2, 4, 2, 2, 2, 4, true>;   // 128 x 256 with four W slices: the LM head at few live rows
using BigFlat = Tile<4, 2, 2, 4>;   // Big without the skew: the sampling epilogue needs its registers

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// LDS chunk swizzle of row r: 16 consecutive rows of one chunk column land in
// 16 different 16-byte bank groups, and so do any 8 consecutive rows.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & (CPR - 1); }

// Workgroup barrier for the LDS rings: each wave has already waited (s_waitcnt
// vmcnt) for its own loads of the stage it is about to read, so no memory fence
// (which would drain every stage still in flight) is needed, only the hardware
// barrier; the empty asm statements keep the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt immediate: at most N vector-memory operations outstanding
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// s_waitcnt with the largest immediate in [LO, HI] that is at most n (n >= LO):
// a binary search over immediates, since vmcnt cannot come from a register.
template <int LO, int HI>
__device__ __forceinline__ void wait_vm_le(int n) {
  if constexpr (LO == HI) {
    wait_vm<LO>();
  } else {
    constexpr int MID = (LO + HI + 1) / 2;
    if (n >= MID) wait_vm_le<MID, HI>(n);
    else wait_vm_le<LO, MID - 1>(n);
  }
}

// Vector-memory loads that may still be outstanding when iteration `it` of a
// k loop of nk slices needs its A and W slices.  Issue order: prologue groups
// j = 0 .. P-1 (A[j] if j < PA, then W[j] if j < PW), then one group per
// iteration i (A[i + PA], then W[i + PW]); slices at or past nk are never
// issued; AJ and BJ are the load instructions of one A and one W slice.  The
// loads issued after the later of A[it] and W[it] may be outstanding.
template <int PA, int PW, int AJ, int BJ>
__device__ __forceinline__ int loads_after(int it, int nk) {
  constexpr int P = PA > PW ? PA : PW;
  const int gA = it < PA ? it : P + it - PA;
  const int gW = it < PW ? it : P + it - PW;
  const bool last_is_a = gA > gW;          // in a shared group W follows A
  const int g = last_is_a ? gA : gW;
  auto has_a = [&](int q) { return q < P ? (q < PA && q < nk) : (q - P + PA < nk); };
  auto has_w = [&](int q) { return q < P ? (q < PW && q < nk) : (q - P + PW < nk); };
  int n = (last_is_a && has_w(g)) ? BJ : 0;
#pragma unroll
  for (int d = 1; d <= P; ++d) {
    const int q = g + d;
    if (q < P + it) n += (has_a(q) ? AJ : 0) + (has_w(q) ? BJ : 0);
  }
  return n;
}

// W row feeding logical tile column group `grp` (global, 32 columns each);
// -1 when the group is past N.
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

template <int EPI>
__device__ __forceinline__ int n_col_tiles(const GemmArgs &a, int TN) {
  return EPI == EPI_SWIGLU ? (a.swiglu_inter + TN / 2 - 1) / (TN / 2) : (a.N + TN - 1) / TN;
}

// QKV epilogue for one RoPE pair of one row: x1, x2 = projections at head
// dimensions j and j + hd/2.  q and k heads are rotated; q goes to out_bf16, k
// and v to the request's cache slot (slots outside the cache are skipped; the
// norm kernel reports them).
__device__ __forceinline__ void qkv_emit(const GemmArgs &a, int gm, int head, int j, float x1, float x2) {
  const int hd = a.head_dim, half = hd >> 1;
  float o1 = x1, o2 = x2;
  if (head < a.n_q + a.n_kv) {
    const float2 r = rope_pair(x1, x2, a.rope_cs[(size_t)gm * half + j]);
    o1 = r.x;
    o2 = r.y;
  }
  if (head < a.n_q) {
    uint16_t *q = a.out_bf16 + (size_t)gm * a.ldo + head * hd;
    q[j] = f2bf(o1);
    q[j + half] = f2bf(o2);
  } else {
    const int req = a.packed_req[gm];
    if ((unsigned)req >= (unsigned)a.n_req) return;   // not a row of this batch
    const int slot = a.packed_pos[gm];
    const int cap = a.kv_cap[req];
    if (slot < 0 || slot >= cap) return;
    const int g = (head < a.n_q + a.n_kv) ? head - a.n_q : head - a.n_q - a.n_kv;
    uint16_t *dst = (head < a.n_q + a.n_kv ? a.kv_k : a.kv_v) + a.kv_base[req] + ((size_t)g * cap + slot) * hd;
    dst[j] = f2bf(o1);
    dst[j + half] = f2bf(o2);
  }
}

template <int EPI, class T>
__device__ __forceinline__ void gemm_tasks(const GemmArgs &a) {
  constexpr int GN = T::GN, WM = T::WM, WN = T::WN, NWV = T::NWV;
  constexpr int TM = T::TM, TN = T::TN, NA = T::NA, NB = T::NB;
  constexpr int AJ = TM / (NWV * RPI), BJ = TN / (NWV * RPI);   // load instructions per wave per stage
  static_assert(AJ * NWV * RPI == TM && BJ * NWV * RPI == TN, "tile rows must fill whole wave loads");
  extern __shared__ __align__(16) uint16_t lds[];   // [NA][TM*TK] (A), then [NB][TN*TK] (W)
  uint16_t *const ldsA = lds;
  uint16_t *const ldsW = lds + NA * TM * TK;

  // the wave index is uniform: kept in a scalar register, so LDS destinations
  // of the operand loads are scalar arithmetic
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / GN, wn = wave % GN;
  const int l32 = lane & 31, kh = lane >> 5;
  const int lr = lane / CPR, lc = lane % CPR;

  // live tasks: (row tile, column tile, split), row tile fastest, split slowest
  const int M = min(*a.m_count, a.M_max);
  const int nMT = a.tiles ? *a.n_tiles : (M + TM - 1) / TM;
  const int nNT = n_col_tiles<EPI>(a, TN);
  const int splits = a.splits > 1 ? a.splits : 1;
  const int ntask = nMT * nNT * splits;
  const int xcd = blockIdx.x & 7, per_xcd = gridDim.x >> 3;
  const int lo = (int)((long long)ntask * xcd / 8), hi = (int)((long long)ntask * (xcd + 1) / 8);

  const int nk_all = (a.K + TK - 1) / TK;
  const int per_split = (nk_all + splits - 1) / splits;
  // Buffer resources take 32-bit offsets: each task addresses A from its first
  // row (or, for gathered rows, from the start of A) and W from the first
  // weight row of its column tile, so the offsets stay below 2^31 for any
  // operand size the host checks admit (gemm_span_ok).
  const int a_rows_ext = a.a_extent > 0 ? a.a_extent : a.M_max;
  const int w_rows_ext = (EPI == EPI_SWIGLU) ? 2 * a.swiglu_inter : a.N;
  constexpr unsigned OOB = 0x80000000u;
  auto rsrc = [](const uint16_t *base, long long bytes) {
    return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0,
                                             (int)(bytes < 0x7fffffffLL ? bytes : 0x7fffffffLL), 0x00020000);
  };

  // fragment read offsets within a stage (row r at r*TK, chunk swizzled)
  int afrag[WM], bfrag[WN], arx[WM], brx[WN];
#pragma unroll
  for (int i = 0; i < WM; ++i) {
    const int r = wm * WM * 32 + i * 32 + l32;
    afrag[i] = r * TK;
    arx[i] = swz(r);
  }
#pragma unroll
  for (int j = 0; j < WN; ++j) {
    const int r = wn * WN * 32 + j * 32 + l32;
    bfrag[j] = r * TK;
    brx[j] = swz(r);
  }

  for (int task = lo + (int)(blockIdx.x >> 3); task < hi; task += per_xcd) {
    const int mt = task % nMT;
    const int rest = task / nMT;
    const int nt = rest % nNT, sp = rest / nNT;
    int m0 = mt * TM, Mlim = M;
    const uint16_t *Wb = a.W;
    if (a.tiles) {
      const int e = a.tiles[3 * mt];
      m0 = a.tiles[3 * mt + 1];
      Mlim = a.tiles[3 * mt + 2];
      Wb += (size_t)e * a.w_stride;
    }
    const int grp0 = nt * (TN / 32);
    // the lowest W row of the tile: its first column group (gate rows precede
    // up rows; a head's first group is its first 32 dimensions)
    const int wrow0 = max(group_wrow<EPI>(a, grp0), 0);
    const __amdgpu_buffer_rsrc_t rsW = rsrc(Wb + (size_t)wrow0 * a.ldw, (long long)(w_rows_ext - wrow0) * a.ldw * 2);
    const int arow0 = a.a_rows ? 0 : m0;
    const __amdgpu_buffer_rsrc_t rsA = rsrc(a.A + (size_t)arow0 * a.lda, (long long)(a_rows_ext - arow0) * a.lda * 2);

    // Each wave load instruction fills one 1 KB block = 8 rows x 64 k; row r's
    // 16-byte chunk c holds global chunk c ^ swz(r).  Rows past the operand and
    // k past K get an offset beyond the buffer, which reads as zeros.
    unsigned aoff[AJ], boff[BJ];
    // k chunk (elements) that load j of this lane fetches within a 64-k slice
    auto kchunk = [&](int j) { return 8 * (lc ^ swz(RPI * (wave + NWV * j) + lr)); };
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
      const int r = RPI * (wave + NWV * j) + lr;
      const int gm = m0 + r;
      unsigned off = OOB;
      if (gm < Mlim) {
        const int src = a.a_rows ? a.a_rows[gm] : gm;
        off = (unsigned)(((long long)(src - arow0) * a.lda + kchunk(j)) * 2);
      }
      aoff[j] = off;
    }
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int r = RPI * (wave + NWV * j) + lr;
      const int grp = grp0 + (r >> 5);
      const int wr = group_wrow<EPI>(a, grp);
      bool ok = wr >= 0;
      if (EPI == EPI_SWIGLU) ok = ok && ((grp >> 1) * 32 + (r & 31)) < a.swiglu_inter;
      else ok = ok && wr + (r & 31) < a.N;
      boff[j] = ok ? (unsigned)(((long long)(wr + (r & 31) - wrow0) * a.ldw + kchunk(j)) * 2) : OOB;
    }
    // The k offset of a slice goes in the scalar offset; the per-lane offsets
    // stay fixed over the k loop.  Rows past the operand carry OOB, which stays
    // beyond the buffer with any scalar offset added.  Only a slice reaching
    // past K (K not a multiple of TK) masks its chunks beyond K lane by lane.
    auto issueA = [&](int kt, int slot) {
      const int k0 = kt * TK;
      uint16_t *sa = ldsA + slot * (TM * TK);
      const bool tail = k0 + TK > a.K;
#pragma unroll
      for (int j = 0; j < AJ; ++j) {
        const unsigned off = (tail && k0 + kchunk(j) >= a.K) ? OOB : aoff[j];
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (__attribute__((address_space(3))) void *)(sa + (wave + NWV * j) * 512),
                                                 16, off, k0 * 2, 0, 0);
      }
    };
    auto issueW = [&](int kt, int slot) {
      const int k0 = kt * TK;
      uint16_t *sb = ldsW + slot * (TN * TK);
      const bool tail = k0 + TK > a.K;
#pragma unroll
      for (int j = 0; j < BJ; ++j) {
        const unsigned off = (tail && k0 + kchunk(j) >= a.K) ? OOB : boff[j];
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, (__attribute__((address_space(3))) void *)(sb + (wave + NWV * j) * 512),
                                                 16, off, k0 * 2, 0, 0);
      }
    };

    floatx16 acc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int kt0 = sp * per_split;
    const int nk = max(0, min(nk_all, kt0 + per_split) - kt0);
    constexpr int PA = NA - 1, PW = NB - 1;   // slices in flight ahead of the one multiplied
    constexpr int PMAX = PA > PW ? PA : PW;
    static_assert(PMAX * (AJ + BJ) <= 63, "outstanding loads within the vmcnt range");
    // prologue: A[0 .. PA-1] and W[0 .. PW-1], interleaved by slice
#pragma unroll
    for (int j = 0; j < PMAX; ++j) {
      if (j < PA && j < nk) issueA(kt0 + j, j % NA);
      if (j < PW && j < nk) issueW(kt0 + j, j % NB);
    }
    // One 16-k sub-step: the WM x WN MFMAs on the fragments in (fa, fb), each
    // fragment register refilled with sub-step nks of the slice at (na, nb)
    // right after its last use (A fragment i after MFMA (i, WN-1), W fragment
    // j after MFMA (WM-1, j)), so one set of fragment registers serves the
    // pipeline; nks < 0 refills nothing.
    auto substep = [&](bf16x8 (&fa)[WM], bf16x8 (&fb)[WN], const uint16_t *na, const uint16_t *nb, int nks) {
      const int kc = 2 * nks + kh;
#pragma unroll
      for (int i = 0; i < WM; ++i) {
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          if (nks >= 0 && i == WM - 1) {
            fb[j] = *(const bf16x8 *)(nb + bfrag[j] + 8 * (kc ^ brx[j]));
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
        }
        if (nks >= 0) {
          fa[i] = *(const bf16x8 *)(na + afrag[i] + 8 * (kc ^ arx[i]));
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    };
    auto first_frags = [&](const uint16_t *sa, const uint16_t *sb, bf16x8 (&fa)[WM], bf16x8 (&fb)[WN]) {
#pragma unroll
      for (int i = 0; i < WM; ++i) fa[i] = *(const bf16x8 *)(sa + afrag[i] + 8 * (kh ^ arx[i]));
#pragma unroll
      for (int j = 0; j < WN; ++j) fb[j] = *(const bf16x8 *)(sb + bfrag[j] + 8 * (kh ^ brx[j]));
    };
    bf16x8 fa[WM], fb[WN];
    if (T::SKEW && wave >= NWV / 2) {
      // The second half of the waves runs one 16-k sub-step behind the first:
      // at each barrier it holds the last sub-step of the previous slice in
      // registers, so on every SIMD one wave has MFMAs ready while the other
      // waits for its first fragments.  Each accumulator still takes the k
      // sub-steps in order.
      for (int it = 0; it < nk; ++it) {
        wait_vm_le<0, PMAX * (AJ + BJ)>(loads_after<PA, PW, AJ, BJ>(it, nk));
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the previous slice is out of LDS
        ring_barrier();
        const uint16_t *sa = ldsA + (it % NA) * (TM * TK);
        const uint16_t *sb = ldsW + (it % NB) * (TN * TK);
        if (it == 0) first_frags(sa, sb, fa, fb);
        else substep(fa, fb, sa, sb, 0);            // last sub-step of the previous slice
        if (it + PA < nk) issueA(kt0 + it + PA, (it + PA) % NA);
        if (it + PW < nk) issueW(kt0 + it + PW, (it + PW) % NB);
#pragma unroll
        for (int ks = 0; ks < TK / 16 - 1; ++ks) substep(fa, fb, sa, sb, ks + 1);
      }
      if (nk > 0) substep(fa, fb, nullptr, nullptr, -1);
    } else {
      for (int it = 0; it < nk; ++it) {
        // this wave's loads of A[it] and W[it] are done once at most the loads
        // issued after them remain
        wait_vm_le<0, PMAX * (AJ + BJ)>(loads_after<PA, PW, AJ, BJ>(it, nk));
        ring_barrier();
        const uint16_t *sa = ldsA + (it % NA) * (TM * TK);
        const uint16_t *sb = ldsW + (it % NB) * (TN * TK);
        // first 16-k fragments, then the next slices' loads while they are in flight
        first_frags(sa, sb, fa, fb);
        if (it + PA < nk) issueA(kt0 + it + PA, (it + PA) % NA);
        if (it + PW < nk) issueW(kt0 + it + PW, (it + PW) % NB);
#pragma unroll
        for (int ks = 0; ks < TK / 16; ++ks) substep(fa, fb, sa, sb, ks + 1 < TK / 16 ? ks + 1 : -1);
      }
    }
    // every wave is done with the rings before the next task's prologue refills them
    ring_barrier();

    if (splits > 1) {
      // split-K partial tile at the true output columns; the reduce pass adds
      // the splits in order and applies the epilogue
      float *part = a.split_part + (size_t)sp * a.M_max * a.N;
      const int rb_ = m0 + wm * WM * 32 + 4 * (lane >> 5);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int wr = group_wrow<EPI>(a, grp0 + wn * WN + j);
          const int col = wr + l32;
          if (wr < 0 || col >= a.N) continue;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int gm = rb_ + i * 32 + 8 * (r >> 2) + (r & 3);
            if (gm < Mlim) part[(size_t)gm * a.N + col] = acc[i][j][r];
          }
        }
      continue;
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
            if (gm >= Mlim) continue;
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
            if (gm >= Mlim) continue;
            float g = acc[i][2 * p][r], u = acc[i][2 * p + 1][r];
            a.out_bf16[(size_t)gm * a.ldo + col] = f2bf(silu(g) * u);
          }
        }
    } else if (EPI == EPI_QKV_ROPE) {
      const int hd = a.head_dim, gph = hd / 32;
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
            if (gm < Mlim) qkv_emit(a, gm, head, j, acc[i][2 * p][r], acc[i][2 * p + 1][r]);
          }
        }
    } else if constexpr (EPI == EPI_ARGMAX || EPI == EPI_SAMPLE) {
      // One key per row and wave column range (WN * 32 columns), stored and
      // merged by a later pass.  Each lane first takes the maximum over its WN
      // columns; the 32 column keys of each of 32 rows then go through LDS (idle
      // after the k loop) and one lane per row takes their maximum, which avoids
      // a chain of dependent cross-lane shuffles per row.
      constexpr int KS = 33;                        // keys per LDS row, one pad
      static_assert((size_t)NWV * 32 * KS * 8 <= T::LDS, "key transpose fits the rings");
      unsigned long long *kl = (unsigned long long *)lds + (size_t)wave * 32 * KS;
      const int slot = nt * GN + wn;
      const int col0 = (grp0 + wn * WN) * 32 + l32;   // this lane's column in group j: col0 + 32 j
      if (a.logits) {
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int gm = rbase + i * 32 + 8 * (r >> 2) + (r & 3);
            if (gm < Mlim)
#pragma unroll
              for (int j = 0; j < WN; ++j)
                if (col0 + 32 * j < a.N) a.logits[(size_t)gm * a.ld_logits + col0 + 32 * j] = acc[i][j][r];
          }
      }
      // the row blocks go through a compile-time index: a plain loop over them
      // is too large to unroll once sampling is fused in, and a run-time index
      // into acc would move the accumulators to scratch memory
      auto row_block = [&](auto ic) {
        constexpr int i = decltype(ic)::value;
        // branch-free per-lane maximum over the WN columns (increasing with j):
        // a strictly larger order key replaces, so the lowest column wins ties
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float noise[WN];
          if constexpr (EPI == EPI_SAMPLE) {
            // one Philox call per row and lane covers this lane's WN columns:
            // counter (32 (c >> 7) + (c & 31), pos, req, 0), word (c >> 5) & 3
            const int gm = min(rbase + i * 32 + 8 * (r >> 2) + (r & 3), a.M_max - 1);
            const uint4 w = philox4x32_10(make_uint4((uint32_t)(32 * (col0 >> 7) + l32), (uint32_t)a.row_pos[gm],
                                                     (uint32_t)a.row_req[gm], 0u), a.seed_lo, a.seed_hi);
            const int w0 = (col0 >> 5) & 3;
#pragma unroll
            for (int j = 0; j < WN; ++j) {
              const int k = (w0 + j) & 3;     // selects, not an indexed array (which would live in scratch)
              const uint32_t wk = k == 0 ? w.x : k == 1 ? w.y : k == 2 ? w.z : w.w;
              noise[j] = gumbel_of(wk);
            }
          }
          uint32_t bo = 0u, bc = 0xffffffffu;
#pragma unroll
          for (int j = 0; j < WN; ++j) {
            const uint32_t c = (uint32_t)(col0 + 32 * j);
            float v = acc[i][j][r];
            if constexpr (EPI == EPI_SAMPLE) v = v * a.inv_temp + noise[j];
            const uint32_t o = c < (uint32_t)a.N ? order_key(v) : 0u;
            const bool up = o > bo;
            bo = up ? o : bo;
            bc = up ? c : bc;
          }
          const int q = 8 * (r >> 2) + 4 * kh + (r & 3);   // row within these 32
          kl[q * KS + l32] = ((unsigned long long)bo << 32) | (0xffffffffu - bc);
        }
        __builtin_amdgcn_wave_barrier();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (lane < 32) {
          unsigned long long best = 0ull;
#pragma unroll 8
          for (int c = 0; c < 32; ++c) {
            const unsigned long long v = kl[lane * KS + c];
            best = v > best ? v : best;
          }
          const int gm = m0 + wm * WM * 32 + i * 32 + lane;
          if (gm < Mlim) a.amax_keys[(size_t)gm * a.amax_slots + slot] = best;
        }
        __builtin_amdgcn_wave_barrier();
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if constexpr (EPI == EPI_SAMPLE) {
          // the row's log-partition partials over the same column range: each
          // lane's (max, rescaled sum) over its WN columns, merged per row
          // through the same LDS transpose
          if (a.lse_part) {
            float2 *kf = (float2 *)kl;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              float x[WN];
              float m = -__builtin_inff();
#pragma unroll
              for (int j = 0; j < WN; ++j) {
                x[j] = col0 + 32 * j < a.N ? acc[i][j][r] * a.inv_temp : -__builtin_inff();
                m = fmaxf(m, x[j]);
              }
              float sum = 0.0f;
#pragma unroll
              for (int j = 0; j < WN; ++j) sum += __expf(x[j] - m);
              if (m == -__builtin_inff()) sum = 0.0f;
              kf[(8 * (r >> 2) + 4 * kh + (r & 3)) * KS + l32] = make_float2(m, sum);
            }
            __builtin_amdgcn_wave_barrier();
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            if (lane < 32) {
              float m = -__builtin_inff();
#pragma unroll 8
              for (int c = 0; c < 32; ++c) m = fmaxf(m, kf[lane * KS + c].x);
              float sum = 0.0f;
              if (m != -__builtin_inff()) {
#pragma unroll 8
                for (int c = 0; c < 32; ++c) {
                  const float2 v = kf[lane * KS + c];
                  sum += v.y * __expf(v.x - m);
                }
              }
              const int gm = m0 + wm * WM * 32 + i * 32 + lane;
              if (gm < Mlim) a.lse_part[(size_t)gm * a.amax_slots + slot] = make_float2(m, sum);
            }
            __builtin_amdgcn_wave_barrier();
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          }
        }
      };
      static_assert(WM >= 1 && WM <= 4, "row blocks per wave");
      row_block(std::integral_constant<int, 0>{});
      if constexpr (WM > 1) row_block(std::integral_constant<int, 1>{});
      if constexpr (WM > 2) row_block(std::integral_constant<int, 2>{});
      if constexpr (WM > 3) row_block(std::integral_constant<int, 3>{});
      // the next task's prologue refills the LDS this pass used
      ring_barrier();
    }
  }
}

template <int EPI, class T>
__global__ void __launch_bounds__(T::THREADS)
k_gemm(GemmArgs a) {
  gemm_tasks<EPI, T>(a);
}

// Dense GEMM whose tile shape follows the live row count M (read on the device):
// SwiGLU: 128 x 256 tiles when they take fewer rounds of the persistent grid
// than 256 x 256 tiles would (counting a 128-row task as half a 256-row one),
// else 256 x 256.  Argmax LM head: 128 x 256 tiles with four W slices when the
// last 256-row tile would be at most half full.  Every element is the
// same sequence of MFMA k-steps in both shapes, so the choice never changes a
// result bit.
template <int EPI>
__global__ void __launch_bounds__(Big::THREADS)
k_gemm_dual(GemmArgs a) {
  static_assert(Mid::THREADS == Big::THREADS && Mid::LDS <= Big::LDS, "one launch shape for both tiles");
  static_assert(MidDeep::THREADS == Big::THREADS && MidDeep::LDS <= Big::LDS, "one launch shape for both tiles");
  const int M = min(*a.m_count, a.M_max);
  if constexpr (EPI == EPI_SWIGLU) {
    // rounds of the persistent grid: a Mid task is half a Big one
    const long long nct = n_col_tiles<EPI>(a, Big::TN), G = gridDim.x;
    const long long big_rounds = ((M + Big::TM - 1) / Big::TM * nct + G - 1) / G;
    const long long mid_rounds = ((M + Mid::TM - 1) / Mid::TM * nct + G - 1) / G;
    if (mid_rounds < 2 * big_rounds) gemm_tasks<EPI, Mid>(a);
    else gemm_tasks<EPI, Big>(a);
  } else {
    if (lm_head_mid_tile(M)) gemm_tasks<EPI, MidDeep>(a);
    else gemm_tasks<EPI, Big>(a);
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
  float4 *o = (float4 *)(out + (size_t)m * ldo + n);
  const float4 x = accumulate ? *o : make_float4(0.f, 0.f, 0.f, 0.f);
  float4 acc = sum_splits<float4>(splits, [&](int s) {
    return *(const float4 *)(part + ((size_t)s * M_max + m) * N + n);
  });
  if (accumulate) {
    acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
  }
  *o = acc;
}

// QKV split-K epilogue: one thread per (row, head, four consecutive RoPE pairs);
// the partials of dimensions j..j+3 and j+hd/2..j+hd/2+3 added in split order,
// then the QKV epilogue on each pair (the element-wise operations of qkv_emit),
// stored four bf16 at a time.
__global__ void __launch_bounds__(256)
k_qkv_reduce(GemmArgs a) {
  const int m = blockIdx.y;
  if (m >= *a.m_count) return;
  const int hd = a.head_dim, half = hd >> 1, nh = a.n_q + 2 * a.n_kv;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= nh * (half / 4)) return;
  const int head = idx / (half / 4), j = 4 * (idx - head * (half / 4));
  const size_t c1 = (size_t)head * hd + j, c2 = c1 + half;
  const f4x2 x = sum_splits<f4x2>(a.splits, [&](int s) {
    const float *q = a.split_part + ((size_t)s * a.M_max + m) * a.N;
    return f4x2{*(const float4 *)(q + c1), *(const float4 *)(q + c2)};
  });
  float o1[4] = {x.a.x, x.a.y, x.a.z, x.a.w}, o2[4] = {x.b.x, x.b.y, x.b.z, x.b.w};
  if (head < a.n_q + a.n_kv) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float2 r = rope_pair(o1[e], o2[e], a.rope_cs[(size_t)m * half + j + e]);
      o1[e] = r.x;
      o2[e] = r.y;
    }
  }
  uint16_t *dst;
  if (head < a.n_q) {
    dst = a.out_bf16 + (size_t)m * a.ldo + head * hd;
  } else {
    const int req = a.packed_req[m];
    if ((unsigned)req >= (unsigned)a.n_req) return;   // not a row of this batch
    const int slot = a.packed_pos[m];
    const int cap = a.kv_cap[req];
    if (slot < 0 || slot >= cap) return;
    const int g = (head < a.n_q + a.n_kv) ? head - a.n_q : head - a.n_q - a.n_kv;
    dst = (head < a.n_q + a.n_kv ? a.kv_k : a.kv_v) + a.kv_base[req] + ((size_t)g * cap + slot) * hd;
  }
  if (((uintptr_t)(dst + j) & 7) == 0) {
    *(uint2 *)(dst + j) = make_uint2(pack_bf2(o1[0], o1[1]), pack_bf2(o1[2], o1[3]));
    *(uint2 *)(dst + j + half) = make_uint2(pack_bf2(o2[0], o2[1]), pack_bf2(o2[2], o2[3]));
  } else {   // a cache slab base that is not a multiple of four elements
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      dst[j + e] = f2bf(o1[e]);
      dst[j + half + e] = f2bf(o2[e]);
    }
  }
}

// Compute units of the current device, cached per device (atomic: calls from
// several host threads may fill the cache at once, all with the same value).
int cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0, c = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < 64) {
    const int n = cached[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
  }
  if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0) return 256;
  if (dev >= 0 && dev < 64) cached[dev].store(c, std::memory_order_relaxed);
  return c;
}

template <int EPI, class T>
int launch_tile(int kid, const GemmArgs &a, hipStream_t s) {
  const int nMT = a.tiles ? a.m_tiles : (a.M_max + T::TM - 1) / T::TM;
  const int nNT = EPI == EPI_SWIGLU ? (a.swiglu_inter + T::TN / 2 - 1) / (T::TN / 2) : (a.N + T::TN - 1) / T::TN;
  const int splits = a.splits > 1 ? a.splits : 1;
  if ((EPI == EPI_ARGMAX || EPI == EPI_SAMPLE) && (!a.amax_keys || a.amax_slots < nNT * T::GN))
    return DCUT_EINVAL;
  if (EPI == EPI_SAMPLE && (!a.row_req || !a.row_pos || !(a.inv_temp >= 0.0f))) return DCUT_EINVAL;
  if (splits > 1 && ((EPI != EPI_RESID_F32 && EPI != EPI_STORE_F32 && EPI != EPI_QKV_ROPE) || a.tiles ||
                     !a.split_part || a.N % 4 || (EPI != EPI_QKV_ROPE && a.ldo % 4)))
    return DCUT_EINVAL;
  // persistent grid: one wave of workgroups, a multiple of 8 (one share per XCD)
  const long long tasks = (long long)nMT * nNT * splits;
  long long g = (long long)cu_count() * T::PER_CU;
  if (tasks < g) g = tasks;
  g = (g + 7) / 8 * 8;
  if (g < 8) g = 8;
  DCUT_TRY(launch(kid, k_gemm<EPI, T>, dim3((unsigned)g), dim3(T::THREADS), T::LDS, s, a));
  if (splits > 1 && a.defer_reduce) return DCUT_OK;
  if (splits > 1 && EPI == EPI_QKV_ROPE) {
    const int quads = (a.n_q + 2 * a.n_kv) * (a.head_dim / 8);
    return launch(DCUT_KERNEL_NONE, k_qkv_reduce, dim3((quads + 255) / 256, a.M_max), dim3(256), 0, s, a);
  }
  if (splits > 1)
    return launch(DCUT_KERNEL_NONE, k_splitk_reduce, dim3((a.N + 1023) / 1024, a.M_max), dim3(256), 0, s,
                  (const float *)a.split_part, splits, a.M_max, a.N, a.m_count, a.out_f32, a.ldo,
                  EPI == EPI_RESID_F32 ? 1 : 0);
  return DCUT_OK;
}

// Big tiles for dense GEMMs with at least one Big tile per CU at M_max rows
// (the SwiGLU and LM-head GEMMs pick Big or a 128-row tile on the device from
// the live rows); Small
// tiles for the others, for grouped (MoE row tiles of 128) and for split-K
// GEMMs.
template <int EPI>
int launch_epi(int kid, const GemmArgs &a, hipStream_t s) {
  if (a.tiles || a.splits > 1) return launch_tile<EPI, Small>(kid, a, s);
  const long long big_tasks = (long long)((a.M_max + Big::TM - 1) / Big::TM) *
      (EPI == EPI_SWIGLU ? (a.swiglu_inter + Big::TN / 2 - 1) / (Big::TN / 2) : (a.N + Big::TN - 1) / Big::TN);
  if (big_tasks < cu_count()) return launch_tile<EPI, Small>(kid, a, s);
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_ARGMAX) {
    // tile shape chosen on the device from the live row count (one workgroup per CU);
    // the sampling epilogue keeps the 256-row tile (both paths in one kernel would spill)
    if (EPI == EPI_ARGMAX && (!a.amax_keys || a.amax_slots < (a.N + MidDeep::TN - 1) / MidDeep::TN * MidDeep::GN))
      return DCUT_EINVAL;
    const int g = (cu_count() + 7) / 8 * 8;
    return launch(kid, k_gemm_dual<EPI>, dim3((unsigned)g), dim3(Big::THREADS), Big::LDS, s, a);
  } else if constexpr (EPI == EPI_SAMPLE) {
    return launch_tile<EPI, BigFlat>(kid, a, s);
  } else {
    return launch_tile<EPI, Big>(kid, a, s);
  }
}

}  // namespace

int gemm_splits(int M_max, int N, int K) {
  // Split-K tasks are Small tiles (128 x 128) over a k range, at most PER_CU of them per CU, and a
  // split-K GEMM at few live rows runs at the per-CU load rate: its time is that of the busiest
  // CU.  The factor minimises a model of that time summed over a quarter, a half, three quarters
  // and all of M_ref = min(M_max, 1024) live rows (a large batch verifies far fewer than its
  // B(D+1) rows at the budgets a cost row picks): the busiest CU's task count (tasks over CUs,
  // rounded up) times a task's operand bytes, its float32 partial tile and a fixed cost per task
  // (prologue and drain) worth about 150 KB of operand loads.  At least 16 k-slices per split;
  // ties go to fewer splits.  The shapes and the CU count decide it, never the live rows.
  const long long M_ref = M_max < 1024 ? M_max : 1024;
  const long long nNT = (N + Small::TN - 1) / Small::TN, nk = (K + TK - 1) / TK;
  long long cap = nk / 16;
  if (cap > 16) cap = 16;
  if (cap < 1) cap = 1;
  const long long cus = cu_count();
  int best = 1;
  double best_cost = 0.0;
  for (int sp = 1; sp <= cap; ++sp) {
    const long long per = (nk + sp - 1) / sp;
    const double bytes = (double)(Small::TM + Small::TN) * per * TK * 2 +
                         (sp > 1 ? (double)Small::TM * Small::TN * 4 : 0.0) + 150e3;
    double cost = 0.0;
    for (int q = 1; q <= 4; ++q) {
      const long long M = M_ref * q / 4 > 0 ? M_ref * q / 4 : 1;
      const long long tasks = (M + Small::TM - 1) / Small::TM * nNT * sp;
      cost += (double)((tasks + cus - 1) / cus) * bytes;
    }
    if (sp == 1 || cost < best_cost) {
      best = sp;
      best_cost = cost;
    }
  }
  return best;
}

void gemm_argmax_slots(const GemmArgs &a, EpiKind epi, int *big, int *mid) {
  const bool big_tiles = !a.tiles && a.splits <= 1 &&
                         (long long)((a.M_max + Big::TM - 1) / Big::TM) * ((a.N + Big::TN - 1) / Big::TN) >= cu_count();
  if (big_tiles) {
    *big = (a.N + Big::TN - 1) / Big::TN * Big::GN;
    *mid = epi == EPI_ARGMAX ? (a.N + MidDeep::TN - 1) / MidDeep::TN * MidDeep::GN : *big;
  } else {
    *big = *mid = (a.N + Small::TN - 1) / Small::TN * Small::GN;
  }
}

int gemm_launch(int kid, EpiKind epi, const GemmArgs &a, hipStream_t s) {
  switch (epi) {
    case EPI_STORE_BF16: return launch_epi<EPI_STORE_BF16>(kid, a, s);
    case EPI_RESID_F32: return launch_epi<EPI_RESID_F32>(kid, a, s);
    case EPI_SWIGLU: return launch_epi<EPI_SWIGLU>(kid, a, s);
    case EPI_QKV_ROPE: return launch_epi<EPI_QKV_ROPE>(kid, a, s);
    case EPI_ARGMAX: return launch_epi<EPI_ARGMAX>(kid, a, s);
    case EPI_SAMPLE: return launch_epi<EPI_SAMPLE>(kid, a, s);
    case EPI_STORE_F32: return launch_epi<EPI_STORE_F32>(kid, a, s);
  }
  return DCUT_EINVAL;
}

}  // namespace dcut
