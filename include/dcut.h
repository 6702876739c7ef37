/*
 * dcut.h -- C ABI of the D-cut verify-step library for AMD MI355X (gfx950).
 *
 * One speculative decoding step of D-cut (adaptive verification depth pruning
 * for batched speculative decoding) on the target model, in four calls:
 *
 *   dcut_select          cross-request selection and packing   (Sec. 3.2, 3.3; Alg. 1; App. C)
 *   dcut_verify_layer    packed ragged forward of one decoder layer (App. C packing)
 *   dcut_lm_head_argmax  final norm, LM head and greedy argmax of every kept row
 *   dcut_accept          greedy longest-prefix acceptance       (Sec. 3.2; App. A)
 *
 * and, for temperature-T target sampling (Sec. 4, sampling regimes), the
 * drop-in replacement of the third call:
 *
 *   dcut_lm_head_sample  final norm, LM head and a Gumbel-max draw per kept row
 *
 * and, for drafters that expose their proposal distributions and targets that
 * verify by rejection sampling (App. B), replacements of the first and last:
 *
 *   dcut_select_rs       shifted scores with a causal budget choice
 *   dcut_accept_rs       RS acceptance with residual sampling
 *
 * Conventions shared by every call
 *   - All pointers marked "dev" are device pointers on the current HIP device;
 *     "host" pointers are read during the call only.  The caller owns every
 *     buffer; the library never allocates device memory.  Scratch memory comes
 *     from the caller through (ws, ws_bytes); dcut_workspace_bytes() gives the
 *     size.
 *   - Calls are asynchronous on `stream` and never synchronise the host.  No
 *     result depends on an earlier call.  State the library does keep:
 *     dcut_profile_arm sets a per-thread timing hook that later launches from
 *     the same host thread honour until it is disarmed (it records events
 *     only); the host side memoises the device's CU count and, per host thread,
 *     each kernel's dynamic-LDS attribute; dcut_lm_head_argmax_static works in
 *     a static device array of its own (see its declaration).  Argument errors a host can see (sizes, limits, null
 *     pointers, budgets, costs, operand spans) are rejected before any launch
 *     with DCUT_EINVAL or DCUT_EUNSUPPORTED; a failed launch returns DCUT_EHIP.
 *   - Faults in device-resident data never abort: they OR a DCUT_DERR_* bit
 *     into *dev_err (when dev_err is not NULL) and the affected outputs are
 *     unspecified, but every access stays in bounds.
 *   - The chosen budget K* never travels to the host: kernels after dcut_select
 *     are launched for the maximum B(D+1) rows and read K* = cu[B] on the device.
 *   - Matrices follow PyTorch nn.Linear layout [out][in], row-major; bf16 values
 *     are raw bits (dcut_bf16), rounded to nearest-even by the producer.
 *   - Supported sizes: 1 <= B <= 4096, 0 <= D, D + 1 <= 64, B (D + 1) <= 8192.
 */
#ifndef DCUT_H
#define DCUT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif
#pragma GCC visibility push(default)

typedef uint16_t dcut_bf16;

enum {
  DCUT_OK = 0,
  DCUT_EINVAL = -1,        /* invalid argument (size, null pointer, budget, cost)   */
  DCUT_EUNSUPPORTED = -2,  /* valid but outside what the kernels implement          */
  DCUT_EWORKSPACE = -3,    /* ws NULL or ws_bytes below dcut_workspace_bytes()      */
  DCUT_EHIP = -4           /* a HIP launch or runtime call failed                   */
};

/* bits OR-ed into *dev_err by the kernels */
enum {
  DCUT_DERR_CONF = 1,      /* a confidence is NaN, has its sign bit set, or exceeds 1 */
  DCUT_DERR_TOKEN = 2,     /* a token id outside [0, vocab)                           */
  DCUT_DERR_CAPACITY = 4   /* ctx_len < 0 or ctx_len + D + 1 > cap for some request   */
};

enum { DCUT_MAX_BLOCK = 64, DCUT_MAX_BATCH = 4096, DCUT_MAX_ROWS = 8192, DCUT_MAX_CANDIDATES = 64 };

/*
 * dcut_select -- score, rank, choose the budget, keep per-request prefixes, pack.
 *
 * Sec. 3.2 Eq. dcut-prefix-score: s_{i,0} = 1, s_{i,k} = s_{i,k-1} * c_{i,k}
 * (one IEEE float32 multiply per depth, in depth order).  Alg. 1: the B(D+1)
 * positions are ranked by s descending, ties to the smaller depth k, then to
 * the smaller request index i (the order App. B states).  For every candidate
 * budget K_r the benefit is the exact sum of u = trunc(s * 2^40) over the
 * top-K_r positions; Sec. 3.3 Eq. dcut-objective picks r* maximising
 * benefit_r * 2^-40 / costs[r] (float64, one IEEE division; the first strict
 * maximum wins, so equal objectives resolve to the smaller budget).  Request i
 * keeps its depths {0..n_i} = the kept positions (a prefix, App. A) and the
 * kept rows are packed request by request (App. C).
 *
 *   B, D      batch size and drafts per request (block of D+1 positions)
 *   conf      dev  [B][D]   float32  c_{i,1..D} in [0, 1]
 *   draft     dev  [B][D+1] int32    z_{i,0..D}; column 0 is the bonus token
 *   ctx_len   dev  [B]      int32    L_i, tokens already in request i's cache
 *   R         number of candidate budgets, 1..64
 *   budgets   host [R]      int32    non-decreasing, B <= K_r <= B(D+1)
 *                                    (Eq. dcut-budget; see dcut_budgets_from_ratios)
 *   costs     host [R]      double   step cost C_r of budget K_r, finite and > 0
 *   keep_len  dev  [B]      int32    out: n_i + 1
 *   cu        dev  [B+1]    int32    out: exclusive prefix sum of keep_len; cu[B] = K*
 *   packed_tok, packed_pos, packed_req
 *             dev  [B(D+1)] int32    out: row t = cu[i] + k holds z_{i,k}, L_i + k, i;
 *                                    rows >= K* are left unspecified
 *   choice    dev  [2]      int32    out: {K*, r*}
 *   benefit   dev  [R]      uint64   out (nullable): sum of u over the top-K_r positions
 *   dev_err   dev  [1]      int32    nullable; DCUT_DERR_CONF on a bad confidence
 *                                    (the position is then scored as 0)
 * Returns DCUT_OK, DCUT_EINVAL, DCUT_EHIP.
 */
int dcut_select(int B, int D, const float *conf, const int32_t *draft, const int32_t *ctx_len,
                int R, const int32_t *budgets, const double *costs,
                int32_t *keep_len, int32_t *cu, int32_t *packed_tok, int32_t *packed_pos,
                int32_t *packed_req, int32_t *choice, uint64_t *benefit, int32_t *dev_err,
                hipStream_t stream);

/*
 * dcut_select_rs -- RS-safe selection (App. B, causality under rejection sampling).
 *
 * As dcut_select, with two changes that keep whether a position is verified
 * independent of its own proposal:
 *   - positions are ranked by the shifted scores of Eq. dcut-shifted-score,
 *     s~_{i,0} = s~_{i,1} = 1 and s~_{i,k} = s~_{i,k-1} * c_{i,k-1} (float32, in
 *     depth order), with the same ties (smaller depth, then smaller request);
 *   - the budget is chosen causally:
 *     DCUT_RS_SCAN   the early-stopping scan.  Positions are admitted in rank
 *                    order from K = B (every bonus position) while the
 *                    objective strictly rises: K* is the first K >= B with
 *                    J(K+1) <= J(K), or B(D+1).  J(K) = P(K) * 2^-40 / C(K),
 *                    P(K) the exact sum of trunc(s~ * 2^40) over the first K
 *                    ranks, and C(K) the cost table interpolated linearly
 *                    between consecutive budgets (K_r, C_r), flat outside
 *                    [K_0, K_{R-1}], the last of equal budgets holding at K_r:
 *                    C(K) = C_r + ((C_{r+1} - C_r) * (K - K_r)) / (K_{r+1} - K_r),
 *                    float64 in that order.  choice = {K*, the last r with
 *                    K_r <= K*, or -1}.
 *     DCUT_RS_FIXED  a budget fixed before the block was drafted: R must be 1
 *                    and K* = K_0, the global top-K_0 of the shifted scores;
 *                    choice = {K_0, 0}.
 *     DCUT_RS_HISTORY  a budget carried over from the previous step (history-
 *                    based K): K* = k_state[0] clamped to [B, B(D+1)], the
 *                    global top-K* of the shifted scores; then k_state[0]
 *                    becomes the budget the cost model picks for this block
 *                    (the first strict maximum of benefit_r * 2^-40 / costs[r],
 *                    as in dcut_select, on the shifted scores), the next
 *                    step's budget.  choice = {K*, the last r with K_r <= K*,
 *                    or -1}.
 * The paper takes c_{i,k} = q_{i,k}(z_{i,k}), the drafter's probability of its
 * own proposal; causality needs only that c_{i,k} depend on no proposal after
 * z_{i,k}.
 *
 *   mode      DCUT_RS_SCAN, DCUT_RS_FIXED or DCUT_RS_HISTORY
 *   k_state   dev [1] int32, read and written by DCUT_RS_HISTORY (the caller
 *             sets the first step's budget), ignored (may be NULL) otherwise
 *   every other argument as for dcut_select (benefit[r] sums shifted scores)
 * Returns DCUT_OK, DCUT_EINVAL (also for an unknown mode, R != 1 with
 * DCUT_RS_FIXED, or a NULL k_state with DCUT_RS_HISTORY), DCUT_EHIP.
 */
enum { DCUT_RS_SCAN = 0, DCUT_RS_FIXED = 1, DCUT_RS_HISTORY = 2 };
int dcut_select_rs(int B, int D, const float *conf, const int32_t *draft, const int32_t *ctx_len,
                   int mode, int R, const int32_t *budgets, const double *costs, int32_t *k_state,
                   int32_t *keep_len, int32_t *cu, int32_t *packed_tok, int32_t *packed_pos,
                   int32_t *packed_req, int32_t *choice, uint64_t *benefit, int32_t *dev_err,
                   hipStream_t stream);

/* Shape of one decoder layer.  n_exp == 0 selects the dense SwiGLU MLP of width
 * `inter`; n_exp > 0 selects a routed MoE with top_k experts of width exp_inter.
 * max_ctx bounds cap_i for every request (it sizes the attention scratch). */
typedef struct {
  int hidden, n_q, n_kv, head_dim;
  int inter;
  int n_exp, top_k, exp_inter;
  int vocab;
  int max_ctx;
  float rms_eps, rope_theta;
} dcut_layer_cfg;

/* Layer weights (dev, bf16, [out][in]).  embed may be NULL when x_in is given.
 *   w_qkv [(n_q + 2 n_kv) head_dim][hidden]: q heads, then k heads, then v heads
 *   w_o [hidden][n_q head_dim]; w_gate_up [2 inter][hidden]: gate rows then up rows;
 *   w_down [hidden][inter]; MoE: w_router [n_exp][hidden],
 *   w_exp_gate_up [n_exp][2 exp_inter][hidden], w_exp_down [n_exp][hidden][exp_inter]. */
typedef struct {
  const dcut_bf16 *embed, *attn_norm, *w_qkv, *w_o, *mlp_norm, *w_gate_up, *w_down;
  const dcut_bf16 *w_router, *w_exp_gate_up, *w_exp_down;
} dcut_layer_w;

/* Key/value cache: request i owns the slab starting at element base[i] of k and
 * of v, laid out [n_kv][cap_i][head_dim] (keys stored after RoPE).  Slots
 * 0..L_i-1 hold the accepted prefix. */
typedef struct {
  dcut_bf16 *k, *v;
  const int64_t *base;   /* dev [B] */
  const int32_t *cap;    /* dev [B] */
} dcut_kv;

/*
 * dcut_verify_layer -- one pre-norm decoder layer over the K* packed rows.
 *
 * App. C: the kept prefixes form one contiguous batch and every kept position
 * is scored against its request's accepted prefix.  For row t = (i, k):
 *   x = x_in[t] (or embed[packed_tok[t]]); h = RMSNorm(x) * attn_norm;
 *   q, k, v = h W_qkv^T; RoPE (pairs j, j + head_dim/2; angle
 *   packed_pos[t] * rope_theta^(-2j/head_dim)) on q and k; k and v are written
 *   to cache slot L_i + k; attention of head h over slots 0..L_i + k of kv
 *   head h / (n_q / n_kv), scale 1/sqrt(head_dim); y = x + attn W_o^T;
 *   out = y + MLP(RMSNorm(y) * mlp_norm), MLP = SwiGLU, or for MoE the
 *   renormalised top_k mixture of expert SwiGLUs under softmax routing.
 * Row results depend only on the row's own request prefix: they are bitwise
 * identical whatever other rows are kept.
 *
 *   cu, packed_*  from dcut_select (dev); ctx_len dev [B]
 *   x_in    dev [B(D+1)][hidden] float32 residual, or NULL to gather embed rows
 *           (x_in may equal x_out)
 *   kv      cache descriptor (the struct itself is host memory)
 *   x_out   dev [B(D+1)][hidden] float32, out: residual after the layer (rows < K*)
 *   dev_err DCUT_DERR_TOKEN, DCUT_DERR_CAPACITY
 *   ws      dev scratch of dcut_workspace_bytes(1, cfg, B, D) bytes, 256-byte aligned
 * Supported: head_dim in {64, 128}; n_q % n_kv == 0; (n_q / n_kv)(D+1) <= 256;
 * hidden, inter, exp_inter multiples of 8; max_ctx * head_dim * 2 bytes (one
 * request's key or value slab) below 2 GiB; (inter + 256) * hidden * 2 bytes
 * (the weight rows one gate/up tile spans) below 2 GiB.  Weight matrices of any
 * total size are addressed per tile.  cu and packed_* must be what
 * dcut_select wrote (their values are trusted); ctx_len and the cache
 * descriptor are device data checked as above.
 */
int dcut_verify_layer(const dcut_layer_cfg *cfg, const dcut_layer_w *w, int B, int D,
                      const int32_t *cu, const int32_t *packed_tok, const int32_t *packed_pos,
                      const int32_t *packed_req, const int32_t *ctx_len, const float *x_in,
                      const dcut_kv *kv, float *x_out, int32_t *dev_err,
                      void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * dcut_lm_head_argmax -- greedy target token of every kept row.
 *
 * f = RMSNorm(x) * final_norm (eps), logits = f W_lm^T accumulated in float32,
 * argmax = the lowest vocabulary id among the row maxima (greedy target
 * decoding, Sec. 4.1).  Logits are never materialised unless `logits` is given;
 * the workspace holds the normalised rows and up to one partial maximum per row
 * and 64 columns of the vocabulary.
 *
 *   H, V     hidden size and vocabulary
 *   cu       dev [B+1] from dcut_select (K* = cu[B])
 *   x        dev [B(D+1)][H] float32 (rows < K* are read)
 *   w_lm     dev [V][H] bf16
 *   argmax   dev [B(D+1)] int32 out;   max_logit dev [B(D+1)] float32 out (nullable)
 *   logits   dev [B(D+1)][V] float32 out (nullable, for checking only)
 *   ws       dev scratch of dcut_workspace_bytes(2, cfg with hidden = H and vocab = V,
 *            B, D) bytes, 256-byte aligned
 * Supported: H multiple of 8, 512 H bytes (one 256-row tile of W) below 2 GiB;
 * any V (W is addressed per column tile, so weights past 2 GiB are read like
 * any others).  DCUT_EUNSUPPORTED otherwise, before any launch.
 */
int dcut_lm_head_argmax(int H, int V, int B, int D, const int32_t *cu, const float *x,
                        const dcut_bf16 *final_norm, float eps, const dcut_bf16 *w_lm,
                        int32_t *argmax, float *max_logit, float *logits,
                        void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * dcut_lm_head_argmax_static -- dcut_lm_head_argmax without a workspace, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * serving loops that must not call hipMalloc, harnesses that forbid it.
 *
 * Same arguments, kernels and results (bit for bit) as dcut_lm_head_argmax,
 * minus (ws, ws_bytes): the scratch (normalised rows and partial argmax keys)
 * lives in a static device array of dcut_lm_head_static_scratch_bytes()
 * bytes (32 MiB) that every device the library runs on holds until the process
 * ends.  The call allocates nothing and calls no allocating routine; the first
 * call on a device looks up that device's copy of the array.  Every call on one
 * device shares the array: calls that overlap on a device (different streams,
 * different host threads without ordering) race and give unspecified results.
 * Nothing in the array needs clearing between calls (every value read was
 * written by the same call).
 * Returns DCUT_EUNSUPPORTED, before any launch, when the scratch the shape needs,
 * 2 B(D+1) H + 32 B(D+1) ceil(V / 256) bytes (each part rounded up to 256), exceeds
 * the array (the batch-64 step with V = 128256 and H = 4096 needs 23.7 MiB at
 * B(D+1) = 1024); DCUT_EHIP if the array's address cannot be looked up; otherwise
 * as dcut_lm_head_argmax.
 */
int dcut_lm_head_argmax_static(int H, int V, int B, int D, const int32_t *cu, const float *x,
                               const dcut_bf16 *final_norm, float eps, const dcut_bf16 *w_lm,
                               int32_t *argmax, float *max_logit, float *logits, hipStream_t stream);
/* Size in bytes of the static scratch array of dcut_lm_head_argmax_static. */
size_t dcut_lm_head_static_scratch_bytes(void);

/*
 * dcut_lm_head_sample -- target token of every kept row drawn at temperature T.
 *
 * Temperature-T target sampling with target-only verification (Sec. 4,
 * robustness across sampling regimes; App. A, correctness): the token of row t
 * is argmax_c (logits[t][c] / T + G(t, c)), the lowest id among equal scores,
 * which is distributed as softmax(logits[t] / T).  G = -ln(-ln u) is standard
 * Gumbel noise; u comes from Philox4x32-10 (Salmon et al., SC 2011) keyed by
 * `seed` (low 32 bits first):
 *   counter = (32 * (c >> 7) + (c & 31), packed_pos[t], packed_req[t], 0),
 *   u = (word (c >> 5) & 3 of the output + 0.5) / 2^32,
 * so the draw of a (request, position) never depends on what else the batch
 * keeps.  Logits, scaling and noise are float32.  dcut_accept then takes
 * `token` in place of the greedy argmax.
 *
 *   packed_req, packed_pos  dev [B(D+1)] from dcut_select
 *   temperature             > 0 and finite
 *   token     dev [B(D+1)] int32 out;   max_score dev [B(D+1)] float32 out (nullable):
 *             the winning logits / T + G
 *   logits    dev [B(D+1)][V] float32 out (nullable): the raw logits of rows < K*
 *   lse       dev [B(D+1)] float32 out (nullable): ln sum_c exp(logits[t][c] * (1/T)),
 *             the row's log-partition function, from the GEMM's float32
 *             accumulators (dcut_accept_rs takes logits and lse)
 *   other arguments and the workspace as for dcut_lm_head_argmax
 * Errors: DCUT_EINVAL for a null request/position array or a temperature that
 * is not positive and finite, otherwise as dcut_lm_head_argmax.
 */
int dcut_lm_head_sample(int H, int V, int B, int D, const int32_t *cu, const int32_t *packed_req,
                        const int32_t *packed_pos, const float *x, const dcut_bf16 *final_norm,
                        float eps, const dcut_bf16 *w_lm, float temperature, uint64_t seed,
                        int32_t *token, float *max_score, float *logits, float *lse, void *ws,
                        size_t ws_bytes, hipStream_t stream);

/*
 * dcut_accept -- greedy target-only acceptance (Sec. 3.2, App. A).
 *
 * a_i = the largest m <= n_i such that draft[i][j] == argmax[cu[i] + j - 1]
 * for every 1 <= j <= m; next_tok[i] = argmax[cu[i] + a_i];
 * total = sum_i (a_i + 1), the tokens the step commits.
 *
 *   draft dev [B][D+1]; keep_len dev [B]; cu dev [B+1]; argmax dev [B(D+1)]
 *   accept_len dev [B] out; next_tok dev [B] out; total dev [1] out
 *   ctx_len_inout dev [B], nullable: incremented by a_i + 1
 */
int dcut_accept(int B, int D, const int32_t *draft, const int32_t *keep_len, const int32_t *cu,
                const int32_t *argmax, int32_t *accept_len, int32_t *next_tok, int32_t *total,
                int32_t *ctx_len_inout, hipStream_t stream);

/*
 * dcut_accept_rs -- rejection-sampling acceptance (App. B, distributional correctness).
 *
 * Request i verifies its kept drafts in order.  Draft z = draft[i][j] is
 * checked at row r = cu[i] + j - 1 against p_r = softmax(logits[r] / T):
 * accepted when u_r * q[i][j-1][z] < p_r(z) (float64; probability
 * min(1, p/q)), with u_r = (w + 0.5) / 2^32, w word 0 of Philox4x32-10 at
 * counter (0, packed_pos[r], i, 1) under `seed`.  At the first rejection the
 * committed token is argmax_c ln((p_r(c) - q[i][j-1][c])_+) + G(r, c), G the
 * row's Gumbel noise of dcut_lm_head_sample (same seed), or token[r] if no
 * column has p_r(c) > q[i][j-1][c]; when every kept draft is accepted it is
 * token[cu[i] + n_i], the target's own draw.  p in the residual is float32.
 *
 *   V, temperature, seed   as given to dcut_lm_head_sample for the same rows
 *   draft      dev [B][D+1] int32; q dev [B][D][V] float32, q[i][k-1] = the
 *              proposal distribution of z_{i,k}
 *   keep_len, cu, packed_pos  dev, from the selection call
 *   logits     dev [B(D+1)][V] float32, lse dev [B(D+1)] float32, token dev
 *              [B(D+1)] int32: the outputs of dcut_lm_head_sample
 *   accept_len dev [B] out; next_tok dev [B] out; total dev [1] out: sum (a_i + 1)
 *   ctx_len_inout dev [B], nullable: incremented by a_i + 1
 *   ws         dev scratch of dcut_workspace_bytes(4, cfg with vocab = V, B, D)
 *              bytes, 256-byte aligned
 *   dev_err    nullable; DCUT_DERR_TOKEN for a draft outside [0, V), which is
 *              then rejected
 * Only the rows a request consults are read: the rejecting row's logits and
 * q[i][j-1] in full, one column of the others.
 * Returns DCUT_OK, DCUT_EINVAL, DCUT_EWORKSPACE, DCUT_EHIP.
 */
int dcut_accept_rs(int B, int D, int V, float temperature, uint64_t seed, const int32_t *draft,
                   const float *q, const int32_t *keep_len, const int32_t *cu,
                   const int32_t *packed_pos, const float *logits, const float *lse,
                   const int32_t *token, int32_t *accept_len, int32_t *next_tok, int32_t *total,
                   int32_t *ctx_len_inout, void *ws, size_t ws_bytes, int32_t *dev_err,
                   hipStream_t stream);

/* Scratch bytes for call `which` (0 select and select_rs, 1 verify_layer,
 * 2 lm_head_argmax and lm_head_sample, 3 accept, 4 accept_rs, which reads
 * cfg->vocab); cfg may be NULL for 0 and 3.  Returns 0 when none is needed and
 * (size_t)-1 for invalid shapes. */
size_t dcut_workspace_bytes(int which, const dcut_layer_cfg *cfg, int B, int D);

/* Static message for a DCUT_* status. */
const char *dcut_strerror(int status);

/* Host helper for Eq. dcut-budget: out[r] = max(B, ceil(num[r] B (D+1) / den[r]))
 * in exact integer arithmetic, for ratios 0 <= num[r]/den[r] <= 1.  Returns
 * DCUT_OK or DCUT_EINVAL. */
int dcut_budgets_from_ratios(int B, int D, int R, const int32_t *num, const int32_t *den,
                             int32_t *out);

/* Host helper for the cost-table lookup of App. C: index of the captured batch
 * size nearest to B (ties to the larger captured size), or -1 if n < 1. */
int dcut_nearest_batch(int B, int n, const int32_t *captured);

/* Kernel timing hook for profilers.  Arms `kernel` (a DCUT_KERNEL_* id) on the
 * calling thread: its next launches on this thread record `start` before and
 * `stop` after the kernel on the launch stream (an id launched several times
 * per call keeps the last launch).  DCUT_KERNEL_NONE disarms.  This is the
 * library's only state kept between calls: one (kernel, start, stop) triple per
 * host thread, which changes how the armed kernel is launched (with events)
 * but never what it computes.  The events must outlive the armed period.  In a routed-MoE
 * layer the grouped expert GEMMs carry the GEMM_GATE_UP and GEMM_DOWN ids and
 * the router, routing, grouping and combine kernels carry MOE. */
enum {
  DCUT_KERNEL_NONE = 0, DCUT_KERNEL_SELECT /* selection and packing */,
  DCUT_KERNEL_PACK /* no kernel of its own: packing runs in the selection kernel */, DCUT_KERNEL_NORM,
  DCUT_KERNEL_GEMM_QKV, DCUT_KERNEL_ATTN, DCUT_KERNEL_ATTN_COMBINE, DCUT_KERNEL_GEMM_O,
  DCUT_KERNEL_GEMM_GATE_UP, DCUT_KERNEL_GEMM_DOWN, DCUT_KERNEL_MOE, DCUT_KERNEL_LM_HEAD,
  DCUT_KERNEL_ARGMAX_FINAL, DCUT_KERNEL_ACCEPT, DCUT_KERNEL_RS_DECIDE, DCUT_KERNEL_RS_RESIDUAL,
  DCUT_KERNEL_RS_FINISH,
  DCUT_KERNEL_ATTN_PLAN /* no kernel of its own: the attention work order is built by an extra
                           workgroup of the layer's first norm kernel */
};
int dcut_profile_arm(int kernel, hipEvent_t start, hipEvent_t stop);

/* Measurement aid (not a step of the method): streams `bytes` from the dev
 * buffer `src` into LDS the way the GEMM and attention kernels load their
 * operands (buffer loads with the LDS destination, 16 bytes per lane, eight
 * 1 KB loads in flight per wave, non-temporal as the attention's cache
 * stream), and writes nothing.  `workgroups` workgroups
 * of four waves split the buffer into equal contiguous ranges, one per wave.
 * Timing the call on `stream` gives the HBM stream rate attainable through
 * this load path (with at least one workgroup per CU) or one CU's share (with
 * fewer workgroups than CUs); bench.py reports it beside the roofline.
 * Requirements: src 16-byte aligned, 1 <= workgroups <= 65536, bytes a
 * non-zero multiple of workgroups * 4 KB (DCUT_EINVAL otherwise), and at most
 * 2 GiB - 1 KB per wave (DCUT_EUNSUPPORTED otherwise).  The buffer is read
 * only and stays owned by the caller. */
int dcut_stream_probe(const void *src, size_t bytes, int workgroups, hipStream_t stream);

#pragma GCC visibility pop
#ifdef __cplusplus
}
#endif
#endif /* DCUT_H */
