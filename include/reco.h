/*
 * reco.h -- C ABI of the MI355X (gfx950) hot path of reward-coordinated
 * KV-cache compression and decoding.
 *
 * The method (Section 3 of the paper) runs, after every completed reasoning
 * step, a compression of the accumulated KV cache whose size is set by the
 * step's process reward (Section 3.2), and controls the following generation
 * with a reward-banded reflection-token penalty and an answer-perplexity stop
 * rule (Section 3.3).  This library implements the data-parallel kernels of
 * that loop:
 *
 *   reco_score           window attention mass of every cached key   (Eq. 2)
 *   reco_select_compact  keep the top-m keys plus the window, compact
 *                        the K/V rows in place                       (Sec. 3.2)
 *   reco_pool_scores     optional max / mean pooling of the prefix
 *                        scores before selection (policy variant)    (Sec. 1)
 *   reco_decode_attn     GQA decode attention over the ragged,
 *                        compacted cache (optionally appending the
 *                        new token first)                            (Sec. 1, 3.2)
 *   reco_logit_penalty   banded reflection-token logit penalty       (Eq. 3, 4)
 *   reco_penalty_sample  the same penalty, then the next token drawn
 *                        from softmax(z~ / T), one pass per row      (Eq. 4, Sec. 3.3)
 *   reco_answer_ppl      answer perplexity and stop flag             (Eq. 5, 6)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every pointer is a DEVICE pointer unless marked [host].  The caller owns
 *   all memory and keeps it alive until the work on `stream` has finished.
 * - Calls are asynchronous on `stream`; none synchronises, allocates device
 *   memory or keeps state between calls.  Calls that take a workspace need
 *   `ws_bytes >= reco_*_workspace_size(...)`; workspace contents need not be
 *   initialised and are clobbered.
 * - Host-side validation runs first: a call that returns anything other
 *   than RECO_OK has launched nothing and changed nothing.
 * - Device-side precondition failures (an append past capacity, a retention
 *   outside (0, 1], a NaN or negative score, a token id out of range, a
 *   stored length outside [0, capacity]) are reported through the optional
 *   `dev_err` word: the first failing code is stored with an atomic
 *   compare-and-swap from 0, so the caller should zero it before a call and
 *   read it after synchronising.  A failing unit is left unchanged (select /
 *   compact) or computed on clamped indices (decode); the call still returns
 *   RECO_OK because the host cannot see device data.
 * - KV cache layout: K and V are each
 *       [n_layers][batch][n_kv_heads][capacity][head_dim]
 *   in the cache dtype (fp32 or bf16), row-major; one (layer, sequence,
 *   kv head) "unit" is a contiguous block of `capacity` rows.  `len`
 *   ([n_layers][batch][n_kv_heads], int32) holds the number of valid rows of
 *   each unit; rows at or beyond len are never read as keys.
 * - GQA: query head hq (0 <= hq < n_q_heads) attends through KV head
 *   hq / G with G = n_q_heads / n_kv_heads (1 <= G <= 16).
 * - A call covers layers [layer0, layer0 + n_layers) of the cache; per-layer
 *   inputs and outputs (queries, scores, outputs) are laid out with a
 *   leading [n_layers] dimension for exactly those layers.
 */
#ifndef RECO_H
#define RECO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RECO_ABI_VERSION 3

typedef enum reco_status {
  RECO_OK = 0,
  RECO_ERR_INVALID_ARG = 1,   /* null pointer, bad size, bad layer range ... */
  RECO_ERR_UNSUPPORTED = 2,   /* valid but not implemented (head_dim, G, dtype) */
  RECO_ERR_WORKSPACE = 3,     /* ws is null or smaller than required */
  RECO_ERR_HIP = 4            /* a HIP launch failed */
} reco_status_t;

typedef enum reco_dtype { RECO_F32 = 0, RECO_BF16 = 1 } reco_dtype_t;

/* Codes stored into *dev_err by kernels (first one wins). */
enum {
  RECO_DEV_OK = 0,
  RECO_DEV_APPEND_OVERFLOW = 1,  /* decode append with len == capacity */
  RECO_DEV_BAD_RETENTION = 2,    /* retention r not in (0, 1] (or NaN) */
  RECO_DEV_BAD_SCORE = 3,        /* NaN or negative importance score */
  RECO_DEV_BAD_TOKEN_ID = 4,     /* reflection id or answer token outside [0, vocab) */
  RECO_DEV_BAD_LENGTH = 5,       /* stored len outside [0, capacity] */
  RECO_DEV_BAD_LOGIT = 6         /* a logit row with no non-NaN value to sample */
};

/* reco_score flags */
enum { RECO_SCORE_CAUSAL = 1u };  /* window query at position p sees keys 0..p only */

/* [host] description of a KV cache; read during the call, not retained. */
typedef struct reco_kv_cache {
  void *k;              /* [n_layers][batch][n_kv_heads][capacity][head_dim] */
  void *v;              /* same layout as k */
  int32_t *len;         /* [n_layers][batch][n_kv_heads], valid rows per unit (in/out) */
  int32_t n_layers;     /* layers held by the cache (>= 1) */
  int32_t batch;        /* sequences (>= 1) */
  int32_t n_kv_heads;   /* KV heads per layer (>= 1) */
  int32_t capacity;     /* rows per unit (>= 1) */
  int32_t head_dim;     /* 64 or 128 */
  int32_t dtype;        /* reco_dtype_t; every cache-typed tensor uses it */
} reco_kv_cache_t;

/* ------------------------------------------------------------------------ */
/* Eq. 2 (Section 3.2, attention-guided selection): importance of every cached
 * key as the attention mass it receives from the w most recent tokens.
 * For every unit (layer, sequence, kv head h) with L = len[unit] and
 * w_eff = min(w, L), the window query of position p = L - w + t (row t of
 * q_win, rows with p < 0 are ignored) of each query head in h's group gives a
 * softmax over keys 0..L-1 (0..p when RECO_SCORE_CAUSAL is set) of
 * scale * <q, k_j>; scores[unit][j] is the sum of these softmax rows over the
 * window and the group, for every j < L.  Entries j >= L are left untouched.
 *   q_win : [n_layers][batch][n_q_heads][w][head_dim], cache dtype
 *   scale : logit scale, normally 1/sqrt(head_dim)
 *   row_stats : nullable [n_layers][batch][n_q_heads][w][2] fp32.  NULL: the
 *           softmax normalisers of the window rows come from a first pass
 *           over K (two passes in all).  Given: row t holds the (M, Z) pair
 *           reco_decode_attn wrote when the token at position L - w + t was
 *           decoded, and K is read once.  Exact (up to rounding) only when
 *           no compression happened since the oldest window token was
 *           decoded (the keys it saw then are keys 0..p now), with the same
 *           scale; requires RECO_SCORE_CAUSAL.
 *   scores: [n_layers][batch][n_kv_heads][capacity] fp32 (output)
 * Requires 1 <= w <= capacity, G * w <= 4096 and capacity <= 2^29 (larger:
 * RECO_ERR_UNSUPPORTED).  Accumulation is fp32. */
size_t reco_score_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers,
                                 int32_t n_q_heads, int32_t w);
reco_status_t reco_score(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                         const void *q_win, int32_t n_q_heads, int32_t w, float scale,
                         uint32_t flags, const float *row_stats, float *scores, void *ws,
                         size_t ws_bytes,
                         int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Section 3.2 (reward-driven retention and attention-guided selection):
 * per unit with L = len[unit], w_eff = min(w, L) and
 * r = retention[lc * retention_layer_stride + seq] (lc = layer - layer0),
 *   m = min(L, max(w_eff, ceil(r * L)))      (r * L as an IEEE fp64 product)
 * rows are kept: the window [L - w_eff, L) and the k = m - w_eff prefix
 * positions with the largest scores[unit][j] (ties: lower j first).  The kept
 * rows of K and V are moved, in ascending order, to rows 0..m-1 of the same
 * unit (bit-exact copies; rows >= m keep unspecified contents) and len is set
 * to m.
 *   scores    : [n_layers][batch][n_kv_heads][capacity] fp32, >= 0 (from reco_score)
 *   retention : fp64 in (0, 1]; [batch] with retention_layer_stride = 0
 *               (one retention level per sequence, as Section 3.2 sets it)
 *               or [n_layers][batch] with stride = batch (per-layer
 *               budgets, a policy variant; see reco_layer_retention)
 *   kept_idx  : nullable [n_layers][batch][n_kv_heads][capacity] int32 output;
 *               the first m entries of each unit receive the kept positions
 *               (ascending, in pre-compaction numbering)
 * A unit whose r or scores are invalid is left unchanged and dev_err is set. */
size_t reco_select_compact_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers);
reco_status_t reco_select_compact(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                                  const float *scores, const double *retention,
                                  int64_t retention_layer_stride, int32_t w, int32_t *kept_idx,
                                  void *ws, size_t ws_bytes, int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Score pooling before selection, a policy variant on the same kernels (the
 * clustering idea of the eviction methods the paper cites, Section 1).  Per
 * unit with L = len[unit] and prefix P = L - min(w, L):
 *   pooled[j] = max  (mode RECO_POOL_MAX)  or
 *               mean (mode RECO_POOL_MEAN) of scores[i] over the prefix
 *               positions i with |i - j| <= kernel / 2,        for j < P
 *   pooled[j] = scores[j]                                      for P <= j < L
 * Entries at or beyond L are not written.  Means are summed in fp64 in index
 * order and rounded to fp32 once; maxima are exact.
 *   scores, pooled : [n_layers][batch][n_kv_heads][capacity] fp32, disjoint
 *   kernel         : odd, 1 <= kernel <= 65 (1 copies the scores)
 * A stored len outside [0, capacity] sets RECO_DEV_BAD_LENGTH (unit skipped). */
#define RECO_POOL_MAX 0
#define RECO_POOL_MEAN 1
reco_status_t reco_pool_scores(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                               int32_t w, const float *scores, float *pooled, int32_t kernel,
                               int32_t mode, int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Decode attention over the retained cache (the per-token attention cost of
 * Section 1 that compression reduces).  For every query head hq of every
 * covered (layer, sequence), with h = hq / G and n = len[unit of h]:
 *   if k_new != NULL the new token's row (k_new, v_new) takes part as key n
 *   (it attends to itself) and, after the attention, is written to row n of
 *   the cache and len is incremented;
 *   out[hq] = sum_j softmax_j(scale * <q[hq], k_j>) v_j over the keys j,
 *   lse[hq] = natural log-sum-exp of the scaled logits.
 * With no keys at all out is 0 and lse is -inf.
 *   q            : [n_layers][batch][n_q_heads][head_dim], cache dtype
 *   k_new, v_new : both NULL (no append) or [n_layers][batch][n_kv_heads][head_dim]
 *   out          : [n_layers][batch][n_q_heads][head_dim], cache dtype (output)
 *   lse          : nullable [n_layers][batch][n_q_heads] fp32 (output)
 *   row_stats    : nullable [n_layers][batch][n_q_heads][2] fp32 (output):
 *                  (M, Z) with x_j = scale * log2(e) * <q, k_j>, M = max_j x_j
 *                  and Z = sum_j 2^(x_j - M), so lse = (M + log2 Z) ln 2;
 *                  kept for the window rows, they let reco_score skip its
 *                  normaliser pass (empty: (-inf, 0))
 * An append with len == capacity is not performed (the token still takes part
 * in the attention) and sets RECO_DEV_APPEND_OVERFLOW.
 * The work is split over the compute units of the current device, so the
 * workspace size depends on that device: query it with the device current
 * that the call will run on. */
size_t reco_decode_attn_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers,
                                       int32_t n_q_heads);
reco_status_t reco_decode_attn(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                               const void *q, int32_t n_q_heads, float scale,
                               const void *k_new, const void *v_new, void *out, float *lse,
                               float *row_stats, void *ws, size_t ws_bytes, int32_t *dev_err,
                               hipStream_t stream);

/* reco_decode_attn for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same computation, arguments and errors as reco_decode_attn, without the
 * workspace: the split partials go to a static array inside the library
 * (8 MiB on each device it runs on, held until the process ends), so the call
 * allocates nothing and the caller passes only inputs and outputs.  Every call
 * on one device shares that array and the array keeps the last call's
 * contents (no call depends on them): calls that overlap on one device race,
 * so serialise them (one stream, or events).  The work is split as in
 * reco_decode_attn, so the results agree bit for bit, except for a call with
 * more units (n_layers * batch * n_kv_heads) than the device has compute
 * units whose two-way split would need more than the 8 MiB: it finalises each
 * unit in one workgroup instead, and its results may then differ from
 * reco_decode_attn's in the last bits (within the decode tolerances).
 * Returns RECO_ERR_WORKSPACE if the call would still need more than 8 MiB of
 * partials (with fewer units than compute units a call needs at most
 * compute_units * (16 * head_dim + 32) * 4 bytes, 2.1 MB on a 256-CU
 * MI355X), and RECO_ERR_HIP if the array's device address cannot be looked
 * up; the device current at the call must be the one `stream` belongs to. */
reco_status_t reco_decode_attn_noalloc(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                                       const void *q, int32_t n_q_heads, float scale, const void *k_new,
                                       const void *v_new, void *out, float *lse, float *row_stats,
                                       int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Eq. 3 and Eq. 4 (Section 3.3, reward-banded reflection penalty): for every
 * row b, beta_b = beta_lo if reward[b] <= tau_lo, beta_hi if
 * reward[b] >= tau_hi, beta_mid otherwise (fp32 comparisons), and
 * logits[b][u] -= beta_b (one fp32 subtraction) for every DISTINCT id u in
 * refl_ids.  All other logits are untouched (bit-exact).
 *   logits   : [rows][ld] fp32, in place; ld >= vocab; 1 <= vocab <= 2^30
 *              (larger: RECO_ERR_UNSUPPORTED); 1 <= rows <= 65535
 *   refl_ids : [n_refl] int32, 0 <= n_refl <= 4096, each in [0, vocab)
 *   reward   : [rows] fp32
 * An id outside [0, vocab) is skipped and sets RECO_DEV_BAD_TOKEN_ID. */
reco_status_t reco_logit_penalty(float *logits, int32_t rows, int32_t vocab, int64_t ld,
                                 const int32_t *refl_ids, int32_t n_refl, const float *reward,
                                 float tau_lo, float tau_hi, float beta_lo, float beta_mid,
                                 float beta_hi, int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Eq. 3 and Eq. 4, then sampling (Section 3.3: the next token is drawn from
 * the softmax of the penalised logits), fused into one pass over each row.
 * The penalty is exactly reco_logit_penalty's (written back in place,
 * bit-exact).  Then
 *   T == 0 : tokens[b] = argmax_u z~[b][u]   (greedy; lowest index on ties)
 *   T  > 0 : tokens[b] = argmax_u (z~[b][u] / T + G[b][u])   (Gumbel-max,
 *            an exact draw from softmax(z~[b] / T)), every step in fp32,
 *            G = -log(-log U), U = ((x >> 9) + 1/2) * 2^-23, and x the
 *            (u % 4)-th word of Philox4x32-10 (Salmon et al., SC 2011) on
 *            counter (u / 4, b, offset low, offset high), key (seed low,
 *            seed high).  (seed, offset, b, u) fixes the draw: advance
 *            `offset` once per generated token for fresh noise.
 *   logits   : [rows][ld] fp32, in place; ld >= vocab; 1 <= vocab <= 2^30
 *   refl_ids : [n_refl] int32, 0 <= n_refl <= 4096 (nullable when 0)
 *   reward   : [rows] fp32
 *   tokens   : [rows] int32 (output)
 *   temperature : [host] finite, >= 0 (RECO_ERR_INVALID_ARG otherwise)
 * NaN values never win; a row of NaNs gets token -1 and sets
 * RECO_DEV_BAD_LOGIT.  An id outside [0, vocab) is skipped and sets
 * RECO_DEV_BAD_TOKEN_ID.  rows <= 65535. */
size_t reco_penalty_sample_workspace_size(int32_t rows, int32_t vocab);
reco_status_t reco_penalty_sample(float *logits, int32_t rows, int32_t vocab, int64_t ld,
                                  const int32_t *refl_ids, int32_t n_refl, const float *reward,
                                  float tau_lo, float tau_hi, float beta_lo, float beta_mid,
                                  float beta_hi, float temperature, uint64_t seed, uint64_t offset,
                                  int32_t *tokens, void *ws, size_t ws_bytes, int32_t *dev_err,
                                  hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Eq. 5 and Eq. 6 (Section 3.3, early stopping via answer confidence): for
 * every sequence b, ppl[b] = exp((1/n) sum_t (LSE(logits[b][t]) -
 * logits[b][t][tokens[b][t]])) with natural logarithms, and
 * stop[b] = (ppl[b] <= tau_p).
 *   logits : [batch][n][vocab] fp32 (the probe answer's raw logits),
 *            1 <= vocab <= 2^30 (larger: RECO_ERR_UNSUPPORTED)
 *   tokens : [batch][n] int32 in [0, vocab)
 *   ppl    : [batch] fp32 (output);  stop : nullable [batch] int32 (output)
 *   batch * n <= 65535 (larger: RECO_ERR_UNSUPPORTED)
 * Row log-sum-exps are fp32 partials merged in fp64.  A token out of range
 * makes ppl NaN for its sequence and sets RECO_DEV_BAD_TOKEN_ID. */
size_t reco_answer_ppl_workspace_size(int32_t batch, int32_t n, int32_t vocab);
reco_status_t reco_answer_ppl(const float *logits, const int32_t *tokens, int32_t batch,
                              int32_t n, int32_t vocab, float tau_p, float *ppl, int32_t *stop,
                              void *ws, size_t ws_bytes, int32_t *dev_err, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* [host] Reward -> retention policies (Section 3.2).  Pure functions.
 * reco_retention_from_reward: r = clamp(1 - v/2, lo, hi) in fp64.
 * reco_retention_eq1: Eq. 1, lambda_i = lambda - delta * (v_i - mean) /
 *   (max - min) over v_hist[0..n) (latest last, included); lambda when all
 *   rewards are equal; NaN when n < 1 or v_hist is NULL. */
double reco_retention_from_reward(double v, double lo, double hi);
double reco_retention_eq1(const double *v_hist, int32_t n, double lambda, double delta);

/* [host] Per-layer budgets (policy variant, the pyramid idea cited in
 * Section 1): r_l = min(1, r * (1 + spread * (1 - 2 l / (n_layers - 1)))),
 * a line falling with depth whose mean over layers is r (before the cap);
 * r_l = r when n_layers = 1.  Evaluated in fp64 in exactly this order.  NaN
 * unless 0 < r <= 1, 0 <= spread < 1 and 0 <= layer < n_layers. */
double reco_layer_retention(double r, int32_t layer, int32_t n_layers, double spread);

/* [host] The kept count of Section 3.2 that reco_select_compact uses:
 * m = min(L, max(min(w, L), ceil(r * L))) with r * L an IEEE fp64 product;
 * -1 when r is not in (0, 1], L < 0 or w < 1.  Lets a host controller track
 * cache lengths without reading them back from the device. */
int32_t reco_kept_count(int32_t L, int32_t w, double r);

/* [host] Human-readable status and the ABI version (RECO_ABI_VERSION). */
const char *reco_status_str(reco_status_t status);
int32_t reco_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* RECO_H */
