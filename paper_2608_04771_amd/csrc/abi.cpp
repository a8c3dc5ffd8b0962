// C ABI of the library: host-side argument validation, workspace sizing and
// launches.  Every entry point validates everything it can see on the host
// before launching anything, so a non-OK status means no side effects.
#include "reco.h"

#include <hip/hip_runtime.h>
#include <math.h>

#include <atomic>
#include <stddef.h>
#include <stdint.h>

#include "reco_kernels.hpp"

namespace {

// Largest vocabulary the logit kernels take: chunk ends (start + chunk
// length) and row offsets then stay far inside int32.
constexpr int32_t kMaxVocab = 1 << 30;

// Largest capacity the score kernels take: their grid spans 8 x chunks
// workgroups of 256 threads along x, which must stay below 2^32 work-items.
constexpr int32_t kMaxScoreCapacity = 1 << 29;

bool cache_ok(const reco_kv_cache_t *c) {
  return c && c->k && c->v && c->len && c->n_layers >= 1 && c->batch >= 1 && c->n_kv_heads >= 1 &&
         c->capacity >= 1;
}

reco_status_t cache_supported(const reco_kv_cache_t *c) {
  if (c->head_dim != 64 && c->head_dim != 128) return RECO_ERR_UNSUPPORTED;
  if (c->dtype != RECO_F32 && c->dtype != RECO_BF16) return RECO_ERR_UNSUPPORTED;
  return RECO_OK;
}

bool layers_ok(const reco_kv_cache_t *c, int32_t layer0, int32_t n_layers) {
  return layer0 >= 0 && n_layers >= 1 && static_cast<int64_t>(layer0) + n_layers <= c->n_layers;
}

// units = n_layers * batch * n_kv_heads must fit an int and a grid dimension.
bool units_ok(const reco_kv_cache_t *c, int32_t n_layers) {
  const int64_t units = static_cast<int64_t>(n_layers) * c->batch * c->n_kv_heads;
  return units >= 1 && units <= 65535;
}

int group_of(const reco_kv_cache_t *c, int32_t n_q_heads) {
  if (n_q_heads < 1 || n_q_heads % c->n_kv_heads != 0) return -1;
  return n_q_heads / c->n_kv_heads;
}

reco_status_t hip_status(hipError_t e) { return e == hipSuccess ? RECO_OK : RECO_ERR_HIP; }

// Compute units of the current device, read once per device (256 on a whole
// MI355X; a partitioned GPU shows fewer).  Falls back to 256 if the query
// fails, which only changes the split count, never correctness.
int current_compute_units() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cached[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
  cached[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace

extern "C" {

const char *reco_status_str(reco_status_t s) {
  switch (s) {
    case RECO_OK: return "ok";
    case RECO_ERR_INVALID_ARG: return "invalid argument";
    case RECO_ERR_UNSUPPORTED: return "unsupported configuration";
    case RECO_ERR_WORKSPACE: return "workspace missing or too small";
    case RECO_ERR_HIP: return "HIP launch failure";
  }
  return "unknown status";
}

int32_t reco_abi_version(void) { return RECO_ABI_VERSION; }

double reco_retention_from_reward(double v, double lo, double hi) {
  double r = 1.0 - 0.5 * v;
  if (r < lo) r = lo;
  if (r > hi) r = hi;
  return r;
}

double reco_retention_eq1(const double *v_hist, int32_t n, double lambda, double delta) {
  if (!v_hist || n < 1) return NAN;
  double sum = 0.0, vmin = v_hist[0], vmax = v_hist[0];
  for (int32_t i = 0; i < n; ++i) {
    sum += v_hist[i];
    if (v_hist[i] < vmin) vmin = v_hist[i];
    if (v_hist[i] > vmax) vmax = v_hist[i];
  }
  if (vmax == vmin) return lambda;
  const double mean = sum / n;
  return lambda - delta * (v_hist[n - 1] - mean) / (vmax - vmin);
}

double reco_layer_retention(double r, int32_t layer, int32_t n_layers, double spread) {
  if (!(r > 0.0 && r <= 1.0) || !(spread >= 0.0 && spread < 1.0) || n_layers < 1 || layer < 0 ||
      layer >= n_layers)
    return NAN;
  if (n_layers == 1) return r;
  const double t = static_cast<double>(layer) / static_cast<double>(n_layers - 1);
  const double x = r * (1.0 + spread * (1.0 - 2.0 * t));
  return x < 1.0 ? x : 1.0;
}

int32_t reco_kept_count(int32_t L, int32_t w, double r) {
  if (!(r > 0.0 && r <= 1.0) || L < 0 || w < 1) return -1;
  const int32_t w_eff = w < L ? w : L;
  int32_t m = static_cast<int32_t>(ceil(r * static_cast<double>(L)));
  if (m < w_eff) m = w_eff;
  if (m > L) m = L;
  return m;
}

// ---------------------------------------------------------------- score
size_t reco_score_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers, int32_t n_q_heads, int32_t w) {
  if (!cache_ok(cache) || !units_ok(cache, n_layers) || w < 1 || cache->capacity > kMaxScoreCapacity) return 0;
  const int G = group_of(cache, n_q_heads);
  if (G < 1 || static_cast<int64_t>(G) * w > reco::kScoreMaxRows) return 0;
  const int units = n_layers * cache->batch * cache->n_kv_heads;
  return reco::score_workspace_bytes(units, cache->capacity, G * w);
}

reco_status_t reco_score(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers, const void *q_win,
                         int32_t n_q_heads, int32_t w, float scale, uint32_t flags, const float *row_stats,
                         float *scores, void *ws, size_t ws_bytes, int32_t *dev_err, hipStream_t stream) {
  if (!cache_ok(cache) || !q_win || !scores) return RECO_ERR_INVALID_ARG;
  if (row_stats && !(flags & RECO_SCORE_CAUSAL)) return RECO_ERR_INVALID_ARG;   // decode statistics are causal
  if (!layers_ok(cache, layer0, n_layers) || !units_ok(cache, n_layers)) return RECO_ERR_INVALID_ARG;
  if (w < 1 || w > cache->capacity || !isfinite(scale) || (flags & ~RECO_SCORE_CAUSAL)) return RECO_ERR_INVALID_ARG;
  const int G = group_of(cache, n_q_heads);
  if (G < 1) return RECO_ERR_INVALID_ARG;
  reco_status_t st = cache_supported(cache);
  if (st != RECO_OK) return st;
  if (static_cast<int64_t>(G) * w > reco::kScoreMaxRows) return RECO_ERR_UNSUPPORTED;
  if (cache->capacity > kMaxScoreCapacity) return RECO_ERR_UNSUPPORTED;
  const size_t need = reco_score_workspace_size(cache, n_layers, n_q_heads, w);
  if (!ws || ws_bytes < need) return RECO_ERR_WORKSPACE;

  const int units = n_layers * cache->batch * cache->n_kv_heads;
  reco::ScoreParams p{};
  p.k = cache->k;
  p.len = cache->len;
  p.q_win = q_win;
  p.scores = scores;
  p.rows = G * w;
  p.rows_pad = (p.rows + 15) / 16 * 16;
  p.chunks = (cache->capacity + reco::kScoreChunk - 1) / reco::kScoreChunk;
  p.chunk_keys = reco::kScoreChunk;
  p.cus = current_compute_units();
  p.row_part = reinterpret_cast<float *>(ws);
  p.row_stat = p.row_part + static_cast<size_t>(units) * p.chunks * p.rows_pad * 2;
  p.given = row_stats;
  p.dev_err = dev_err;
  p.layer0 = layer0;
  p.n_layers = n_layers;
  p.batch = cache->batch;
  p.hkv = cache->n_kv_heads;
  p.cap = cache->capacity;
  p.group = G;
  p.hq = n_q_heads;
  p.w = w;
  p.causal = (flags & RECO_SCORE_CAUSAL) ? 1 : 0;
  p.scale_log2 = scale * 1.4426950408889634f;
  return hip_status(reco::launch_score(p, cache->dtype, cache->head_dim, stream));
}

// ---------------------------------------------------------------- select + compact
size_t reco_select_compact_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers) {
  if (!cache_ok(cache) || !units_ok(cache, n_layers)) return 0;
  const int units = n_layers * cache->batch * cache->n_kv_heads;
  return reco::select_workspace_bytes(units, cache->capacity, true);
}

reco_status_t reco_select_compact(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers,
                                  const float *scores, const double *retention, int64_t retention_layer_stride,
                                  int32_t w, int32_t *kept_idx, void *ws, size_t ws_bytes, int32_t *dev_err,
                                  hipStream_t stream) {
  if (!cache_ok(cache) || !scores || !retention || retention_layer_stride < 0) return RECO_ERR_INVALID_ARG;
  if (!layers_ok(cache, layer0, n_layers) || !units_ok(cache, n_layers)) return RECO_ERR_INVALID_ARG;
  if (w < 1 || w > cache->capacity) return RECO_ERR_INVALID_ARG;
  reco_status_t st = cache_supported(cache);
  if (st != RECO_OK) return st;
  const int units = n_layers * cache->batch * cache->n_kv_heads;
  const size_t need = reco::select_workspace_bytes(units, cache->capacity, kept_idx == nullptr);
  if (!ws || ws_bytes < need) return RECO_ERR_WORKSPACE;

  reco::SelectParams p{};
  p.k = cache->k;
  p.v = cache->v;
  p.len = cache->len;
  p.scores = scores;
  p.retention = retention;
  p.ret_stride = retention_layer_stride;
  p.kept = reinterpret_cast<int32_t *>(ws);
  const size_t kept_bytes = (static_cast<size_t>(units) * sizeof(int32_t) + 255) / 256 * 256;
  p.idx = kept_idx ? kept_idx : reinterpret_cast<int32_t *>(reinterpret_cast<char *>(ws) + kept_bytes);
  p.dev_err = dev_err;
  p.layer0 = layer0;
  p.n_layers = n_layers;
  p.batch = cache->batch;
  p.hkv = cache->n_kv_heads;
  p.cap = cache->capacity;
  p.w = w;
  return hip_status(reco::launch_select_compact(p, cache->dtype, cache->head_dim, stream));
}

// ---------------------------------------------------------------- pooling
reco_status_t reco_pool_scores(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers, int32_t w,
                               const float *scores, float *pooled, int32_t kernel, int32_t mode, int32_t *dev_err,
                               hipStream_t stream) {
  if (!cache_ok(cache) || !scores || !pooled) return RECO_ERR_INVALID_ARG;
  if (!layers_ok(cache, layer0, n_layers) || !units_ok(cache, n_layers)) return RECO_ERR_INVALID_ARG;
  if (w < 1 || w > cache->capacity) return RECO_ERR_INVALID_ARG;
  if (kernel < 1 || kernel > reco::kPoolMaxKernel || kernel % 2 == 0) return RECO_ERR_INVALID_ARG;
  if (mode != RECO_POOL_MAX && mode != RECO_POOL_MEAN) return RECO_ERR_INVALID_ARG;
  const size_t bytes = static_cast<size_t>(n_layers) * cache->batch * cache->n_kv_heads * cache->capacity * 4;
  const char *a = reinterpret_cast<const char *>(scores), *o = reinterpret_cast<const char *>(pooled);
  if (a < o + bytes && o < a + bytes) return RECO_ERR_INVALID_ARG;     // in and out must not overlap
  reco::PoolParams p{};
  p.len = cache->len;
  p.scores = scores;
  p.pooled = pooled;
  p.dev_err = dev_err;
  p.layer0 = layer0;
  p.n_layers = n_layers;
  p.batch = cache->batch;
  p.hkv = cache->n_kv_heads;
  p.cap = cache->capacity;
  p.w = w;
  p.kernel = kernel;
  p.mode = mode;
  return hip_status(reco::launch_pool_scores(p, stream));
}

// ---------------------------------------------------------------- decode
size_t reco_decode_attn_workspace_size(const reco_kv_cache_t *cache, int32_t n_layers, int32_t n_q_heads) {
  if (!cache_ok(cache) || !units_ok(cache, n_layers) || group_of(cache, n_q_heads) < 1) return 0;
  const int units = n_layers * cache->batch * cache->n_kv_heads;
  return reco::decode_workspace_bytes(units, cache->capacity, cache->head_dim, current_compute_units());
}

}  // extern "C"

namespace {

// Shared by both decode entry points: host validation, then the launch with
// the split partials in `ws` (caller workspace) or, when `ws` is null, in the
// library's static per-device scratch array.
reco_status_t decode_common(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers, const void *q,
                            int32_t n_q_heads, float scale, const void *k_new, const void *v_new, void *out,
                            float *lse, float *row_stats, void *ws, size_t ws_bytes, bool use_scratch,
                            int32_t *dev_err, hipStream_t stream) {
  if (!cache_ok(cache) || !q || !out) return RECO_ERR_INVALID_ARG;
  if ((k_new == nullptr) != (v_new == nullptr)) return RECO_ERR_INVALID_ARG;
  if (!layers_ok(cache, layer0, n_layers) || !units_ok(cache, n_layers) || !isfinite(scale))
    return RECO_ERR_INVALID_ARG;
  const int G = group_of(cache, n_q_heads);
  if (G < 1) return RECO_ERR_INVALID_ARG;
  reco_status_t st = cache_supported(cache);
  if (st != RECO_OK) return st;
  if (G > 16) return RECO_ERR_UNSUPPORTED;
  const int units = n_layers * cache->batch * cache->n_kv_heads;
  const int cus = current_compute_units();
  if (use_scratch) {
    if (reco::decode_scratch_bytes(units, cache->capacity, cache->head_dim, cus) > reco::kDecodeScratchBytes)
      return RECO_ERR_WORKSPACE;
    if (reco::decode_scratch(&ws) != hipSuccess) return RECO_ERR_HIP;
  } else {
    const size_t need = reco::decode_workspace_bytes(units, cache->capacity, cache->head_dim, cus);
    if (!ws || ws_bytes < need) return RECO_ERR_WORKSPACE;
  }

  reco::DecodeParams p{};
  p.k = cache->k;
  p.v = cache->v;
  p.len = cache->len;
  p.q = q;
  p.k_new = k_new;
  p.v_new = v_new;
  p.out = out;
  p.lse = lse;
  p.row_stats = row_stats;
  p.splits = use_scratch ? reco::decode_scratch_splits(units, cache->capacity, cache->head_dim, cus)
                         : reco::decode_splits(units, cache->capacity, cus);
  p.part_o = reinterpret_cast<float *>(ws);
  p.part_ml = p.part_o + static_cast<size_t>(units) * p.splits * 16 * cache->head_dim;
  p.dev_err = dev_err;
  p.layer0 = layer0;
  p.n_layers = n_layers;
  p.batch = cache->batch;
  p.hkv = cache->n_kv_heads;
  p.cap = cache->capacity;
  p.group = G;
  p.hq = n_q_heads;
  p.scale_log2 = scale * 1.4426950408889634f;
  return hip_status(reco::launch_decode(p, cache->dtype, cache->head_dim, stream));
}

}  // namespace

extern "C" {

reco_status_t reco_decode_attn(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers, const void *q,
                               int32_t n_q_heads, float scale, const void *k_new, const void *v_new, void *out,
                               float *lse, float *row_stats, void *ws, size_t ws_bytes, int32_t *dev_err,
                               hipStream_t stream) {
  return decode_common(cache, layer0, n_layers, q, n_q_heads, scale, k_new, v_new, out, lse, row_stats, ws,
                       ws_bytes, false, dev_err, stream);
}

reco_status_t reco_decode_attn_noalloc(const reco_kv_cache_t *cache, int32_t layer0, int32_t n_layers, const void *q,
                                       int32_t n_q_heads, float scale, const void *k_new, const void *v_new,
                                       void *out, float *lse, float *row_stats, int32_t *dev_err,
                                       hipStream_t stream) {
  return decode_common(cache, layer0, n_layers, q, n_q_heads, scale, k_new, v_new, out, lse, row_stats, nullptr,
                       0, true, dev_err, stream);
}

// ---------------------------------------------------------------- penalty
reco_status_t reco_logit_penalty(float *logits, int32_t rows, int32_t vocab, int64_t ld, const int32_t *refl_ids,
                                 int32_t n_refl, const float *reward, float tau_lo, float tau_hi, float beta_lo,
                                 float beta_mid, float beta_hi, int32_t *dev_err, hipStream_t stream) {
  if (!logits || !reward || rows < 1 || rows > 65535 || vocab < 1 || ld < vocab) return RECO_ERR_INVALID_ARG;
  if (vocab > kMaxVocab) return RECO_ERR_UNSUPPORTED;
  if (n_refl < 0 || n_refl > 4096 || (n_refl > 0 && !refl_ids)) return RECO_ERR_INVALID_ARG;
  if (n_refl == 0) return RECO_OK;
  return hip_status(reco::launch_logit_penalty(logits, rows, vocab, ld, refl_ids, n_refl, reward, tau_lo, tau_hi,
                                               beta_lo, beta_mid, beta_hi, dev_err, stream));
}

// ---------------------------------------------------------------- penalty + sampling
size_t reco_penalty_sample_workspace_size(int32_t rows, int32_t vocab) {
  if (rows < 1 || vocab < 1 || vocab > kMaxVocab) return 0;
  return reco::penalty_sample_workspace_bytes(rows, vocab);
}

reco_status_t reco_penalty_sample(float *logits, int32_t rows, int32_t vocab, int64_t ld, const int32_t *refl_ids,
                                  int32_t n_refl, const float *reward, float tau_lo, float tau_hi, float beta_lo,
                                  float beta_mid, float beta_hi, float temperature, uint64_t seed, uint64_t offset,
                                  int32_t *tokens, void *ws, size_t ws_bytes, int32_t *dev_err, hipStream_t stream) {
  if (!logits || !reward || !tokens || rows < 1 || rows > 65535 || vocab < 1 || ld < vocab)
    return RECO_ERR_INVALID_ARG;
  if (n_refl < 0 || n_refl > 4096 || (n_refl > 0 && !refl_ids)) return RECO_ERR_INVALID_ARG;
  if (!(temperature >= 0.f) || !isfinite(temperature)) return RECO_ERR_INVALID_ARG;
  if (vocab > kMaxVocab) return RECO_ERR_UNSUPPORTED;
  const size_t need = reco::penalty_sample_workspace_bytes(rows, vocab);
  if (!ws || ws_bytes < need) return RECO_ERR_WORKSPACE;
  return hip_status(reco::launch_penalty_sample(logits, rows, vocab, ld, refl_ids, n_refl, reward, tau_lo, tau_hi,
                                                beta_lo, beta_mid, beta_hi, temperature, seed, offset, tokens, ws,
                                                dev_err, stream));
}

// ---------------------------------------------------------------- answer PPL
size_t reco_answer_ppl_workspace_size(int32_t batch, int32_t n, int32_t vocab) {
  if (batch < 1 || n < 1 || vocab < 1 || vocab > kMaxVocab) return 0;
  return reco::ppl_workspace_bytes(batch, n, vocab);
}

reco_status_t reco_answer_ppl(const float *logits, const int32_t *tokens, int32_t batch, int32_t n, int32_t vocab,
                              float tau_p, float *ppl, int32_t *stop, void *ws, size_t ws_bytes, int32_t *dev_err,
                              hipStream_t stream) {
  if (!logits || !tokens || !ppl || batch < 1 || n < 1 || vocab < 1) return RECO_ERR_INVALID_ARG;
  if (vocab > kMaxVocab) return RECO_ERR_UNSUPPORTED;
  if (batch > 65535 || static_cast<int64_t>(batch) * n > 65535) return RECO_ERR_UNSUPPORTED;
  const size_t need = reco::ppl_workspace_bytes(batch, n, vocab);
  if (!ws || ws_bytes < need) return RECO_ERR_WORKSPACE;
  return hip_status(reco::launch_answer_ppl(logits, tokens, batch, n, vocab, tau_p, ppl, stop, ws, dev_err, stream));
}

}  // extern "C"
