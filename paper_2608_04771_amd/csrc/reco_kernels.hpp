// Internal launch interface between the C-ABI layer (abi.cpp) and the kernel
// translation units.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "decode_attn.hpp"
#include "decode_plan.hpp"

namespace reco {

// ---- window attention-mass scoring --------------------------------------------
struct ScoreParams {
  const void *k;          // cache K base
  const int32_t *len;
  const void *q_win;      // [n_layers][batch][hq][w][D]
  float *scores;          // [n_layers][batch][hkv][cap]
  float *row_part;        // [units][chunks][rows_pad][2]  per-chunk (max, sum) in log2 domain
  float *row_stat;        // [units][rows_pad][2]          (max, 1/sum)
  const float *given;     // nullable [n_layers][batch][hq][w][2] window-row (max, sum) from decode
  int32_t *dev_err;
  int layer0, n_layers, batch, hkv, cap, group, hq, w, rows, rows_pad, chunks;
  int chunk_keys;         // keys per work item (set by launch_score; chunks = ceil(cap / chunk_keys))
  int cus;                // compute units of the device (persistent grids)
  int causal;
  float scale_log2;
};
constexpr int kScoreChunk = 512;      // keys per workgroup of the row-split kernels (workspace sizing)
constexpr int kScoreMaxRows = 4096;   // G * w limit
size_t score_workspace_bytes(int units, int capacity, int rows);
hipError_t launch_score(const ScoreParams &p, int dtype, int head_dim, hipStream_t s);

// ---- selection + in-place compaction ----------------------------------------
struct SelectParams {
  void *k;                // cache K base
  void *v;
  int32_t *len;
  const float *scores;    // [n_layers][batch][hkv][cap]
  const double *retention;  // [batch], or [n_layers][batch] with ret_stride = batch
  int32_t *idx;           // [n_layers][batch][hkv][cap]  kept positions (user buffer or workspace)
  int32_t *kept;          // [units] kept count m, or -1 for "leave unchanged"
  int32_t *dev_err;
  int64_t ret_stride;     // retention of (covered layer lc, seq b) = retention[lc * ret_stride + b]
  int layer0, n_layers, batch, hkv, cap, w;
};
size_t select_workspace_bytes(int units, int capacity, bool need_idx);
hipError_t launch_select_compact(const SelectParams &p, int dtype, int head_dim, hipStream_t s);

// ---- score pooling (policy variant) ---------------------------------------------
constexpr int kPoolMaxKernel = 65;
struct PoolParams {
  const int32_t *len;
  const float *scores;    // [n_layers][batch][hkv][cap]
  float *pooled;          // same shape, must not overlap scores
  int32_t *dev_err;
  int layer0, n_layers, batch, hkv, cap, w, kernel, mode;
};
hipError_t launch_pool_scores(const PoolParams &p, hipStream_t s);

// ---- reflection penalty ------------------------------------------------------
hipError_t launch_logit_penalty(float *logits, int rows, int vocab, int64_t ld, const int32_t *ids,
                                int n_ids, const float *reward, float tau_lo, float tau_hi,
                                float b_lo, float b_mid, float b_hi, int32_t *dev_err,
                                hipStream_t s);

// ---- fused penalty + sampling -----------------------------------------------
size_t penalty_sample_workspace_bytes(int rows, int vocab);
hipError_t launch_penalty_sample(float *logits, int rows, int vocab, int64_t ld, const int32_t *ids, int n_ids,
                                 const float *reward, float tau_lo, float tau_hi, float b_lo, float b_mid,
                                 float b_hi, float temperature, uint64_t seed, uint64_t offset, int32_t *tokens,
                                 void *ws, int32_t *dev_err, hipStream_t s);

// ---- answer perplexity -----------------------------------------------------------
size_t ppl_workspace_bytes(int batch, int n, int vocab);
hipError_t launch_answer_ppl(const float *logits, const int32_t *tokens, int batch, int n, int vocab,
                             float tau_p, float *ppl, int32_t *stop, void *ws, int32_t *dev_err,
                             hipStream_t s);

}  // namespace reco
