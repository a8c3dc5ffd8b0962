// Launch interface of the decode-attention kernels (decode_attn.hip), kept
// apart from the other kernels' declarations.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace reco {

// ---- decode attention ------------------------------------------------------
struct DecodeParams {
  void *k;                // cache K base (whole cache); the append commit writes it
  void *v;                // cache V base
  int32_t *len;           // [cache layers][batch][hkv]
  const void *q;          // [n_layers][batch][hq][D]
  const void *k_new;      // nullable [n_layers][batch][hkv][D]
  const void *v_new;
  void *out;              // [n_layers][batch][hq][D]
  float *lse;             // nullable [n_layers][batch][hq]
  float *row_stats;       // nullable [n_layers][batch][hq][2]: (max, sum) of the log2-domain logits
  float *part_o;          // [units][splits][16][D]
  float *part_ml;         // [units][splits][32]  (16 maxima, 16 sums)
  int32_t *dev_err;
  int layer0, n_layers, batch, hkv, cap, group, hq, splits;
  float scale_log2;       // logit scale * log2(e)
};
hipError_t launch_decode(const DecodeParams &p, int dtype, int head_dim, hipStream_t s);

// ---- allocation-free decode: split partials in a file-scope device array ----
// (kDecodeScratchBytes on every device; see decode_plan.hpp for its size and
// the split rule of such calls.)
// Device address of the current device's array, looked up with
// hipGetSymbolAddress on the first call per device and kept.
hipError_t decode_scratch(void **ptr);

}  // namespace reco
