// Work split of the decode-attention kernels: the rule and the partial sizes
// it implies (host code).
#include "decode_plan.hpp"

namespace reco {

// Splits per unit: at most one workgroup per compute unit of the device
// (256 on a whole MI355X, fewer on a partition of it).  Measured on the
// 7B-shaped cache, a single resident round with one workgroup per CU streams
// fastest: two workgroups sharing a CU finish later than the rest, and a
// second round adds its ramp to the tail.  At least four 32-key tiles per
// split at capacity.  With more units than compute units the grid runs in
// several rounds anyway; there long units (8K rows or more at capacity) are
// cut in two, which halves the work of the last workgroups to finish (the
// ragged 7B batch: 4.49 -> 4.27 ms per call; the 32B 64K batch 12.03 ->
// 11.91 ms).
int decode_splits(int units, int capacity, int compute_units) {
  const int tiles_cap = (capacity + 1 + kDecodeTile - 1) / kDecodeTile;
  int splits = compute_units / units;
  if (units > compute_units && tiles_cap >= 256) splits = 2;
  int max_splits = tiles_cap / 4;
  if (max_splits > kDecodeMaxSplits) max_splits = kDecodeMaxSplits;
  if (max_splits < 1) max_splits = 1;
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  return splits;
}

namespace {
size_t partial_bytes(int units, int splits, int head_dim) {
  return static_cast<size_t>(units) * splits * (16 * static_cast<size_t>(head_dim) + 32) * sizeof(float);
}
}  // namespace

size_t decode_workspace_bytes(int units, int capacity, int head_dim, int compute_units) {
  return partial_bytes(units, decode_splits(units, capacity, compute_units), head_dim);
}

int decode_scratch_splits(int units, int capacity, int head_dim, int compute_units) {
  const int splits = decode_splits(units, capacity, compute_units);
  // Many-unit calls whose two-way split would not fit the array finalise
  // each unit in one workgroup instead (no partials).
  if (splits > 1 && units > compute_units && partial_bytes(units, splits, head_dim) > kDecodeScratchBytes) return 1;
  return splits;
}

size_t decode_scratch_bytes(int units, int capacity, int head_dim, int compute_units) {
  const int splits = decode_scratch_splits(units, capacity, head_dim, compute_units);
  if (splits == 1) return 0;   // finalised in place, no partials
  return partial_bytes(units, splits, head_dim);
}

}  // namespace reco
