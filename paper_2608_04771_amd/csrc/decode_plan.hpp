// Work split of the decode-attention kernels (decode_attn.hip): how many
// workgroups share one unit's keys, and the bytes of split partials that
// implies.  Host code only; kept apart from the kernel sources so that
// tuning the split rule leaves the kernels' files untouched.
#pragma once

#include <stddef.h>

namespace reco {

constexpr int kDecodeTile = 32;          // keys per wave iteration of the attention kernel
constexpr int kDecodeMaxSplits = 128;    // most splits the merge kernels take

// compute_units: CUs of the device the call runs on (sets the split count).
int decode_splits(int units, int capacity, int compute_units);
size_t decode_workspace_bytes(int units, int capacity, int head_dim, int compute_units);

// Size of the allocation-free entry point's static partials array on every
// device (the split partials of one call with at most compute_units units
// need at most compute_units * (16 * head_dim + 32) * 4 bytes: 2.1 MB on a
// 256-CU device at head_dim 128).
constexpr size_t kDecodeScratchBytes = size_t(8) << 20;
// Split count of an allocation-free call: decode_splits, except that a call
// with more units than compute units whose partials would not fit the array
// takes one split per unit.
int decode_scratch_splits(int units, int capacity, int head_dim, int compute_units);
// Bytes of the array one call uses (0 when every unit is a single split,
// which needs no partials).
size_t decode_scratch_bytes(int units, int capacity, int head_dim, int compute_units);

}  // namespace reco
