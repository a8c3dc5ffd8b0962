// Device-side helpers shared by the gfx950 kernels: element types, MFMA
// fragment traits, wave64 reductions and the device error word.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reco {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// Storage type of a bf16 element: raw 16-bit pattern.
struct bf16_t {
  uint16_t bits;
};

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x.bits) << 16);
}

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
  __bf16 b = static_cast<__bf16>(x);  // v_cvt_pk_bf16_f32, round to nearest even
  return bf16_t{__builtin_bit_cast(uint16_t, b)};
}

// ---------------------------------------------------------------------------
// MFMA 16x16 fragments.  For v_mfma_f32_16x16x32_bf16 each lane holds 8
// consecutive k-elements of one row of A (row = lane % 16) and of one column
// of B (column = lane % 16), k-group lane / 16; the 16x16 fp32 result holds
// rows 4 * (lane / 16) + i, i = 0..3, of column lane % 16.  The fp32 variant
// v_mfma_f32_16x16x4_f32 is the same with one k-element per lane.  Only the
// pairing "same lane group, same element slot" matters to the callers, which
// use one consistent permutation of the contraction index for A and B.
// ---------------------------------------------------------------------------
template <typename T>
struct Mfma;

template <>
struct Mfma<bf16_t> {
  static constexpr int kPerLane = 8;    // contraction elements per lane per instruction
  static constexpr int kPerOp = 32;     // contraction length of one instruction
  using frag = bf16x8_t;
  __device__ __forceinline__ static f32x4_t mma(frag a, frag b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mfma<float> {
  static constexpr int kPerLane = 1;
  static constexpr int kPerOp = 4;
  using frag = float;
  __device__ __forceinline__ static f32x4_t mma(frag a, frag b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// 16-byte load that does not allocate in the caches (streamed data read once).
typedef unsigned int u32x4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 nt_load_u4(const void *p) {
  const u32x4v w = __builtin_nontemporal_load(reinterpret_cast<const u32x4v *>(p));
  return make_uint4(w.x, w.y, w.z, w.w);
}

// Load kPerLane consecutive elements starting at p as one MFMA fragment.
__device__ __forceinline__ bf16x8_t load_frag(const bf16_t *p) {
  uint4 u = *reinterpret_cast<const uint4 *>(p);
  return __builtin_bit_cast(bf16x8_t, u);
}
__device__ __forceinline__ float load_frag(const float *p) { return *p; }

__device__ __forceinline__ bf16x8_t zero_frag(bf16x8_t) {
  return __builtin_bit_cast(bf16x8_t, make_uint4(0, 0, 0, 0));
}
__device__ __forceinline__ float zero_frag(float) { return 0.f; }

// Pack 8 fp32 values into a bf16 fragment (round to nearest even).
__device__ __forceinline__ bf16x8_t pack_frag8(const float (&x)[8]) {
  bf16x8_t r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = static_cast<__bf16>(x[j]);
  return r;
}

// ---------------------------------------------------------------------------
// Wave64 cross-lane helpers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, kWave); }

// Reduce over the four lanes {l, l^16, l^32, l^48} (the k-groups of one MFMA column).
__device__ __forceinline__ float group4_max(float v) {
  v = fmaxf(v, shfl_xor(v, 16));
  v = fmaxf(v, shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ float group4_sum(float v) {
  v += shfl_xor(v, 16);
  v += shfl_xor(v, 32);
  return v;
}
// Reduce over the 16 lanes of one lane group (lanes 16g .. 16g+15).
__device__ __forceinline__ float row16_sum(float v) {
  v += shfl_xor(v, 1);
  v += shfl_xor(v, 2);
  v += shfl_xor(v, 4);
  v += shfl_xor(v, 8);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v = fmaxf(v, shfl_xor(v, m));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) v += shfl_xor(v, m);
  return v;
}

// Record a device precondition failure: the first code wins.
__device__ __forceinline__ void report(int32_t *dev_err, int32_t code) {
  if (dev_err) atomicCAS(dev_err, 0, code);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace reco
