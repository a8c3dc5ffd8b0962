// Window attention-mass scoring of every cached key (Eq. 2), gfx950.
//
// For one unit (layer, sequence, kv head h) the window rows are the G * w
// (query head of h's group, window position) pairs.  Row r = g * w + t is the
// query of head h*G + g at absolute position pos = L - w + t.  Scoring takes
// the softmax normaliser (max, sum) of every window row (a statistics pass
// over K, or the values decode wrote for the window tokens), then the mass
// pass adds exp2(x - max) / sum over all rows of each key.  Logits come from
// the matrix cores (16 keys x 16 rows per v_mfma_f32_16x16x32_bf16, bf16
// products accumulated in fp32).
//
// Two kernel families:
// * key-split (most shapes): a persistent grid of one eight-wave workgroup
//   per CU.  A workgroup stages the unit's window rows in LDS once per
//   segment of its share of the keys, and every wave walks its own groups of
//   64 keys, loading their K fragments from global memory straight into
//   registers and multiplying them against every row tile read from LDS;
//   each score is summed in registers and written once, and no barrier runs
//   inside the key loop.
// * row-split (window rows that do not fit the LDS of a CU next to the
//   per-wave state, and fp32 at head_dim 128): per (unit, 512-key chunk)
//   four waves split the window rows, held as MFMA fragments in registers,
//   and stream the chunk's keys through a double-buffered LDS stage; a row
//   merge kernel combines the per-chunk statistics.
//
// Measured on the gfx950 issue model: a 16x16x32 bf16 MFMA occupies a SIMD
// for 16 cycles and hides only about 5 cycles of exp or 8-11 of FMA issue
// from its own wave (3-8 from the other wave of the SIMD), v_exp_f32 takes
// about 8 cycles and an FMA 4 (2 with two waves per SIMD).  Each (row, key) pair
// needs a quarter of an MFMA plus one exp2 and two FMA-class operations per
// pass, so the passes are bound by MFMA + VALU issue combined, not by either
// alone; both families keep the per-pair work at that minimum.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

#include <math.h>

namespace reco {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;       // waves per scoring workgroup
constexpr int kBlock = 32;        // keys per LDS block (two 16-key MFMA tiles)

// Sum over the four lanes {l, l^16, l^32, l^48} without an LDS round trip:
// gfx950's row swaps hand each lane its partner row's value (rows 0/1 and
// 2/3 for the 16-lane swap, 0/2 and 1/3 for the 32-lane swap), so two
// butterfly steps leave the group's total in every lane.  Each step adds the
// same two values as a shuffle-based butterfly, so the result is the same.
__device__ __forceinline__ float group4_sum_swap(float v) {
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

struct UnitInfo {
  int lc, b, h;
  size_t cunit;   // unit index in the whole cache
  size_t ounit;   // unit index among the covered layers
  int L;
};

__device__ __forceinline__ UnitInfo unit_info(const ScoreParams &p, int unit) {
  UnitInfo u;
  const int per_layer = p.batch * p.hkv;
  u.lc = unit / per_layer;
  u.b = (unit % per_layer) / p.hkv;
  u.h = unit % p.hkv;
  u.cunit = (static_cast<size_t>(p.layer0 + u.lc) * p.batch + u.b) * p.hkv + u.h;
  u.ounit = static_cast<size_t>(unit);
  int L = p.len[u.cunit];
  u.L = L < 0 ? 0 : (L > p.cap ? p.cap : L);
  return u;
}

// Workgroup -> (chunk, unit) for the statistics and mass passes.  The
// dispatcher hands consecutive workgroup ids to the eight XCDs in turn, and
// every XCD has its own L2; ids are laid out so that all chunks of a unit
// share one id residue mod 8 (one XCD), so each unit's window queries, which
// every chunk of the unit reads, come from HBM once instead of once per XCD.
// The grid is (8 x chunks, units / 8 rounded up): workgroup (x, y) has id
// y * 8 * chunks + x, so id mod 8 = x mod 8; it takes unit 8y + x mod 8 and
// chunk x / 8.  Padding workgroups (unit past the last) return at once.
__device__ __forceinline__ bool xcd_chunk_unit(const ScoreParams &p, int &chunk, int &unit) {
  unit = static_cast<int>(blockIdx.y) * 8 + static_cast<int>(blockIdx.x & 7);
  chunk = static_cast<int>(blockIdx.x >> 3);
  return unit < p.n_layers * p.batch * p.hkv;
}

template <typename T, int D>
struct ScoreCfg {
  using MF = Mfma<T>;
  static constexpr int dq = D / 4;                       // head-dim elements per lane group
  static constexpr int steps = dq / MF::kPerLane;        // MFMAs per 16x16 logit tile
  static constexpr int row_bytes = D * (int)sizeof(T);
  static constexpr int k_stride = row_bytes + 16;        // padded, 16-byte aligned LDS pitch
  static constexpr int stage_bytes = kBlock * k_stride;
  static constexpr int lanes_per_row = row_bytes / 16;
  static constexpr int pieces = kBlock * lanes_per_row;              // 16-byte pieces per block
  static constexpr int max_loads = pieces / (kWaves * kWave);        // per thread (4-wave workgroups)
};

template <typename T, int D, int RTW>
struct RowBlock {
  using MF = Mfma<T>;
  using frag = typename MF::frag;
  static constexpr int steps = ScoreCfg<T, D>::steps;
  frag q[RTW][steps];
  int pos[RTW];      // absolute position of the lane's row (for causality)
  bool valid[RTW];   // the lane's row exists

  // Rows of tiles tile0 + k (k < RTW) for lane (col, grp).
  __device__ __forceinline__ void load(const ScoreParams &p, const UnitInfo &u, int tile0, int col, int grp) {
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      const int r = (tile0 + k) * 16 + col;
      const int g = r / p.w;
      const int t = r - g * p.w;
      const int ps = u.L - p.w + t;
      valid[k] = (r < p.rows) && (ps >= 0);
      pos[k] = ps;
      const T *qrow = reinterpret_cast<const T *>(p.q_win) +
                      (((static_cast<size_t>(u.lc) * p.batch + u.b) * p.hq + u.h * p.group + (valid[k] ? g : 0)) * p.w +
                       (valid[k] ? t : 0)) * D + grp * ScoreCfg<T, D>::dq;
#pragma unroll
      for (int c = 0; c < steps; ++c)
        q[k][c] = valid[k] ? load_frag(qrow + c * MF::kPerLane) : zero_frag(frag{});
    }
  }
};

// The thread's 16-byte pieces of one 32-key block of K (piece i * 256 + thread).
template <typename T, int D>
struct BlockRegs {
  uint4 r[ScoreCfg<T, D>::max_loads];
};

// Global -> registers: the thread's pieces of the 32-key block at kb (rows
// past the end of the cache read row 0 and are masked later).
template <typename T, int D>
__device__ __forceinline__ void load_block(BlockRegs<T, D> &regs, const T *kbase, int kb, int L) {
  using Cfg = ScoreCfg<T, D>;
#pragma unroll
  for (int i = 0; i < Cfg::max_loads; ++i) {
    const int piece = i * kThreads + static_cast<int>(threadIdx.x);
    const int r = piece / Cfg::lanes_per_row;
    const int key = kb + r;
    const unsigned char *src =
        reinterpret_cast<const unsigned char *>(kbase + static_cast<size_t>(key < L ? key : 0) * D);
    regs.r[i] = nt_load_u4(src + (piece % Cfg::lanes_per_row) * 16);
  }
}

template <typename T, int D>
__device__ __forceinline__ void store_block(unsigned char *stage, const BlockRegs<T, D> &regs) {
  using Cfg = ScoreCfg<T, D>;
#pragma unroll
  for (int i = 0; i < Cfg::max_loads; ++i) {
    const int piece = i * kThreads + static_cast<int>(threadIdx.x);
    const int r = piece / Cfg::lanes_per_row;
    *reinterpret_cast<uint4 *>(stage + r * Cfg::k_stride + (piece % Cfg::lanes_per_row) * 16) = regs.r[i];
  }
}

// MFMA operand of 16-key tile kt of the staged block: lane holds key
// kt*16 + col, head-dim slice grp*dq + c*kpl.
template <typename T, int D>
__device__ __forceinline__ void key_frags(const unsigned char *stage, int kt, int col, int grp,
                                          typename Mfma<T>::frag (&kf)[ScoreCfg<T, D>::steps]) {
  using Cfg = ScoreCfg<T, D>;
  const T *row = reinterpret_cast<const T *>(stage + (kt * 16 + col) * Cfg::k_stride) + grp * Cfg::dq;
#pragma unroll
  for (int c = 0; c < Cfg::steps; ++c) kf[c] = load_frag(row + c * Mfma<T>::kPerLane);
}

// Statistics pass body for one 32-key block (two 16-key tiles): S^T = K.Q^T,
// lane holds keys kb + kt*16 + 4*grp + i of row (tile0 + k)*16 + col; online
// (max, sum) per lane over its 8 keys of the block at once (one rescale per
// block), merged over the lane groups at the end of the chunk.  With a
// positive scale the maximum is taken on the raw products and each term is
// one fused multiply-add into the exponent.
template <typename T, int D, int RTW, bool FULL>
__device__ __forceinline__ void stats_block(const ScoreParams &p, const UnitInfo &u, const RowBlock<T, D, RTW> &rb,
                                            const unsigned char *stage, int kb, int col, int grp,
                                            float (&m)[RTW], float (&z)[RTW]) {
  using MF = Mfma<T>;
  using Cfg = ScoreCfg<T, D>;
  typename MF::frag kf[2][Cfg::steps];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) key_frags<T, D>(stage, kt, col, grp, kf[kt]);
  const float c = p.scale_log2;
#pragma unroll
  for (int k = 0; k < RTW; ++k) {
    f32x4_t s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < Cfg::steps; ++st) s[kt] = MF::mma(kf[kt][st], rb.q[k][st], s[kt]);
    }
    float v[8];
    bool vis[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[e] = s[e >> 2][e & 3];
      if constexpr (FULL) {
        vis[e] = true;
      } else {
        const int key = kb + (e >> 2) * 16 + 4 * grp + (e & 3);
        vis[e] = key < u.L && (!p.causal || key <= rb.pos[k]);
      }
    }
    if (c > 0.f) {
      float vmax = -INFINITY;
#pragma unroll
      for (int e = 0; e < 8; ++e) vmax = fmaxf(vmax, vis[e] ? v[e] : -INFINITY);
      const float mn = fmaxf(m[k], vmax * c);
      if (FULL || mn != -INFINITY) {
        float sum = z[k] * fast_exp2(m[k] - mn);
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += vis[e] ? fast_exp2(fmaf(v[e], c, -mn)) : 0.f;
        z[k] = sum;
        m[k] = mn;
      }
    } else {
      float x[8];
      float tmax = -INFINITY;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = vis[e] ? v[e] * c : -INFINITY;
        tmax = fmaxf(tmax, x[e]);
      }
      const float mn = fmaxf(m[k], tmax);
      if (FULL || mn != -INFINITY) {
        float sum = z[k] * fast_exp2(m[k] - mn);
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += fast_exp2(x[e] - mn);
        z[k] = sum;
        m[k] = mn;
      }
    }
  }
}

template <typename T, int D, int RTW>
__global__ __launch_bounds__(kThreads, 2) void score_stats_kernel(ScoreParams p) {
  constexpr int n_waves = kWaves;
  using Cfg = ScoreCfg<T, D>;
  using RB = RowBlock<T, D, RTW>;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][Cfg::stage_bytes];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  int chunk, unit;
  if (!xcd_chunk_unit(p, chunk, unit)) return;
  const UnitInfo u = unit_info(p, unit);
  const int k0 = chunk * kScoreChunk;
  if (k0 >= u.L) return;
  const int k1 = min(u.L, k0 + kScoreChunk);
  const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
  const int row_tiles = p.rows_pad / 16;
  // Keys every valid window row sees: below L, and (causal) up to L - w.
  const int full_end = p.causal ? min(u.L, u.L - p.w + 1) : u.L;

  for (int tg = 0; tg < row_tiles; tg += n_waves * RTW) {
    const int tile0 = tg + wave * RTW;   // tiles past row_tiles hold zero queries; never stored
    RB rb;
    rb.load(p, u, tile0, col, grp);
    float m[RTW], z[RTW];
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      m[k] = -INFINITY;
      z[k] = 0.f;
    }
    BlockRegs<T, D> regs;
    load_block<T, D>(regs, kbase, k0, u.L);
    int buf = 0;
    for (int kb = k0; kb < k1; kb += kBlock, buf ^= 1) {
      store_block<T, D>(stage[buf], regs);
      __syncthreads();   // block kb staged; every wave is done with the other buffer
      if (kb + kBlock < k1) load_block<T, D>(regs, kbase, kb + kBlock, u.L);
      if (kb + kBlock <= full_end)
        stats_block<T, D, RTW, true>(p, u, rb, stage[buf], kb, col, grp, m, z);
      else
        stats_block<T, D, RTW, false>(p, u, rb, stage[buf], kb, col, grp, m, z);
    }
    __syncthreads();   // the stage is reused by the next row-tile group
    // Merge the four lane groups that hold the same row, then store.
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      const float M = group4_max(m[k]);
      const float zz = (m[k] == -INFINITY) ? 0.f : z[k] * fast_exp2(m[k] - M);
      const float Z = group4_sum(zz);
      if (grp == 0 && tile0 + k < row_tiles) {
        const int r = (tile0 + k) * 16 + col;
        float *dst = p.row_part + ((u.ounit * p.chunks + chunk) * p.rows_pad + r) * 2;
        dst[0] = M;
        dst[1] = Z;
      }
    }
  }
}

// Mass pass body for one 32-key block: S = Q.K^T, lane holds rows
// (tile0 + k)*16 + 4*grp + i of key kb + kt*16 + col, so the lane sums its
// rows in registers and only the four lane groups meet at the end.  Both
// 16-key tiles are processed per row tile, so each row tile's normalisers are
// read from LDS once per block; each key's sum still runs over the rows in
// the same order.
template <typename T, int D, int RTW, bool FULL>
__device__ __forceinline__ void mass_block(const ScoreParams &p, const UnitInfo &u, const RowBlock<T, D, RTW> &rb,
                                           const unsigned char *stage, int kb, int tile0, int col, int grp,
                                           const float *smax, const float *sinv, float (&acc)[2]) {
  using MF = Mfma<T>;
  using Cfg = ScoreCfg<T, D>;
  typename MF::frag kf[2][Cfg::steps];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) key_frags<T, D>(stage, kt, col, grp, kf[kt]);
#pragma unroll
  for (int k = 0; k < RTW; ++k) {
    const float4 mx = *reinterpret_cast<const float4 *>(smax + k * 16 + 4 * grp);
    const float4 iv = *reinterpret_cast<const float4 *>(sinv + k * 16 + 4 * grp);
    const float rmax[4] = {mx.x, mx.y, mx.z, mx.w};
    const float rinv[4] = {iv.x, iv.y, iv.z, iv.w};
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int key = kb + kt * 16 + col;
      f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < Cfg::steps; ++c) s = MF::mma(rb.q[k][c], kf[kt][c], s);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = fast_exp2(fmaf(s[i], p.scale_log2, -rmax[i]));
        if constexpr (FULL) {
          acc[kt] = fmaf(e, rinv[i], acc[kt]);
        } else {
          const int r = (tile0 + k) * 16 + 4 * grp + i;
          const int pos = u.L - p.w + r % p.w;
          const bool vis = key < u.L && (!p.causal || key <= pos);
          acc[kt] += vis ? e * rinv[i] : 0.f;
        }
      }
    }
  }
}

template <typename T, int D, int RTW>
// Two workgroups per CU (two waves per SIMD): the window rows' normalisers sit
// in LDS rather than registers, which (with a small spill) fits 256 registers
// and measured faster than one wave per SIMD with everything in registers.
__global__ __launch_bounds__(kThreads, 2) void score_mass_kernel(ScoreParams p) {
  constexpr int n_waves = kWaves;
  using Cfg = ScoreCfg<T, D>;
  using RB = RowBlock<T, D, RTW>;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][Cfg::stage_bytes];
  __shared__ float part[kWaves][kScoreChunk];
  __shared__ __attribute__((aligned(16))) float s_max[kWaves * RTW * 16];
  __shared__ __attribute__((aligned(16))) float s_inv[kWaves * RTW * 16];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  int chunk, unit;
  if (!xcd_chunk_unit(p, chunk, unit)) return;
  const UnitInfo u = unit_info(p, unit);
  const int k0 = chunk * kScoreChunk;
  if (k0 >= u.L) return;
  const int k1 = min(u.L, k0 + kScoreChunk);
  const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
  const int row_tiles = p.rows_pad / 16;
  const int full_end = p.causal ? min(u.L, u.L - p.w + 1) : u.L;

  for (int tg = 0; tg < row_tiles; tg += n_waves * RTW) {
    const int tile0 = tg + wave * RTW;
    RB rb;
    rb.load(p, u, tile0, col, grp);
    // Normalisers of this group's rows, staged in LDS (absent rows: +inf, 0).
    for (int i = threadIdx.x; i < kWaves * RTW * 16; i += kThreads) {
      const int r = tg * 16 + i;
      const bool in = r < p.rows_pad;
      const float *st = p.row_stat + (u.ounit * p.rows_pad + (in ? r : 0)) * 2;
      s_max[i] = in ? st[0] : INFINITY;
      s_inv[i] = in ? st[1] : 0.f;
    }
    const float *smax = s_max + wave * RTW * 16;
    const float *sinv = s_inv + wave * RTW * 16;
    BlockRegs<T, D> regs;
    load_block<T, D>(regs, kbase, k0, u.L);
    int buf = 0;
    for (int kb = k0; kb < k1; kb += kBlock, buf ^= 1) {
      store_block<T, D>(stage[buf], regs);
      __syncthreads();   // block kb staged; every wave is done with the other buffer
      if (kb + kBlock < k1) load_block<T, D>(regs, kbase, kb + kBlock, u.L);
      float acc[2] = {0.f, 0.f};
      if (kb + kBlock <= full_end)
        mass_block<T, D, RTW, true>(p, u, rb, stage[buf], kb, tile0, col, grp, smax, sinv, acc);
      else
        mass_block<T, D, RTW, false>(p, u, rb, stage[buf], kb, tile0, col, grp, smax, sinv, acc);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const float tot = group4_sum_swap(acc[kt]);
        if (grp == 0) {
          // The first row group writes every column sum the final loop reads.
          if (tg == 0) part[wave][kb - k0 + kt * 16 + col] = tot;
          else part[wave][kb - k0 + kt * 16 + col] += tot;
        }
      }
    }
    __syncthreads();   // the stage is reused by the next row-tile group
  }
  __syncthreads();
  float *out = p.scores + u.ounit * p.cap;
  for (int j = threadIdx.x; j < k1 - k0; j += kThreads) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < n_waves; ++w) s += part[w][j];
    out[k0 + j] = s;
  }
}

// Row normalisers: (max, 1/sum) of every valid window row; absent rows get
// (+inf, 0) so that the mass pass adds exactly zero for them.
__global__ __launch_bounds__(kThreads) void score_rowmerge_kernel(ScoreParams p) {
  const UnitInfo u = unit_info(p, blockIdx.y);
  const int r = blockIdx.x * kThreads + threadIdx.x;
  if (r >= p.rows_pad) return;
  const int t = r % p.w;
  const bool valid = r < p.rows && u.L - p.w + t >= 0;
  const int active = (u.L + p.chunk_keys - 1) / p.chunk_keys;
  float M = -INFINITY;
  for (int c = 0; c < active; ++c) M = fmaxf(M, p.row_part[((u.ounit * p.chunks + c) * p.rows_pad + r) * 2]);
  double Z = 0.0;
  if (M != -INFINITY) {
    for (int c = 0; c < active; ++c) {
      const float *src = p.row_part + ((u.ounit * p.chunks + c) * p.rows_pad + r) * 2;
      if (src[0] != -INFINITY) Z += static_cast<double>(src[1]) * static_cast<double>(fast_exp2(src[0] - M));
    }
  }
  float *dst = p.row_stat + (u.ounit * p.rows_pad + r) * 2;
  const bool ok = valid && M != -INFINITY && Z > 0.0;
  dst[0] = ok ? M : INFINITY;
  dst[1] = ok ? static_cast<float>(1.0 / Z) : 0.f;
}

// Row normalisers taken from the decode steps of the window tokens: the
// (max, sum) pair decode wrote for query head g at position L - w + t is row
// g * w + t's statistic; absent or empty rows get (+inf, 0) as above.
__global__ __launch_bounds__(kThreads) void score_given_stats_kernel(ScoreParams p) {
  const UnitInfo u = unit_info(p, blockIdx.y);
  const int r = blockIdx.x * kThreads + threadIdx.x;
  if (r >= p.rows_pad) return;
  const int g = r / p.w;
  const int t = r - g * p.w;
  const bool valid = r < p.rows && u.L - p.w + t >= 0;
  float M = INFINITY, Z = 0.f;
  if (valid) {
    const float *src =
        p.given + ((((static_cast<size_t>(u.lc) * p.batch + u.b) * p.hq + u.h * p.group + g) * p.w) + t) * 2;
    M = src[0];
    Z = src[1];
  }
  const bool ok = valid && M != -INFINITY && M != INFINITY && Z > 0.f;
  float *dst = p.row_stat + (u.ounit * p.rows_pad + r) * 2;
  dst[0] = ok ? M : INFINITY;
  dst[1] = ok ? 1.f / Z : 0.f;
}


// ---------------------------------------------------------------------------
// Key-split kernels.  One workgroup of eight waves (two per SIMD) per CU,
// resident for the whole call; the unit's window rows Q (and, for the mass
// pass, each row's normaliser) are staged in LDS once per segment, and every
// wave then walks its own groups of 64 keys: the group's K fragments are
// loaded from global memory straight into registers in the MFMA operand
// layout (the next group's while the current one is computed) and multiplied
// against every row tile of Q read from LDS.  No barrier is needed inside the
// key loop, and a wave covers all window rows of its keys, so each score is
// summed in registers and written once.  Fragment element e of lane group grp
// in step c is contraction index (4c + grp) * kpl + e, the same for Q and K,
// so the four lane groups of a key read 4 * 16 consecutive bytes of its row
// per load.
// ---------------------------------------------------------------------------
constexpr int kV2Waves = 8;
constexpr int kV2Threads = kV2Waves * kWave;
constexpr int kV2KT = 4;                  // 16-key tiles per wave group
constexpr int kV2Group = kV2KT * 16;      // keys per wave group

// The K fragments of one wave group and the Q fragments of one row tile.
template <typename T, int D>
struct V2Keys {
  static constexpr int steps = D / (4 * Mfma<T>::kPerLane);
  typename Mfma<T>::frag k[kV2KT][steps];
};
template <typename T, int D>
struct V2Rows {
  static constexpr int steps = D / (4 * Mfma<T>::kPerLane);
  typename Mfma<T>::frag q[steps];
};

template <typename T, int D, int RTM>
struct V2Cfg {
  using MF = Mfma<T>;
  using frag = typename MF::frag;
  static constexpr int kpl = MF::kPerLane;
  static constexpr int steps = D / (4 * kpl);           // MFMAs per 16x16 tile
  static constexpr int row_bytes = D * (int)sizeof(T);
  static constexpr int q_stride = row_bytes + 16;       // padded LDS pitch of a window row
  static constexpr int max_rows = 16 * RTM;
  static constexpr int q_bytes = max_rows * q_stride;
  static constexpr int merge_bytes = kV2Waves * max_rows * 2 * 4;   // per-wave row (reference, sum) of the statistics
  static constexpr int const_bytes = max_rows * 2 * 4;             // row (max, 1/sum) of the mass pass
  static constexpr int stage_bytes = q_bytes;
  static constexpr int lds_bytes = q_bytes + (merge_bytes > const_bytes ? merge_bytes : const_bytes);
};

// Window rows of the unit into LDS (rows that do not exist are zero).  A
// thread's loads go out in two batches, each issued before its stores, so
// the staging costs two memory round trips and few registers; absent rows
// load the unit's first window row (always a valid address) and store zero.
template <typename T, int D, int RTM>
__device__ __forceinline__ void v2_stage_window(const ScoreParams &p, const UnitInfo &u, unsigned char *qs) {
  using C = V2Cfg<T, D, RTM>;
  constexpr int pieces = C::row_bytes / 16;
  constexpr int per_thread = (C::max_rows * pieces + kV2Threads - 1) / kV2Threads;
  constexpr int half = (per_thread + 1) / 2;
  const unsigned char *base = reinterpret_cast<const unsigned char *>(p.q_win) +
      (((size_t)u.lc * p.batch + u.b) * p.hq + (size_t)u.h * p.group) * p.w * (size_t)C::row_bytes;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint4 v[half];
    bool ok[half];
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const int i = (h * half + j) * kV2Threads + static_cast<int>(threadIdx.x);
      const int r = i / pieces;
      const int pc = i - r * pieces;
      const int g = r / p.w;
      const int t = r - g * p.w;
      ok[j] = (h * half + j < per_thread) && r < p.rows && u.L - p.w + t >= 0;
      // row g * w + t of the unit's group is window row t of query head h * G + g
      const size_t off = ok[j] ? (static_cast<size_t>(r) * C::row_bytes + pc * 16) : 0;
      v[j] = *reinterpret_cast<const uint4 *>(base + off);
    }
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const int i = (h * half + j) * kV2Threads + static_cast<int>(threadIdx.x);
      const int r = i / pieces;
      if (h * half + j < per_thread)
        *reinterpret_cast<uint4 *>(qs + r * C::q_stride + (i - r * pieces) * 16) = ok[j] ? v[j] : make_uint4(0, 0, 0, 0);
    }
  }
}

// K fragments of the wave group at g0 (keys at or past L read row 0 of the
// unit and are masked by the caller).
template <typename T, int D>
__device__ __forceinline__ void v2_load_keys(V2Keys<T, D> &kf, const T *kbase, int g0, int L, int col, int grp) {
  constexpr int kpl = Mfma<T>::kPerLane;
#pragma unroll
  for (int kt = 0; kt < kV2KT; ++kt) {
    const int key = g0 + kt * 16 + col;
    const T *src = kbase + static_cast<size_t>(key < L ? key : 0) * D + grp * kpl;
#pragma unroll
    for (int c = 0; c < V2Keys<T, D>::steps; ++c) kf.k[kt][c] = load_frag(src + c * 4 * kpl);
  }
}

template <typename T, int D>
__device__ __forceinline__ void v2_load_q(V2Rows<T, D> &qf, const unsigned char *qs, int rt, int col, int grp) {
  constexpr int kpl = Mfma<T>::kPerLane;
  constexpr int q_stride = D * (int)sizeof(T) + 16;
  const T *row = reinterpret_cast<const T *>(qs + (rt * 16 + col) * q_stride) + grp * kpl;
#pragma unroll
  for (int c = 0; c < V2Rows<T, D>::steps; ++c) qf.q[c] = load_frag(row + c * 4 * kpl);
}

// Mass of one row tile for one wave group: S = Q.K^T, lane (col, grp) holds
// rows 16 rt + 4 grp + i of key g0 + 16 kt + col and adds exp2(x - max) / sum
// of those rows into acc[kt].
template <typename T, int D, bool FULL>
__device__ __forceinline__ void v2_mass_tile(const ScoreParams &p, const UnitInfo &u, const V2Rows<T, D> &qf,
                                             const float4 mx, const float4 iv, const V2Keys<T, D> &kf, int g0,
                                             int rt, int col, int grp, float (&acc)[kV2KT]) {
  using MF = Mfma<T>;
  const float rmax[4] = {mx.x, mx.y, mx.z, mx.w};
  const float rinv[4] = {iv.x, iv.y, iv.z, iv.w};
#pragma unroll
  for (int kt = 0; kt < kV2KT; ++kt) {
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < V2Keys<T, D>::steps; ++c) s = MF::mma(qf.q[c], kf.k[kt][c], s);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float e = fast_exp2(fmaf(s[i], p.scale_log2, -rmax[i]));
      if constexpr (FULL) {
        acc[kt] = fmaf(e, rinv[i], acc[kt]);
      } else {
        const int r = rt * 16 + 4 * grp + i;
        const int pos = u.L - p.w + r % p.w;
        const int key = g0 + kt * 16 + col;
        const bool vis = key < u.L && (!p.causal || key <= pos);
        acc[kt] += vis ? e * rinv[i] : 0.f;
      }
    }
  }
}

template <typename T, int D, bool FULL>
__device__ __forceinline__ void v2_mass_group(const ScoreParams &p, const UnitInfo &u, const unsigned char *qs,
                                              const float *cmx, const float *cin, const V2Keys<T, D> &kf, int g0,
                                              int row_tiles, int col, int grp, float (&acc)[kV2KT]) {
  for (int rt = 0; rt < row_tiles; rt += 2) {
    V2Rows<T, D> qa, qb;
    v2_load_q<T, D>(qa, qs, rt, col, grp);
    v2_load_q<T, D>(qb, qs, rt + 1, col, grp);
    const float4 ma = *reinterpret_cast<const float4 *>(cmx + rt * 16 + 4 * grp);
    const float4 ia = *reinterpret_cast<const float4 *>(cin + rt * 16 + 4 * grp);
    const float4 mb = *reinterpret_cast<const float4 *>(cmx + rt * 16 + 16 + 4 * grp);
    const float4 ib = *reinterpret_cast<const float4 *>(cin + rt * 16 + 16 + 4 * grp);
    v2_mass_tile<T, D, FULL>(p, u, qa, ma, ia, kf, g0, rt, col, grp, acc);
    v2_mass_tile<T, D, FULL>(p, u, qb, mb, ib, kf, g0, rt + 1, col, grp, acc);
  }
}

// Work of the key-split kernels: the non-empty chunks of chunk_keys keys of
// every unit (a unit of length L has ceil(L / chunk_keys) of them), taken
// unit-major.  The grid is persistent (one workgroup per CU, all resident for
// the whole call) and workgroup b takes an equal share of those chunks, a
// contiguous run [c_begin, c_end) of the global order; it walks the run as
// segments, the maximal pieces inside one unit, so the window rows are
// staged once per segment and a segment's key loop needs no barrier.
struct V2Run {
  int unit;       // unit of the run's first chunk
  int chunk;      // that chunk's index within its unit
  long long n;    // chunks in the run
};

// Every workgroup scans the units' lengths (a block-wide prefix sum of the
// chunk counts) to find where its share starts.  `scan` is LDS scratch of
// kV2Threads + 2 entries.
__device__ V2Run v2_run(const ScoreParams &p, long long *scan) {
  const int units = p.n_layers * p.batch * p.hkv;
  const int per_t = (units + kV2Threads - 1) / kV2Threads;
  const int u0 = min(units, static_cast<int>(threadIdx.x) * per_t);
  const int u1 = min(units, u0 + per_t);
  long long mine = 0;
  for (int u = u0; u < u1; ++u) mine += (unit_info(p, u).L + p.chunk_keys - 1) / p.chunk_keys;
  scan[threadIdx.x] = mine;
  __syncthreads();
  // Inclusive scan (Hillis-Steele) over the thread totals.
  for (int off = 1; off < kV2Threads; off <<= 1) {
    const long long v = static_cast<int>(threadIdx.x) >= off ? scan[threadIdx.x - off] : 0;
    __syncthreads();
    scan[threadIdx.x] += v;
    __syncthreads();
  }
  const long long total = scan[kV2Threads - 1];
  const long long b0 = total * blockIdx.x / gridDim.x;
  const long long b1 = total * (blockIdx.x + 1) / gridDim.x;
  const long long before = threadIdx.x ? scan[threadIdx.x - 1] : 0;
  __syncthreads();
  if (threadIdx.x == 0) {
    scan[kV2Threads] = units;            // no chunk of this run: past the last unit
    scan[kV2Threads + 1] = 0;
  }
  __syncthreads();
  if (b0 < b1 && before <= b0 && b0 < before + mine) {
    long long c = before;
    for (int u = u0; u < u1; ++u) {
      const int nc = (unit_info(p, u).L + p.chunk_keys - 1) / p.chunk_keys;
      if (b0 < c + nc) {
        scan[kV2Threads] = u;
        scan[kV2Threads + 1] = static_cast<int>(b0 - c);
        break;
      }
      c += nc;
    }
  }
  __syncthreads();
  V2Run r;
  r.unit = static_cast<int>(scan[kV2Threads]);
  r.chunk = static_cast<int>(scan[kV2Threads + 1]);
  r.n = b1 - b0;
  __syncthreads();                       // the scratch is reused by the caller
  return r;
}

// Next segment of a run: chunks [c0, c1) of `unit`, consuming them from the
// run.  Returns false when the run is exhausted.
__device__ __forceinline__ bool v2_next_segment(const ScoreParams &p, V2Run &r, int &unit, int &c0, int &c1) {
  const int units = p.n_layers * p.batch * p.hkv;
  while (r.n > 0 && r.unit < units) {
    const int nc = (unit_info(p, r.unit).L + p.chunk_keys - 1) / p.chunk_keys;
    if (r.chunk < nc) {
      const long long take = min(static_cast<long long>(nc - r.chunk), r.n);
      unit = r.unit;
      c0 = r.chunk;
      c1 = r.chunk + static_cast<int>(take);
      r.n -= take;
      r.chunk = 0;
      ++r.unit;
      return true;
    }
    r.chunk = 0;
    ++r.unit;
  }
  return false;
}

template <typename T, int D, int RTM>
__global__ __launch_bounds__(kV2Threads, 1) void score_mass_v2_kernel(ScoreParams p) {
  using C = V2Cfg<T, D, RTM>;
  __shared__ __attribute__((aligned(16))) unsigned char smem[C::lds_bytes];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  unsigned char *qs = smem;
  V2Run run = v2_run(p, reinterpret_cast<long long *>(smem));
  float *cmx = reinterpret_cast<float *>(smem + C::stage_bytes);
  float *cin = cmx + C::max_rows;
  const int row_tiles = (p.rows_pad / 16 + 1) & ~1;
  constexpr int stride = kV2Waves * kV2Group;
  int sunit, sc0, sc1;
  while (v2_next_segment(p, run, sunit, sc0, sc1)) {
    const UnitInfo u = unit_info(p, sunit);
    const int k0 = sc0 * p.chunk_keys;
    const int k1 = min(u.L, sc1 * p.chunk_keys);
    const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
    __syncthreads();                        // every wave is done with the previous segment's rows
    v2_stage_window<T, D, RTM>(p, u, qs);
    for (int r = threadIdx.x; r < row_tiles * 16; r += kV2Threads) {
      const bool in = r < p.rows_pad;
      const float *st = p.row_stat + (u.ounit * p.rows_pad + (in ? r : 0)) * 2;
      cmx[r] = in ? st[0] : INFINITY;
      cin[r] = in ? st[1] : 0.f;
    }
    int g0 = k0 + wave * kV2Group;
    V2Keys<T, D> kf;
    v2_load_keys<T, D>(kf, kbase, g0 < k1 ? g0 : k0, u.L, col, grp);
    __syncthreads();
    const int full_end = p.causal ? min(u.L, u.L - p.w + 1) : u.L;
    float *out = p.scores + u.ounit * p.cap;
    for (; g0 < k1; g0 += stride) {
      V2Keys<T, D> kn;
      const int gn = g0 + stride;
      v2_load_keys<T, D>(kn, kbase, gn < k1 ? gn : g0, u.L, col, grp);
      float acc[kV2KT] = {0.f, 0.f, 0.f, 0.f};
      if (g0 + kV2Group <= full_end)
        v2_mass_group<T, D, true>(p, u, qs, cmx, cin, kf, g0, row_tiles, col, grp, acc);
      else
        v2_mass_group<T, D, false>(p, u, qs, cmx, cin, kf, g0, row_tiles, col, grp, acc);
#pragma unroll
      for (int kt = 0; kt < kV2KT; ++kt) {
        const float tot = group4_sum_swap(acc[kt]);
        const int key = g0 + kt * 16 + col;
        if (grp == 0 && key < k1) out[key] = tot;
      }
      kf = kn;
    }
  }
}

// Statistics of one row tile for one wave group: S^T = K.Q^T, lane (col,
// grp) holds keys g0 + 16 kt + 4 grp + i of row 16 rt + col.  Each wave keeps,
// per window row, a reference m and the sum z of 2^(x - m) over its keys in
// LDS (mrow, zrow).  On the wave's first group (MODE 0) m is the row's
// largest logit among the group's first 16 keys, so the largest term of
// every sum is at least 1, and later groups (MODE 1) only add terms, with no
// running maximum.  A logit more than about 120 above m overflows a sum;
// the caller then redoes the wave's keys with a running maximum (MODE 2).
template <typename T, int D, bool FULL, int MODE>
__device__ __forceinline__ void v2_stats_tile(const ScoreParams &p, const UnitInfo &u, const V2Rows<T, D> &qf,
                                              const V2Keys<T, D> &kf, int g0, int rt, int col, int grp, float m_in,
                                              float z_in, float *mrow, float *zrow) {
  using MF = Mfma<T>;
  const float c = p.scale_log2;
  const int r = rt * 16 + col;
  f32x4_t s[kV2KT];
#pragma unroll
  for (int kt = 0; kt < kV2KT; ++kt) {
    s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < V2Keys<T, D>::steps; ++cc) s[kt] = MF::mma(kf.k[kt][cc], qf.q[cc], s[kt]);
  }
  bool vis[kV2KT][4];
  const int pos = u.L - p.w + r % p.w;
#pragma unroll
  for (int kt = 0; kt < kV2KT; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (FULL) {
        vis[kt][i] = true;
      } else {
        const int key = g0 + kt * 16 + 4 * grp + i;
        vis[kt][i] = key < u.L && (!p.causal || key <= pos);
      }
    }
  float m = m_in, zold = z_in;
  if constexpr (MODE == 0) {
    float lm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) lm = fmaxf(lm, vis[0][i] ? s[0][i] * c : -INFINITY);
    m = group4_max(lm);
    zold = 0.f;
  } else if constexpr (MODE == 2) {
    float lm = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < kV2KT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) lm = fmaxf(lm, vis[kt][i] ? s[kt][i] * c : -INFINITY);
    const float mn = fmaxf(m_in, group4_max(lm));
    zold = (m_in == -INFINITY || mn == -INFINITY) ? 0.f : z_in * fast_exp2(m_in - mn);
    m = mn;
  }
  float zz = 0.f;
  if (MODE != 2 || m != -INFINITY) {
#pragma unroll
    for (int kt = 0; kt < kV2KT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = fast_exp2(fmaf(s[kt][i], c, -m));
        if constexpr (FULL) zz += e;
        else zz += vis[kt][i] ? e : 0.f;
      }
  }
  const float zsum = group4_sum_swap(zz);
  if (grp == 0) {
    mrow[r] = m;
    zrow[r] = zold + zsum;
  }
}

template <typename T, int D, bool FULL, int MODE>
__device__ __forceinline__ void v2_stats_group(const ScoreParams &p, const UnitInfo &u, const unsigned char *qs,
                                               const V2Keys<T, D> &kf, int g0, int row_tiles, int col, int grp,
                                               float *mrow, float *zrow) {
  for (int rt = 0; rt < row_tiles; rt += 2) {
    V2Rows<T, D> qa, qb;
    v2_load_q<T, D>(qa, qs, rt, col, grp);
    v2_load_q<T, D>(qb, qs, rt + 1, col, grp);
    float ma = 0.f, za = 0.f, mb = 0.f, zb = 0.f;
    if constexpr (MODE != 0) {
      ma = mrow[rt * 16 + col];
      za = zrow[rt * 16 + col];
      mb = mrow[rt * 16 + 16 + col];
      zb = zrow[rt * 16 + 16 + col];
    }
    v2_stats_tile<T, D, FULL, MODE>(p, u, qa, kf, g0, rt, col, grp, ma, za, mrow, zrow);
    v2_stats_tile<T, D, FULL, MODE>(p, u, qb, kf, g0, rt + 1, col, grp, mb, zb, mrow, zrow);
  }
}

// All groups of a wave's keys; ONLINE selects the running-maximum form.
template <typename T, int D, bool ONLINE>
__device__ __forceinline__ void v2_stats_keys(const ScoreParams &p, const UnitInfo &u, const unsigned char *qs,
                                              const T *kbase, int gstart, int k1, int full_end, int row_tiles,
                                              int col, int grp, float *mrow, float *zrow) {
  constexpr int stride = kV2Waves * kV2Group;
  V2Keys<T, D> kf;
  v2_load_keys<T, D>(kf, kbase, gstart < k1 ? gstart : 0, u.L, col, grp);
  bool first = true;
  for (int g0 = gstart; g0 < k1; g0 += stride) {
    V2Keys<T, D> kn;
    const int gn = g0 + stride;
    v2_load_keys<T, D>(kn, kbase, gn < k1 ? gn : g0, u.L, col, grp);
    const bool full = g0 + kV2Group <= full_end;
    if constexpr (ONLINE) {
      if (full) v2_stats_group<T, D, true, 2>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
      else v2_stats_group<T, D, false, 2>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
    } else if (first) {
      if (full) v2_stats_group<T, D, true, 0>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
      else v2_stats_group<T, D, false, 0>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
    } else {
      if (full) v2_stats_group<T, D, true, 1>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
      else v2_stats_group<T, D, false, 1>(p, u, qs, kf, g0, row_tiles, col, grp, mrow, zrow);
    }
    first = false;
    kf = kn;
  }
}

template <typename T, int D, int RTM>
__global__ __launch_bounds__(kV2Threads, 1) void score_stats_v2_kernel(ScoreParams p) {
  using C = V2Cfg<T, D, RTM>;
  __shared__ __attribute__((aligned(16))) unsigned char smem[C::q_bytes + C::merge_bytes];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  unsigned char *qs = smem;
  V2Run run = v2_run(p, reinterpret_cast<long long *>(smem));
  float *mrow_all = reinterpret_cast<float *>(smem + C::q_bytes);        // [wave][max_rows]
  float *zrow_all = mrow_all + kV2Waves * C::max_rows;                   // [wave][max_rows]
  float *mrow = mrow_all + wave * C::max_rows;
  float *zrow = zrow_all + wave * C::max_rows;
  const int row_tiles = (p.rows_pad / 16 + 1) & ~1;          // even; a pad tile is never reported
  int sunit, sc0, sc1;
  while (v2_next_segment(p, run, sunit, sc0, sc1)) {
    const UnitInfo u = unit_info(p, sunit);
    const int k0 = sc0 * p.chunk_keys;
    const int k1 = min(u.L, sc1 * p.chunk_keys);
    const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
    __syncthreads();                        // the previous segment's rows and partials are consumed
    v2_stage_window<T, D, RTM>(p, u, qs);
    for (int r = lane; r < C::max_rows; r += kWave) {   // a wave without keys reports empty rows
      mrow[r] = -INFINITY;
      zrow[r] = 0.f;
    }
    __syncthreads();
    const int full_end = p.causal ? min(u.L, u.L - p.w + 1) : u.L;
    const int g0 = k0 + wave * kV2Group;
    v2_stats_keys<T, D, false>(p, u, qs, kbase, g0, k1, full_end, row_tiles, col, grp, mrow, zrow);
    bool bad = false;
    for (int r = lane; r < row_tiles * 16; r += kWave) bad |= !(zrow[r] <= 3.402823466e38f);
    if (__any(bad)) {          // a sum overflowed against its reference: redo with a running maximum
      for (int r = lane; r < row_tiles * 16; r += kWave) {
        mrow[r] = -INFINITY;
        zrow[r] = 0.f;
      }
      v2_stats_keys<T, D, true>(p, u, qs, kbase, g0, k1, full_end, row_tiles, col, grp, mrow, zrow);
    }
    __syncthreads();
    // The segment's partial goes to its first chunk slot; its other slots are
    // marked empty, so the row merge reads every slot it covers.
    const int n_out = (sc1 - sc0) * p.rows_pad;
    for (int i = threadIdx.x; i < n_out; i += kV2Threads) {
      const int cs = sc0 + i / p.rows_pad;
      const int r = i - (cs - sc0) * p.rows_pad;
      float M = -INFINITY, Z = 0.f;
      if (cs == sc0) {
#pragma unroll
        for (int w = 0; w < kV2Waves; ++w) M = fmaxf(M, mrow_all[w * C::max_rows + r]);
        if (M != -INFINITY) {
#pragma unroll
          for (int w = 0; w < kV2Waves; ++w) {
            const float mw = mrow_all[w * C::max_rows + r];
            if (mw != -INFINITY) Z += zrow_all[w * C::max_rows + r] * fast_exp2(mw - M);
          }
        }
      }
      float *dst = p.row_part + ((u.ounit * p.chunks + cs) * p.rows_pad + r) * 2;
      dst[0] = M;
      dst[1] = Z;
    }
  }
}

// One resident workgroup per CU (the LDS of one holds the window rows).
inline int v2_grid(const ScoreParams &p, int units) {
  const long long n_items = static_cast<long long>(units) * p.chunks;   // at least the non-empty chunks
  return static_cast<int>(n_items < p.cus ? n_items : p.cus);
}

template <typename T, int D, int RTM>
hipError_t launch_v2(ScoreParams p, int units, hipStream_t s) {
  hipError_t e;
  if (p.given) {
    hipLaunchKernelGGL(score_given_stats_kernel, dim3((p.rows_pad + kThreads - 1) / kThreads, units), dim3(kThreads),
                       0, s, p);
  } else {
    hipLaunchKernelGGL((score_stats_v2_kernel<T, D, RTM>), dim3(v2_grid(p, units)), dim3(kV2Threads), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_rowmerge_kernel, dim3((p.rows_pad + kThreads - 1) / kThreads, units), dim3(kThreads), 0,
                       s, p);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_mass_v2_kernel<T, D, RTM>), dim3(v2_grid(p, units)), dim3(kV2Threads), 0, s, p);
  return hipGetLastError();
}

// Row tiles the key-split kernels are built for, and whether the window rows
// and their normalisers fit the LDS of one CU at that size.
template <typename T, int D, int RTM>
constexpr bool v2_fits() {
  // fp32 at head_dim 128 needs 128 registers per key group and spills: the
  // row-split kernels serve it.
  return V2Cfg<T, D, RTM>::lds_bytes <= 160 * 1024 && !(sizeof(T) == 4 && D == 128);
}

template <typename T, int D>
hipError_t try_launch_v2(const ScoreParams &p0, hipStream_t s, bool &done) {
  done = false;
  const int units = p0.n_layers * p0.batch * p0.hkv;
  const int row_tiles = p0.rows_pad / 16;
  ScoreParams p = p0;
  // Keys per workgroup: 1024, or 2048 when that still gives every CU many workgroups.
  // Chunks are the unit of load balance over the persistent grid: 512 keys
  // when the call is small (a few chunks per CU would leave the shares
  // uneven), 1024 otherwise (fewer per-chunk statistics for the row merge).
  p.chunk_keys = 1024;
  if (static_cast<long long>(units) * ((p.cap + 511) / 512) <= 64LL * p.cus) p.chunk_keys = 512;
  p.chunks = (p.cap + p.chunk_keys - 1) / p.chunk_keys;
  done = true;
  if constexpr (v2_fits<T, D, 8>()) {
    if (row_tiles <= 8) return launch_v2<T, D, 8>(p, units, s);
  }
  if constexpr (v2_fits<T, D, 16>()) {
    if (row_tiles <= 16) return launch_v2<T, D, 16>(p, units, s);
  }
  if constexpr (v2_fits<T, D, 28>()) {
    if (row_tiles <= 28) return launch_v2<T, D, 28>(p, units, s);
  }
  if constexpr (v2_fits<T, D, 34>()) {
    if (row_tiles <= 34) return launch_v2<T, D, 34>(p, units, s);
  }
  done = false;
  return hipSuccess;
}

template <typename T, int D, int RTW>
hipError_t launch_rtw(const ScoreParams &p, int waves, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  hipError_t e;
  if (p.given) {
    hipLaunchKernelGGL(score_given_stats_kernel, dim3((p.rows_pad + kThreads - 1) / kThreads, units), dim3(kThreads),
                       0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else {
    hipLaunchKernelGGL((score_stats_kernel<T, D, RTW>), dim3(8 * p.chunks, (units + 7) / 8), dim3(waves * kWave), 0, s,
                       p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_rowmerge_kernel, dim3((p.rows_pad + kThreads - 1) / kThreads, units), dim3(kThreads), 0,
                       s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((score_mass_kernel<T, D, RTW>), dim3(8 * p.chunks, (units + 7) / 8), dim3(waves * kWave), 0, s,
                     p);
  return hipGetLastError();
}

// Row tiles per wave: the four waves split the G * w window rows evenly, up
// to eight 16-row tiles each (more rows loop over groups of 32 tiles).  Each
// staged K fragment then feeds up to eight MFMA tiles; spreading the rows
// over more waves (4 tiles each) measured 1.4x slower on the 7B window
// (448 rows) despite the higher occupancy.
template <typename T, int D>
hipError_t launch_typed(const ScoreParams &p, hipStream_t s) {
  bool done = false;
  const hipError_t e2 = try_launch_v2<T, D>(p, s, done);
  if (done) return e2;
  const int row_tiles = p.rows_pad / 16;
  switch ((row_tiles + kWaves - 1) / kWaves) {
    case 1: return launch_rtw<T, D, 1>(p, kWaves, s);
    case 2: return launch_rtw<T, D, 2>(p, kWaves, s);
    case 3: return launch_rtw<T, D, 3>(p, kWaves, s);
    case 4: return launch_rtw<T, D, 4>(p, kWaves, s);
    case 5: return launch_rtw<T, D, 5>(p, kWaves, s);
    case 6: return launch_rtw<T, D, 6>(p, kWaves, s);
    case 7: return launch_rtw<T, D, 7>(p, kWaves, s);
    default: return launch_rtw<T, D, 8>(p, kWaves, s);
  }
}

}  // namespace

size_t score_workspace_bytes(int units, int capacity, int rows) {
  const size_t rows_pad = static_cast<size_t>((rows + 15) / 16 * 16);
  const size_t chunks = static_cast<size_t>((capacity + kScoreChunk - 1) / kScoreChunk);
  return static_cast<size_t>(units) * rows_pad * (chunks + 1) * 2 * sizeof(float);
}

hipError_t launch_score(const ScoreParams &p, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0) {
    if (head_dim == 64) return launch_typed<float, 64>(p, s);
    return launch_typed<float, 128>(p, s);
  }
  if (head_dim == 64) return launch_typed<bf16_t, 64>(p, s);
  return launch_typed<bf16_t, 128>(p, s);
}

}  // namespace reco
