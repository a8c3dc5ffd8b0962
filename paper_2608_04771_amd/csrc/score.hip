// Window attention-mass scoring of every cached key (Eq. 2), gfx950.
//
// For one unit (layer, sequence, kv head h) the window rows are the G * w
// (query head of h's group, window position) pairs.  Row r = g * w + t is the
// query of head h*G + g at absolute position pos = L - w + t.  Three kernels:
//   1. score_stats: per (unit, 512-key chunk), the fp32 running (max, sum of
//      exp) of every window row over the chunk's keys (log2 domain), with
//      S^T = K.Q^T so that a lane holds four keys of one row;
//   2. score_rowmerge: per (unit, row), merge the chunk statistics into the
//      row's softmax normaliser (max, 1/sum);
//   3. score_mass: per (unit, chunk), recompute the logits as S = Q.K^T (a
//      lane holds four rows of one key, summed in registers) and add
//      exp2(x - max) / sum over all rows of each key; the waves' column sums
//      meet in LDS, so each score is written once, deterministically.
// Logits are S^T = K . Q^T on the matrix cores (16 keys x 16 rows per MFMA,
// bf16 products accumulated in fp32); each wave owns a slice of row tiles
// whose Q fragments stay in registers while the chunk's keys stream past.
// The workgroup reads each 32-key block of K once, with coalesced
// non-temporal loads (prefetched one block ahead), into a double-buffered
// LDS stage that all its waves read in the MFMA operand layout.  Blocks
// that every window row sees in full take a mask-free path; only the blocks
// that reach into the window or past the end of the cache test each key.
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
  const int active = (u.L + kScoreChunk - 1) / kScoreChunk;
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
