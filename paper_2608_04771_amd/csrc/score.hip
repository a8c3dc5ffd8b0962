// Window attention-mass scoring of every cached key (Eq. 2), gfx950.
//
// For one unit (layer, sequence, kv head h) the window rows are the G * w
// (query head of h's group, window position) pairs.  Row r = g * w + t is the
// query of head h*G + g at absolute position pos = L - w + t.  Three kernels:
//   1. score_stats: per (unit, 512-key chunk), the fp32 running (max, sum of
//      exp) of every window row over the chunk's keys (log2 domain);
//   2. score_rowmerge: per (unit, row), merge the chunk statistics into the
//      row's softmax normaliser (max, 1/sum);
//   3. score_mass: per (unit, chunk), recompute the logits and add
//      exp2(x - max) / sum over all rows of each key; the four waves' column
//      sums meet in LDS, so each score is written once, deterministically.
// Logits are S^T = K . Q^T on the matrix cores (16 keys x 16 rows per MFMA,
// bf16 products accumulated in fp32); each wave owns a slice of row tiles
// whose Q fragments stay in registers while the chunk's keys stream past.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

#include <math.h>

namespace reco {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kKeyTile = 16;

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

template <typename T, int D, int RTW>
struct RowBlock {
  using MF = Mfma<T>;
  using frag = typename MF::frag;
  static constexpr int dq = D / 4;
  static constexpr int steps = dq / MF::kPerLane;
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
                       (valid[k] ? t : 0)) * D + grp * dq;
#pragma unroll
      for (int c = 0; c < steps; ++c)
        q[k][c] = valid[k] ? load_frag(qrow + c * MF::kPerLane) : zero_frag(frag{});
    }
  }
};

template <typename T, int D>
__device__ __forceinline__ void load_key_tile(const T *kbase, int kb, int L, int col, int grp,
                                              typename Mfma<T>::frag (&kf)[D / 4 / Mfma<T>::kPerLane]) {
  const int key = kb + col;
  const T *row = kbase + static_cast<size_t>(key < L ? key : 0) * D + grp * (D / 4);
#pragma unroll
  for (int c = 0; c < D / 4 / Mfma<T>::kPerLane; ++c) kf[c] = load_frag(row + c * Mfma<T>::kPerLane);
}

template <typename T, int D, int RTW>
__global__ __launch_bounds__(kThreads) void score_stats_kernel(ScoreParams p) {
  using MF = Mfma<T>;
  using RB = RowBlock<T, D, RTW>;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  const int chunk = blockIdx.x;
  const UnitInfo u = unit_info(p, blockIdx.y);
  const int k0 = chunk * kScoreChunk;
  if (k0 >= u.L) return;
  const int k1 = min(u.L, k0 + kScoreChunk);
  const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
  const int row_tiles = p.rows_pad / 16;

  for (int tg = 0; tg < row_tiles; tg += kWaves * RTW) {
    const int tile0 = tg + wave * RTW;
    RB rb;
    rb.load(p, u, tile0, col, grp);
    float m[RTW], z[RTW];
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      m[k] = -INFINITY;
      z[k] = 0.f;
    }
    for (int kb = k0; kb < k1; kb += kKeyTile) {
      typename MF::frag kf[RB::steps];
      load_key_tile<T, D>(kbase, kb, u.L, col, grp, kf);
#pragma unroll
      for (int k = 0; k < RTW; ++k) {
        if (tile0 + k >= row_tiles) break;
        f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < RB::steps; ++c) s = MF::mma(kf[c], rb.q[k][c], s);
        float x[4];
        float tmax = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kb + 4 * grp + i;
          const bool vis = key < u.L && (!p.causal || key <= rb.pos[k]);
          x[i] = vis ? s[i] * p.scale_log2 : -INFINITY;
          tmax = fmaxf(tmax, x[i]);
        }
        const float mn = fmaxf(m[k], tmax);
        if (mn != -INFINITY) {
          float acc = z[k] * fast_exp2(m[k] - mn);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc += fast_exp2(x[i] - mn);
          z[k] = acc;
          m[k] = mn;
        }
      }
    }
    // Merge the four lane groups that hold the same row, then store.
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      if (tile0 + k >= row_tiles) break;
      const float M = group4_max(m[k]);
      const float zz = (m[k] == -INFINITY) ? 0.f : z[k] * fast_exp2(m[k] - M);
      const float Z = group4_sum(zz);
      if (grp == 0) {
        const int r = (tile0 + k) * 16 + col;
        float *dst = p.row_part + ((u.ounit * p.chunks + chunk) * p.rows_pad + r) * 2;
        dst[0] = M;
        dst[1] = Z;
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void score_rowmerge_kernel(ScoreParams p) {
  const UnitInfo u = unit_info(p, blockIdx.y);
  const int r = blockIdx.x * kThreads + threadIdx.x;
  if (r >= p.rows_pad) return;
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
  dst[0] = (M == -INFINITY) ? 0.f : M;
  dst[1] = (Z > 0.0) ? static_cast<float>(1.0 / Z) : 0.f;
}

template <typename T, int D, int RTW>
__global__ __launch_bounds__(kThreads) void score_mass_kernel(ScoreParams p) {
  using MF = Mfma<T>;
  using RB = RowBlock<T, D, RTW>;
  __shared__ float part[kWaves][kScoreChunk];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15, grp = lane >> 4;
  const int chunk = blockIdx.x;
  const UnitInfo u = unit_info(p, blockIdx.y);
  const int k0 = chunk * kScoreChunk;
  if (k0 >= u.L) return;
  const int k1 = min(u.L, k0 + kScoreChunk);
  const T *kbase = reinterpret_cast<const T *>(p.k) + u.cunit * p.cap * D;
  const int row_tiles = p.rows_pad / 16;

  for (int i = threadIdx.x; i < kWaves * kScoreChunk; i += kThreads) (&part[0][0])[i] = 0.f;
  __syncthreads();

  for (int tg = 0; tg < row_tiles; tg += kWaves * RTW) {
    const int tile0 = tg + wave * RTW;
    RB rb;
    rb.load(p, u, tile0, col, grp);
    float rmax[RTW], rinv[RTW];
#pragma unroll
    for (int k = 0; k < RTW; ++k) {
      const int r = (tile0 + k) * 16 + col;
      const bool in = (tile0 + k) < row_tiles;
      const float *st = p.row_stat + (u.ounit * p.rows_pad + (in ? r : 0)) * 2;
      rmax[k] = in ? st[0] : 0.f;
      rinv[k] = in ? st[1] : 0.f;
      rb.valid[k] = rb.valid[k] && in;
    }
    for (int kb = k0; kb < k1; kb += kKeyTile) {
      typename MF::frag kf[RB::steps];
      load_key_tile<T, D>(kbase, kb, u.L, col, grp, kf);
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < RTW; ++k) {
        if (tile0 + k >= row_tiles) break;
        f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < RB::steps; ++c) s = MF::mma(kf[c], rb.q[k][c], s);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kb + 4 * grp + i;
          const bool vis = rb.valid[k] && key < u.L && (!p.causal || key <= rb.pos[k]);
          const float e = fast_exp2(s[i] * p.scale_log2 - rmax[k]) * rinv[k];
          acc[i] += vis ? e : 0.f;
        }
      }
      // Sum over the 16 rows of each tile (lanes of one group), then bank the key sums.
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float tot = row16_sum(acc[i]);
        if (col == 0) part[wave][kb - k0 + 4 * grp + i] += tot;
      }
    }
  }
  __syncthreads();
  float *out = p.scores + u.ounit * p.cap;
  for (int j = threadIdx.x; j < k1 - k0; j += kThreads) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[w][j];
    out[k0 + j] = s;
  }
}

template <typename T, int D, int RTW>
hipError_t launch_rtw(const ScoreParams &p, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  hipLaunchKernelGGL((score_stats_kernel<T, D, RTW>), dim3(p.chunks, units), dim3(kThreads), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_rowmerge_kernel, dim3((p.rows_pad + kThreads - 1) / kThreads, units), dim3(kThreads), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_mass_kernel<T, D, RTW>), dim3(p.chunks, units), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_typed(const ScoreParams &p, hipStream_t s) {
  const int row_tiles = p.rows_pad / 16;
  if (row_tiles <= kWaves * 2) return launch_rtw<T, D, 2>(p, s);
  if (row_tiles <= kWaves * 4) return launch_rtw<T, D, 4>(p, s);
  return launch_rtw<T, D, 8>(p, s);
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
