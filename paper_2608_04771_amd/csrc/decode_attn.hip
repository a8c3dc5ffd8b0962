// GQA split-K decode attention over ragged per-head KV caches (gfx950).
//
// One "unit" is a (layer, sequence, kv head) with n valid cache rows and G
// query heads.  The grid is (splits, units): workgroup (s, u) walks a
// contiguous range of 32-key tiles of unit u with its four waves interleaved
// over the tiles, so the workgroup streams one contiguous stretch of K and V.
//
// Per 32-key tile a wave computes, on the matrix cores,
//   S^T = K_tile . Q^T            (M = 16 keys per half, N = 16 padded queries)
//   O^T += V_tile^T . P^T         (M = 16 head-dim rows per d-tile, N = 16 queries)
// The S^T accumulator already holds, per lane, the probabilities the P^T
// operand needs (same lane, same element slot), so P never leaves registers;
// V is staged through LDS to read it column-wise.  Softmax is online in the
// log2 domain with fp32 statistics.  The four waves' (max, sum, O) states are
// merged through LDS and written as one split partial; a second kernel merges
// the splits, writes out / lse and commits the optional append.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

#include <math.h>

namespace reco {

namespace {

constexpr int kTile = 32;        // keys per wave iteration
constexpr int kWavesPerWG = 4;
constexpr int kThreads = kWavesPerWG * kWave;

template <typename T, int D>
struct DecodeCfg {
  using MF = Mfma<T>;
  static constexpr int kpl = MF::kPerLane;
  static constexpr int dq = D / 4;                  // head-dim elements per lane group for Q.K
  static constexpr int qk_steps = dq / kpl;         // MFMAs per 16-key half
  static constexpr int dtiles = D / 16;             // output head-dim tiles
  static constexpr int pv_ops = kTile / MF::kPerOp;  // MFMAs per d-tile per 32-key tile
  static constexpr int row_bytes = D * (int)sizeof(T);
  static constexpr int lds_stride = row_bytes + 8;  // padded row pitch of the V stage
  static constexpr int stage_bytes = kWavesPerWG * kTile * lds_stride;
  static constexpr int merge_bytes = kWavesPerWG * (32 + 16 * D) * 4;
  static constexpr int smem_bytes = stage_bytes > merge_bytes ? stage_bytes : merge_bytes;
  static constexpr int vload_u4 = row_bytes / 2 / 16;  // uint4 per lane for half a V row
};

template <typename T>
__device__ __forceinline__ T lds_elem(const unsigned char *p) {
  return *reinterpret_cast<const T *>(p);
}

// Gather the V^T fragment of MFMA `c` for head-dim column `dcol` from the
// staged tile: element j holds key (e / 4) * 16 + 4 * grp + (e % 4), e = c * kpl + j.
template <typename T, int D>
__device__ __forceinline__ typename Mfma<T>::frag vt_frag(const unsigned char *stage, int c, int grp,
                                                          int dcol) {
  using Cfg = DecodeCfg<T, D>;
  typename Mfma<T>::frag a;
  if constexpr (Cfg::kpl == 1) {
    const int e = c;
    const int kl = (e >> 2) * 16 + 4 * grp + (e & 3);
    a = lds_elem<float>(stage + kl * Cfg::lds_stride + dcol * 4);
  } else {
#pragma unroll
    for (int j = 0; j < Cfg::kpl; ++j) {
      const int e = c * Cfg::kpl + j;
      const int kl = (e >> 2) * 16 + 4 * grp + (e & 3);
      const uint16_t bits = *reinterpret_cast<const uint16_t *>(stage + kl * Cfg::lds_stride + dcol * 2);
      a[j] = __builtin_bit_cast(__bf16, bits);
    }
  }
  return a;
}

// P^T fragment of MFMA `c`: the probabilities pv[e] for e = c * kpl + j.
template <typename T>
__device__ __forceinline__ typename Mfma<T>::frag pt_frag(const float (&pv)[8], int c) {
  if constexpr (Mfma<T>::kPerLane == 1) {
    return pv[c];
  } else {
    return pack_frag8(pv);
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeParams p) {
  using Cfg = DecodeCfg<T, D>;
  using MF = Mfma<T>;
  using frag = typename MF::frag;
  __shared__ __attribute__((aligned(16))) unsigned char smem[Cfg::smem_bytes];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const int split = blockIdx.x;
  const int unit = blockIdx.y;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const size_t qunit = static_cast<size_t>(lc) * per_layer + static_cast<size_t>(b) * p.hkv + h;

  int n_cache = p.len[cunit];
  n_cache = n_cache < 0 ? 0 : (n_cache > p.cap ? p.cap : n_cache);
  const bool append = p.k_new != nullptr;
  const int n_tot = n_cache + (append ? 1 : 0);
  const T *kbase = reinterpret_cast<const T *>(p.k) + cunit * p.cap * D;
  const T *vbase = reinterpret_cast<const T *>(p.v) + cunit * p.cap * D;
  const T *knew = append ? reinterpret_cast<const T *>(p.k_new) + qunit * D : nullptr;
  const T *vnew = append ? reinterpret_cast<const T *>(p.v_new) + qunit * D : nullptr;

  const int ntiles = (n_tot + kTile - 1) / kTile;
  const int tps = (ntiles + p.splits - 1) / p.splits;
  const int t0 = split * tps;
  const int t1 = min(ntiles, t0 + tps);

  // Q^T operand: lane (query col, group grp) holds head-dim elements grp*dq + c*kpl + j.
  frag qf[Cfg::qk_steps];
  {
    const T *qrow = reinterpret_cast<const T *>(p.q) +
                    ((static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group + col) * D + grp * Cfg::dq;
#pragma unroll
    for (int c = 0; c < Cfg::qk_steps; ++c)
      qf[c] = (col < p.group) ? load_frag(qrow + c * Cfg::kpl) : zero_frag(frag{});
  }

  float m_run = -INFINITY;
  float l_run = 0.f;
  f32x4_t o[Cfg::dtiles];
#pragma unroll
  for (int dt = 0; dt < Cfg::dtiles; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  unsigned char *stage = smem + wave * kTile * Cfg::lds_stride;

  for (int t = t0 + wave; t < t1; t += kWavesPerWG) {
    const int kb = t * kTile;
    // K operand: lane holds key kb + hf*16 + col, head-dim slice of its group.
    frag kf[2][Cfg::qk_steps];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int key = kb + hf * 16 + col;
      const T *row = key < n_cache ? kbase + static_cast<size_t>(key) * D
                                   : ((key == n_cache && append) ? knew : kbase);
      row += grp * Cfg::dq;
#pragma unroll
      for (int c = 0; c < Cfg::qk_steps; ++c) kf[hf][c] = load_frag(row + c * Cfg::kpl);
    }
    // V rows for the stage: lane -> row lane/2, half lane%2 (rows past the end are zero).
    uint4 vreg[Cfg::vload_u4];
    {
      const int r = lane >> 1;
      const int key = kb + r;
      const T *row = key < n_cache ? vbase + static_cast<size_t>(key) * D
                                   : ((key == n_cache && append) ? vnew : nullptr);
      if (row) {
        const uint4 *src = reinterpret_cast<const uint4 *>(reinterpret_cast<const unsigned char *>(row) +
                                                           (lane & 1) * (Cfg::row_bytes / 2));
#pragma unroll
        for (int i = 0; i < Cfg::vload_u4; ++i) vreg[i] = src[i];
      } else {
#pragma unroll
        for (int i = 0; i < Cfg::vload_u4; ++i) vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }

    // S^T = K . Q^T for the two 16-key halves.
    f32x4_t s[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      s[hf] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < Cfg::qk_steps; ++c) s[hf] = MF::mma(kf[hf][c], qf[c], s[hf]);
    }

    // Online softmax over this tile (log2 domain).  Lane holds keys
    // kb + hf*16 + 4*grp + i of query col.
    float sv[8];
    float tmax = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = kb + (e >> 2) * 16 + 4 * grp + (e & 3);
      float x = s[e >> 2][e & 3] * p.scale_log2;
      x = key < n_tot ? x : -INFINITY;
      sv[e] = x;
      tmax = fmaxf(tmax, x);
    }
    tmax = group4_max(tmax);
    const float m_new = fmaxf(m_run, tmax);          // finite: the tile holds a valid key
    const float alpha = fast_exp2(m_run - m_new);    // 0 on the first tile
    float pv[8];
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv[e] = fast_exp2(sv[e] - m_new);
      psum += pv[e];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < Cfg::dtiles; ++dt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[dt][i] *= alpha;
    }

    // Stage V (row-major, padded pitch) and read it back column-wise.
    {
      uint2 *dst = reinterpret_cast<uint2 *>(stage + (lane >> 1) * Cfg::lds_stride + (lane & 1) * (Cfg::row_bytes / 2));
#pragma unroll
      for (int i = 0; i < Cfg::vload_u4; ++i) {
        dst[2 * i] = make_uint2(vreg[i].x, vreg[i].y);
        dst[2 * i + 1] = make_uint2(vreg[i].z, vreg[i].w);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int dt = 0; dt < Cfg::dtiles; ++dt) {
#pragma unroll
      for (int c = 0; c < Cfg::pv_ops; ++c) {
        const frag a = vt_frag<T, D>(stage, c, grp, dt * 16 + col);
        o[dt] = MF::mma(a, pt_frag<T>(pv, c), o[dt]);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }

  // Total of the per-lane partial sums of query col.
  const float l_tot = group4_sum(l_run);

  // Cross-wave merge through LDS.
  __syncthreads();
  float *mw = reinterpret_cast<float *>(smem);   // [4][16]
  float *lw = mw + kWavesPerWG * 16;             // [4][16]
  float *ow = lw + kWavesPerWG * 16;             // [4][16][D]
  if (grp == 0) {
    mw[wave * 16 + col] = m_run;
    lw[wave * 16 + col] = l_tot;
  }
#pragma unroll
  for (int dt = 0; dt < Cfg::dtiles; ++dt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) ow[(wave * 16 + col) * D + dt * 16 + 4 * grp + i] = o[dt][i];
  }
  __syncthreads();

  const size_t pbase = static_cast<size_t>(unit) * p.splits + split;
  float *po = p.part_o + pbase * 16 * D;
  float *pml = p.part_ml + pbase * 32;
  for (int idx = threadIdx.x; idx < p.group * D; idx += kThreads) {
    const int qi = idx / D;
    const int d = idx - qi * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWavesPerWG; ++w) M = fmaxf(M, mw[w * 16 + qi]);
    float acc = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWavesPerWG; ++w) acc += ow[(w * 16 + qi) * D + d] * fast_exp2(mw[w * 16 + qi] - M);
    }
    po[qi * D + d] = acc;
    if (d == 0) {
      float L = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < kWavesPerWG; ++w) L += lw[w * 16 + qi] * fast_exp2(mw[w * 16 + qi] - M);
      }
      pml[qi] = M;
      pml[16 + qi] = L;
    }
  }
}

// Merge the split partials of one unit, write out / lse and commit the append.
template <typename T, int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeParams p) {
  const int unit = blockIdx.x;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const size_t qunit = static_cast<size_t>(lc) * per_layer + static_cast<size_t>(b) * p.hkv + h;
  const int len_in = p.len[cunit];
  const bool append = p.k_new != nullptr;

  const float *pml = p.part_ml + static_cast<size_t>(unit) * p.splits * 32;
  const float *po = p.part_o + static_cast<size_t>(unit) * p.splits * 16 * D;
  T *out = reinterpret_cast<T *>(p.out) + ((static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group) * D;
  for (int idx = threadIdx.x; idx < p.group * D; idx += blockDim.x) {
    const int qi = idx / D;
    const int d = idx - qi * D;
    float M = -INFINITY;
    for (int s = 0; s < p.splits; ++s) M = fmaxf(M, pml[s * 32 + qi]);
    float L = 0.f, acc = 0.f;
    if (M != -INFINITY) {
      for (int s = 0; s < p.splits; ++s) {
        const float wgt = fast_exp2(pml[s * 32 + qi] - M);
        L += pml[s * 32 + 16 + qi] * wgt;
        acc += po[(static_cast<size_t>(s) * 16 + qi) * D + d] * wgt;
      }
    }
    out[static_cast<size_t>(qi) * D + d] = from_f32<T>(L > 0.f ? acc / L : 0.f);
    if (d == 0 && p.lse) {
      p.lse[(static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group + qi] =
          L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    }
  }

  if (threadIdx.x == 0 && (len_in < 0 || len_in > p.cap)) report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
  if (!append || len_in < 0 || len_in > p.cap) return;
  if (len_in == p.cap) {
    if (threadIdx.x == 0) report(p.dev_err, 1 /*RECO_DEV_APPEND_OVERFLOW*/);
    return;
  }
  T *kdst = reinterpret_cast<T *>(p.k) + (cunit * p.cap + len_in) * D;
  T *vdst = reinterpret_cast<T *>(p.v) + (cunit * p.cap + len_in) * D;
  const T *ksrc = reinterpret_cast<const T *>(p.k_new) + qunit * D;
  const T *vsrc = reinterpret_cast<const T *>(p.v_new) + qunit * D;
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    kdst[d] = ksrc[d];
    vdst[d] = vsrc[d];
  }
  __syncthreads();
  if (threadIdx.x == 0) p.len[cunit] = len_in + 1;
}

template <typename T, int D>
hipError_t launch_typed(const DecodeParams &p, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  hipLaunchKernelGGL((decode_split_kernel<T, D>), dim3(p.splits, units), dim3(kThreads), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_merge_kernel<T, D>), dim3(units), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

// Splits per unit: aim for a few thousand workgroups over the chip while
// keeping at least four 32-key tiles per workgroup at full capacity.
int decode_splits(int units, int capacity) {
  const int target_wgs = 2048;
  const int tiles_cap = (capacity + 1 + kTile - 1) / kTile;
  int splits = (target_wgs + units - 1) / units;
  int max_splits = tiles_cap / 4;
  if (max_splits < 1) max_splits = 1;
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  return splits;
}

size_t decode_workspace_bytes(int units, int capacity, int head_dim) {
  const size_t splits = static_cast<size_t>(decode_splits(units, capacity));
  return static_cast<size_t>(units) * splits * (16 * static_cast<size_t>(head_dim) + 32) * sizeof(float);
}

hipError_t launch_decode(const DecodeParams &p, int dtype, int head_dim, hipStream_t s) {
  if (dtype == 0) {
    if (head_dim == 64) return launch_typed<float, 64>(p, s);
    return launch_typed<float, 128>(p, s);
  }
  if (head_dim == 64) return launch_typed<bf16_t, 64>(p, s);
  return launch_typed<bf16_t, 128>(p, s);
}

}  // namespace reco
