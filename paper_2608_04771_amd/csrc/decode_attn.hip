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
// operand needs (same lane, same element slot), so P never leaves registers.
// K and V are streamed with coalesced non-temporal 16-byte loads (each 128-byte
// line read whole, nothing allocated in L2) and staged through LDS: K is
// re-read in the MFMA operand layout, V column-wise.  Softmax is online in the
// log2 domain with fp32 statistics.  The four waves' (max, sum, O) states are
// merged through LDS and written as one split partial.  A second kernel
// merges the splits of each unit, writes out / lse and commits the optional
// append (so no workgroup of the attention kernel races on len); a unit
// covered by a single workgroup (one split) is finalised by that workgroup,
// with no second launch.  Merging in
// the last-finishing workgroup instead would need device-scope fences, which
// on this chip write back and invalidate the L2 that the streaming
// workgroups depend on.
#include "reco_device.hpp"
#include "decode_attn.hpp"
#include "decode_plan.hpp"

#include <math.h>

#include <atomic>
#include <mutex>

namespace reco {

namespace {

constexpr int kTile = kDecodeTile;   // keys per wave iteration
constexpr int kWavesPerWG = 4;
constexpr int kThreads = kWavesPerWG * kWave;
constexpr int kMaxSplits = kDecodeMaxSplits;

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
  static constexpr int k_stride = row_bytes + 16;   // padded, 16-byte aligned pitch of the K stage
  static constexpr int wave_stage = kTile * (lds_stride + k_stride);
  static constexpr int stage_bytes = kWavesPerWG * wave_stage;
  static constexpr int merge_bytes = kWavesPerWG * (32 + 16 * D) * 4;
  static constexpr int smem_bytes = stage_bytes > merge_bytes ? stage_bytes : merge_bytes;
  // Coalesced tile loads: per instruction the wave reads 1 KB of consecutive
  // rows (lane l takes 16 bytes at l * 16), so every 128-byte line is read whole.
  static constexpr int lanes_per_row = row_bytes / 16;
  static constexpr int rows_per_inst = kWave / lanes_per_row;
  static constexpr int v_insts = kTile / rows_per_inst;
  // Two workgroups per CU (two waves per SIMD) where the double-buffered
  // tile fits in 256 registers; the fp32 head_dim-128 variant needs more.
  static constexpr int min_wgs = (sizeof(T) == 4 && D == 128) ? 1 : 2;
};

// Registers of one 32-key tile: K and V as coalesced 16-byte pieces bound
// for the LDS stages (K is re-read from LDS in the MFMA operand layout).
template <typename T, int D>
struct TileRegs {
  uint4 kreg[DecodeCfg<T, D>::v_insts];
  uint4 vreg[DecodeCfg<T, D>::v_insts];
};

// Issue the loads of the tile starting at key kb.  Keys >= n_cache come from
// the appended row (key == n_cache) or are zero; every address stays inside
// the unit (rows past the end read row 0 and are masked or zeroed).
template <typename T, int D>
__device__ __forceinline__ void load_tile(TileRegs<T, D> &tr, int kb, int n_cache, bool append, const T *kbase,
                                          const T *vbase, const T *knew, const T *vnew, int lane) {
  using Cfg = DecodeCfg<T, D>;
  const int sub = (lane % Cfg::lanes_per_row) * 16;
#pragma unroll
  for (int i = 0; i < Cfg::v_insts; ++i) {
    const int r = i * Cfg::rows_per_inst + lane / Cfg::lanes_per_row;
    const int key = kb + r;
    const bool in_cache = key < n_cache;
    const bool is_new = key == n_cache && append;
    const size_t off = in_cache ? static_cast<size_t>(key) * D : 0;
    const T *krow = is_new ? knew : kbase + off;
    const T *vrow = is_new ? vnew : vbase + off;
    const uint4 kx = nt_load_u4(reinterpret_cast<const unsigned char *>(krow) + sub);
    const uint4 vx = nt_load_u4(reinterpret_cast<const unsigned char *>(vrow) + sub);
    tr.kreg[i] = kx;                                       // rows past the end are masked
    tr.vreg[i] = (in_cache || is_new) ? vx : make_uint4(0, 0, 0, 0);
  }
}

template <typename T>
__device__ __forceinline__ T lds_elem(const unsigned char *p) {
  return *reinterpret_cast<const T *>(p);
}

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

// Gather the V^T fragment of MFMA `c` for head-dim tile `dt` from the staged
// tile: lane (col, grp) needs, at head-dim column dt*16 + col, the keys of
// element e = c * kpl + j, key (e / 4) * 16 + 4 * grp + (e % 4).
// bf16: two LDS transpose reads.  Within each 16-lane group, lane j supplies
// the 8 bytes at row key0 + j / 4, columns d0 + 4 * (j % 4) .. + 3, and lane i
// receives element i % 4 of the rows supplied by lanes 4r + i / 4, r = 0..3,
// i.e. column d0 + i of rows key0 .. key0 + 3: four consecutive keys of one
// head-dim column, as the operand wants.
template <typename T, int D>
__device__ __forceinline__ typename Mfma<T>::frag vt_frag(const unsigned char *stage, int c, int grp, int dt,
                                                          int col) {
  using Cfg = DecodeCfg<T, D>;
  typename Mfma<T>::frag a;
  if constexpr (Cfg::kpl == 1) {
    const int e = c;
    const int kl = (e >> 2) * 16 + 4 * grp + (e & 3);
    a = lds_elem<float>(stage + kl * Cfg::lds_stride + (dt * 16 + col) * 4);
  } else {
    static_assert(Cfg::lds_stride % 8 == 0, "transpose reads need 8-byte aligned rows");
    const int key0 = 32 * c + 4 * grp + col / 4;
    const int cb = (dt * 16 + 4 * (col % 4)) * 2;
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t *)(stage + key0 * Cfg::lds_stride + cb));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t *)(stage + (key0 + 16) * Cfg::lds_stride + cb));
    const short v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = __builtin_bit_cast(__bf16, v[j]);
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
__global__ __launch_bounds__(kThreads, (DecodeCfg<T, D>::min_wgs)) void decode_split_kernel(DecodeParams p) {
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

  const int len_in = p.len[cunit];
  const int n_cache = len_in < 0 ? 0 : (len_in > p.cap ? p.cap : len_in);
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

  unsigned char *stage = smem + wave * Cfg::wave_stage;           // V, row pitch lds_stride
  unsigned char *kstage = stage + kTile * Cfg::lds_stride;          // K, row pitch k_stride

  TileRegs<T, D> cur;
  if (t0 + wave < t1) load_tile<T, D>(cur, (t0 + wave) * kTile, n_cache, append, kbase, vbase, knew, vnew, lane);
  for (int t = t0 + wave; t < t1; t += kWavesPerWG) {
    const int kb = t * kTile;
    // Prefetch this wave's next tile (the last iteration re-reads its own
    // tile, which stays cached) so loads are in flight during the compute.
    TileRegs<T, D> nxt;
    const int tn = min(t + kWavesPerWG, t1 - 1);
    load_tile<T, D>(nxt, tn * kTile, n_cache, append, kbase, vbase, knew, vnew, lane);
    // K tile -> LDS -> MFMA operand layout (lane holds key hf*16 + col,
    // head-dim slice grp*dq + c*kpl of it).
#pragma unroll
    for (int i = 0; i < Cfg::v_insts; ++i) {
      const int r = i * Cfg::rows_per_inst + lane / Cfg::lanes_per_row;
      *reinterpret_cast<uint4 *>(kstage + r * Cfg::k_stride + (lane % Cfg::lanes_per_row) * 16) = cur.kreg[i];
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    frag kf[2][Cfg::qk_steps];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const T *krow = reinterpret_cast<const T *>(kstage + (hf * 16 + col) * Cfg::k_stride) + grp * Cfg::dq;
#pragma unroll
      for (int c = 0; c < Cfg::qk_steps; ++c) kf[hf][c] = load_frag(krow + c * Cfg::kpl);
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
#pragma unroll
    for (int i = 0; i < Cfg::v_insts; ++i) {
      const int r = i * Cfg::rows_per_inst + lane / Cfg::lanes_per_row;
      uint2 *dst = reinterpret_cast<uint2 *>(stage + r * Cfg::lds_stride + (lane % Cfg::lanes_per_row) * 16);
      dst[0] = make_uint2(cur.vreg[i].x, cur.vreg[i].y);
      dst[1] = make_uint2(cur.vreg[i].z, cur.vreg[i].w);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int dt = 0; dt < Cfg::dtiles; ++dt) {
#pragma unroll
      for (int c = 0; c < Cfg::pv_ops; ++c) {
        const frag a = vt_frag<T, D>(stage, c, grp, dt, col);
        o[dt] = MF::mma(a, pt_frag<T>(pv, c), o[dt]);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    cur = nxt;
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

  if (p.splits == 1) {
    // The workgroup holds its unit's whole softmax: it writes out / lse /
    // row_stats and commits the append itself, with the arithmetic of the
    // merge of a single split (weight exp2(0) * 1/L, added to zero).
    const size_t oq0 = (static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group;
    for (int idx = threadIdx.x; idx < p.group * D; idx += kThreads) {
      const int qi = idx / D;
      const int d = idx - qi * D;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kWavesPerWG; ++w) M = fmaxf(M, mw[w * 16 + qi]);
      float acc = 0.f, L = 0.f;
      if (M != -INFINITY) {
#pragma unroll
        for (int w = 0; w < kWavesPerWG; ++w) {
          const float e = fast_exp2(mw[w * 16 + qi] - M);
          acc += ow[(w * 16 + qi) * D + d] * e;
          L += lw[w * 16 + qi] * e;
        }
      }
      const float inv = L > 0.f ? 1.f / L : 0.f;
      reinterpret_cast<T *>(p.out)[(oq0 + qi) * D + d] = from_f32<T>(fmaf(acc, inv, 0.f));
      if (d == 0) {
        if (p.lse) p.lse[oq0 + qi] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
        if (p.row_stats) {
          p.row_stats[(oq0 + qi) * 2 + 0] = M;
          p.row_stats[(oq0 + qi) * 2 + 1] = L;
        }
      }
    }
    // Every wave has finished reading the cache (barrier above); row n_cache
    // is read by no one in this call (the new key comes from k_new).
    if (threadIdx.x == 0 && (len_in < 0 || len_in > p.cap)) report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
    if (!append || len_in < 0 || len_in > p.cap) return;
    if (len_in == p.cap) {
      if (threadIdx.x == 0) report(p.dev_err, 1 /*RECO_DEV_APPEND_OVERFLOW*/);
      return;
    }
    for (int d = threadIdx.x; d < D; d += kThreads) {
      reinterpret_cast<T *>(p.k)[(cunit * p.cap + len_in) * D + d] = knew[d];
      reinterpret_cast<T *>(p.v)[(cunit * p.cap + len_in) * D + d] = vnew[d];
    }
    if (threadIdx.x == 0) p.len[cunit] = len_in + 1;
    return;
  }

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

// Merge the split partials of every (unit, query head), write out / lse and
// commit the append.  One 64-lane wave per (unit, query head): every lane
// fetches all split statistics at once (one memory round trip), derives the
// merge weights itself, then loads its head-dim slice of every split partial
// (a second round trip).  The appended row is fetched up front.
template <typename T, int D>
__global__ __launch_bounds__(kWave) void decode_merge_kernel(DecodeParams p) {
  constexpr int kPer = D / kWave;                  // head-dim elements per lane
  const int unit = blockIdx.x;
  const int qi = blockIdx.y;
  const int lane = threadIdx.x;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const size_t qunit = static_cast<size_t>(lc) * per_layer + static_cast<size_t>(b) * p.hkv + h;
  const int S = p.splits;
  const bool append = p.k_new != nullptr && qi == 0;

  // Query head 0 of the unit also commits the append: fetch len and the row now.
  const int len_in = qi == 0 ? p.len[cunit] : 0;
  T krow[kPer], vrow[kPer];
  if (append) {
    const T *ksrc = reinterpret_cast<const T *>(p.k_new) + qunit * D;
    const T *vsrc = reinterpret_cast<const T *>(p.v_new) + qunit * D;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      krow[i] = ksrc[lane + i * kWave];
      vrow[i] = vsrc[lane + i * kWave];
    }
  }
  const float *pml = p.part_ml + static_cast<size_t>(unit) * S * 32;
  const float *po = p.part_o + (static_cast<size_t>(unit) * S * 16 + qi) * D;
  // The first kPre splits' output slices are requested together with the
  // statistics, so a call with at most kPre splits costs one memory round trip.
  constexpr int kPre = 4;
  float pre[kPre][kPer];
#pragma unroll
  for (int s = 0; s < kPre; ++s) {
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      pre[s][i] = s < S ? po[static_cast<size_t>(s) * 16 * D + lane + i * kWave] : 0.f;
  }
  // Lane s holds split s's statistics, lane s - 64 the rest (S <= kMaxSplits = 128).
  const float m0 = lane < S ? pml[lane * 32 + qi] : -INFINITY;
  const float l0 = lane < S ? pml[lane * 32 + 16 + qi] : 0.f;
  const float m1 = lane + kWave < S ? pml[(lane + kWave) * 32 + qi] : -INFINITY;
  const float l1 = lane + kWave < S ? pml[(lane + kWave) * 32 + 16 + qi] : 0.f;
  const float M = wave_max(fmaxf(m0, m1));
  float L = 0.f;
  if (M != -INFINITY) L = wave_sum(l0 * fast_exp2(m0 - M) + l1 * fast_exp2(m1 - M));
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const float w0 = (M != -INFINITY) ? fast_exp2(m0 - M) * inv : 0.f;
  const float w1 = (M != -INFINITY) ? fast_exp2(m1 - M) * inv : 0.f;

  float acc[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) acc[i] = 0.f;
#pragma unroll
  for (int s = 0; s < kPre; ++s) {
    const float wgt = __shfl(w0, s, kWave);       // 0 for s >= S
#pragma unroll
    for (int i = 0; i < kPer; ++i) acc[i] += wgt * pre[s][i];
  }
  for (int s = kPre; s < S; ++s) {
    const float wgt = __shfl(s < kWave ? w0 : w1, s & (kWave - 1), kWave);
#pragma unroll
    for (int i = 0; i < kPer; ++i) acc[i] += wgt * po[static_cast<size_t>(s) * 16 * D + lane + i * kWave];
  }
  T *out = reinterpret_cast<T *>(p.out) + ((static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group + qi) * D;
#pragma unroll
  for (int i = 0; i < kPer; ++i) out[lane + i * kWave] = from_f32<T>(acc[i]);
  const size_t oq = (static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group + qi;
  if (p.lse && lane == 0) p.lse[oq] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  if (p.row_stats && lane == 0) {
    p.row_stats[oq * 2 + 0] = M;
    p.row_stats[oq * 2 + 1] = L;
  }

  if (qi != 0) return;
  if (lane == 0 && (len_in < 0 || len_in > p.cap)) report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
  if (!append || len_in < 0 || len_in > p.cap) return;
  if (len_in == p.cap) {
    if (lane == 0) report(p.dev_err, 1 /*RECO_DEV_APPEND_OVERFLOW*/);
    return;
  }
  T *kdst = reinterpret_cast<T *>(p.k) + (cunit * p.cap + len_in) * D;
  T *vdst = reinterpret_cast<T *>(p.v) + (cunit * p.cap + len_in) * D;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    kdst[lane + i * kWave] = krow[i];
    vdst[lane + i * kWave] = vrow[i];
  }
  if (lane == 0) p.len[cunit] = len_in + 1;
}

// Merge for many splits (small calls, e.g. one layer per call): one
// 256-thread workgroup per (unit, query head).  Every split's output slice is
// requested at once (thread group sg loads splits sg, sg + kSG, ... as 16-byte
// pieces) together with the split statistics, so the merge costs one memory
// round trip whatever the split count; the weighted slices meet in LDS.
constexpr int kWideThreads = 256;
constexpr int kWideMinSplits = 9;                  // fewer splits use the one-wave merge

template <typename T, int D>
__global__ __launch_bounds__(kWideThreads) void decode_merge_wide_kernel(DecodeParams p) {
  constexpr int kVec = 4;
  constexpr int kTPS = D / kVec;                   // threads per split slice
  constexpr int kSG = kWideThreads / kTPS;         // split groups
  constexpr int kMaxPer = kMaxSplits / kSG;        // splits per thread at most
  constexpr int kWaves = kWideThreads / kWave;
  __shared__ float s_w[kMaxSplits];
  __shared__ float s_red[kWaves];
  __shared__ __attribute__((aligned(16))) float s_acc[kSG][D];

  const int unit = blockIdx.x;
  const int qi = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const size_t qunit = static_cast<size_t>(lc) * per_layer + static_cast<size_t>(b) * p.hkv + h;
  const int S = p.splits;
  const bool append = p.k_new != nullptr && qi == 0;

  // Everything this workgroup reads is requested up front.
  const int len_in = qi == 0 ? p.len[cunit] : 0;
  T krow = T{}, vrow = T{};
  if (append && tid < D) {
    krow = reinterpret_cast<const T *>(p.k_new)[qunit * D + tid];
    vrow = reinterpret_cast<const T *>(p.v_new)[qunit * D + tid];
  }
  const int sg = tid / kTPS;
  const int dv = (tid % kTPS) * kVec;
  const float *po = p.part_o + (static_cast<size_t>(unit) * S * 16 + qi) * D;
  float4 part[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int sp = sg + kSG * i;
    part[i] = sp < S ? *reinterpret_cast<const float4 *>(po + static_cast<size_t>(sp) * 16 * D + dv)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const float *pml = p.part_ml + static_cast<size_t>(unit) * S * 32;
  const float m_t = tid < S ? pml[tid * 32 + qi] : -INFINITY;
  const float l_t = tid < S ? pml[tid * 32 + 16 + qi] : 0.f;

  // M = max of the split maxima, L = sum of the rescaled split sums.
  float v = wave_max(m_t);
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  float M = s_red[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) M = fmaxf(M, s_red[w]);
  __syncthreads();
  const float e_t = (M != -INFINITY && tid < S) ? fast_exp2(m_t - M) : 0.f;
  v = wave_sum(l_t * e_t);
  if (lane == 0) s_red[wave] = v;
  __syncthreads();
  float L = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) L += s_red[w];
  const float inv = L > 0.f ? 1.f / L : 0.f;
  if (tid < kMaxSplits) s_w[tid] = e_t * inv;
  __syncthreads();

  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int sp = sg + kSG * i;
    const float wgt = sp < S ? s_w[sp] : 0.f;
    acc.x += wgt * part[i].x;
    acc.y += wgt * part[i].y;
    acc.z += wgt * part[i].z;
    acc.w += wgt * part[i].w;
  }
  *reinterpret_cast<float4 *>(&s_acc[sg][dv]) = acc;
  __syncthreads();

  const size_t oq = (static_cast<size_t>(lc) * p.batch + b) * p.hq + h * p.group + qi;
  if (tid < D) {
    float o = 0.f;
#pragma unroll
    for (int g = 0; g < kSG; ++g) o += s_acc[g][tid];
    reinterpret_cast<T *>(p.out)[oq * D + tid] = from_f32<T>(o);
  }
  if (tid == 0) {
    if (p.lse) p.lse[oq] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    if (p.row_stats) {
      p.row_stats[oq * 2 + 0] = M;
      p.row_stats[oq * 2 + 1] = L;
    }
  }

  if (qi != 0) return;
  if (tid == 0 && (len_in < 0 || len_in > p.cap)) report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
  if (!append || len_in < 0 || len_in > p.cap) return;
  if (len_in == p.cap) {
    if (tid == 0) report(p.dev_err, 1 /*RECO_DEV_APPEND_OVERFLOW*/);
    return;
  }
  if (tid < D) {
    reinterpret_cast<T *>(p.k)[(cunit * p.cap + len_in) * D + tid] = krow;
    reinterpret_cast<T *>(p.v)[(cunit * p.cap + len_in) * D + tid] = vrow;
  }
  if (tid == 0) p.len[cunit] = len_in + 1;
}

template <typename T, int D>
hipError_t launch_typed(const DecodeParams &p, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  hipLaunchKernelGGL((decode_split_kernel<T, D>), dim3(p.splits, units), dim3(kThreads), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;   // one split: finalised in place
  if (p.splits >= kWideMinSplits)
    hipLaunchKernelGGL((decode_merge_wide_kernel<T, D>), dim3(units, p.group), dim3(kWideThreads), 0, s, p);
  else
    hipLaunchKernelGGL((decode_merge_kernel<T, D>), dim3(units, p.group), dim3(kWave), 0, s, p);
  return hipGetLastError();
}

}  // namespace

// Split partials of the allocation-free entry point.  Every device holds its
// own copy of this array at its own address until the process ends.  In host
// code `scratch` names a host-side stand-in for the device symbol, not device
// memory: host code uses only the address hipGetSymbolAddress returns for the
// current device, never the name itself.  The decode kernels write every
// partial they later read, so the array never needs clearing; calls that
// overlap on one device share it and race.
static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];

hipError_t decode_scratch(void **ptr) {
  constexpr int kMaxDevices = 64;
  static std::atomic<void *> addr[kMaxDevices];
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void *p = addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(mu);
    p = addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // with `dev` current
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      addr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
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
