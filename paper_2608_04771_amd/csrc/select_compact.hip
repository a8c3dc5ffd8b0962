// Reward-budgeted selection and in-place compaction of the KV cache (gfx950).
//
// select: one 1024-thread workgroup per unit.  The budget m follows from the
//   unit's length and the sequence's retention in fp64; the k = m - w_eff
//   best prefix scores are found with an exact MSB-first radix select on the
//   fp32 bit patterns (non-negative floats order like their bits): three
//   histogram passes of 11, 11 and 10 bits over LDS bins give the k-th value
//   theta and how many of the entries equal to theta are still needed.  A
//   block-wide ordered scan then writes the kept positions in ascending order
//   (entries above theta, plus the first `need` entries equal to theta), and
//   the window positions after them.
// compact: one 256-thread workgroup per (unit, K or V, 128-byte column slice)
//   moves row idx[p] to row p for p = 0..m-1 in ascending chunks of 256
//   rows.  Because idx is strictly increasing, idx[p] >= p: a chunk's sources
//   lie at or after its own destinations, and rows a later chunk reads lie at
//   or after that chunk's destinations, beyond everything stored so far.  So
//   loading a whole chunk, waiting at a barrier, then storing it never
//   overwrites a row that is still to be read; no second buffer is needed.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

#include <math.h>

namespace reco {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kItems = 4;                    // consecutive positions per thread in the ordered scan
constexpr int kCompThreads = 256;
constexpr int kSliceBytes = 128;             // row slice per compaction workgroup
constexpr int kLanesPerRow = kSliceBytes / 16;
constexpr int kRowsPerPass = kCompThreads / kLanesPerRow;  // 32
constexpr int kRowsPerThread = 8;
constexpr int kChunkRows = kRowsPerPass * kRowsPerThread;  // 256

// Inclusive wave scan of an int.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int o = __shfl_up(v, d, kWave);
    if (lane >= d) v += o;
  }
  return v;
}

// Exclusive block scan over 1024 threads; returns the exclusive prefix and
// writes the block total to *total.  Uses `wsum` (kSelWaves ints) of LDS.
__device__ __forceinline__ int block_excl_scan(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int incl = wave_incl_scan(v, lane);
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int x = lane < kSelWaves ? wsum[lane] : 0;
    x = wave_incl_scan(x, lane);
    if (lane < kSelWaves) wsum[lane] = x;       // inclusive wave totals
  }
  __syncthreads();
  const int before = wave == 0 ? 0 : wsum[wave - 1];
  *total = wsum[kSelWaves - 1];
  __syncthreads();
  return before + incl - v;
}

__device__ __forceinline__ uint32_t score_bits(float s, bool *bad) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0;                    // -0 ranks as +0
  if ((u >> 31) || u > 0x7f800000u) *bad = true;  // negative or NaN
  return u;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p) {
  __shared__ int hist[2048];
  __shared__ int wsum[kSelWaves];
  __shared__ int s_bin, s_krem, s_bad;

  const int unit = blockIdx.x;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const int tid = threadIdx.x;

  const int L = p.len[cunit];
  const double r = p.retention[static_cast<int64_t>(lc) * p.ret_stride + b];
  if (L < 0 || L > p.cap) {
    if (tid == 0) {
      report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
      p.kept[unit] = -1;
    }
    return;
  }
  if (!(r > 0.0 && r <= 1.0)) {
    if (tid == 0) {
      report(p.dev_err, 2 /*RECO_DEV_BAD_RETENTION*/);
      p.kept[unit] = -1;
    }
    return;
  }
  const int w_eff = min(p.w, L);
  const double prod = r * static_cast<double>(L);
  int m = static_cast<int>(ceil(prod));
  m = max(w_eff, m);
  m = min(L, m);
  const int k = m - w_eff;
  const int P = L - w_eff;
  const float *sc = p.scores + static_cast<size_t>(unit) * p.cap;
  int32_t *idx = p.idx + static_cast<size_t>(unit) * p.cap;

  if (tid == 0) s_bad = 0;
  __syncthreads();

  // Validate the prefix scores (one pass, fused with the first histogram when k < P).
  uint32_t prefix = 0, pmask = 0;
  int krem = k;
  if (k > 0 && k < P) {
    const int shifts[3] = {21, 10, 0};
    const int nbits[3] = {11, 11, 10};
    for (int pass = 0; pass < 3; ++pass) {
      const int sh = shifts[pass];
      const int nb = 1 << nbits[pass];
      for (int i = tid; i < nb; i += kSelThreads) hist[i] = 0;
      __syncthreads();
      bool bad = false;
      for (int j = tid; j < P; j += kSelThreads) {
        const uint32_t u = score_bits(sc[j], &bad);
        if ((u & pmask) == prefix) atomicAdd(&hist[(u >> sh) & (nb - 1)], 1);
      }
      if (bad) s_bad = 1;
      __syncthreads();
      if (s_bad) break;
      // Find the bin holding the krem-th largest entry (wave 0).
      if (tid < kWave) {
        const int per = nb / kWave;
        const int lo = tid * per;
        int sum = 0;
        for (int i = 0; i < per; ++i) sum += hist[lo + i];
        // suffix sum over higher lanes: exclusive scan of the lane-reversed sums
        const int rev_lane = kWave - 1 - tid;
        const int rsum = __shfl(sum, kWave - 1 - tid, kWave);  // lane t holds lane (63-t)'s sum
        const int rincl = wave_incl_scan(rsum, tid);
        const int above_me = __shfl(rincl - rsum, rev_lane, kWave);  // sum of lanes > tid
        if (above_me < krem && krem <= above_me + sum) {
          int acc = above_me;
          for (int i = per - 1; i >= 0; --i) {
            const int c = hist[lo + i];
            if (acc + c >= krem) {
              s_bin = lo + i;
              s_krem = krem - acc;
              break;
            }
            acc += c;
          }
        }
      }
      __syncthreads();
      prefix |= static_cast<uint32_t>(s_bin) << sh;
      pmask |= static_cast<uint32_t>(nb - 1) << sh;
      krem = s_krem;
      __syncthreads();
    }
  } else {
    bool bad = false;
    for (int j = tid; j < P; j += kSelThreads) (void)score_bits(sc[j], &bad);
    if (bad) s_bad = 1;
    __syncthreads();
  }
  if (s_bad) {
    if (tid == 0) {
      report(p.dev_err, 3 /*RECO_DEV_BAD_SCORE*/);
      p.kept[unit] = -1;
    }
    return;
  }

  // Ordered scan: keep u > theta, and the first `need` entries with u == theta.
  const uint32_t theta = prefix;
  const int need = krem;
  int carry_eq = 0, carry_keep = 0;
  if (k == 0) {
    // only the window survives
  } else if (k == P) {
    for (int j = tid; j < P; j += kSelThreads) idx[j] = j;
    carry_keep = P;
  } else {
    for (int base = 0; base < P; base += kSelThreads * kItems) {
      uint32_t u[kItems];
      int n_eq = 0;
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        const int j = base + tid * kItems + i;
        bool dummy = false;
        u[i] = j < P ? score_bits(sc[j], &dummy) : 0u;
        if (j < P && u[i] == theta) ++n_eq;
      }
      int eq_total;
      const int eq_before = carry_eq + block_excl_scan(n_eq, wsum, &eq_total);
      bool keep[kItems];
      int n_keep = 0, eq_run = eq_before;
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        const int j = base + tid * kItems + i;
        const bool in = j < P;
        const bool is_eq = in && u[i] == theta;
        keep[i] = in && (u[i] > theta || (is_eq && eq_run < need));
        eq_run += is_eq ? 1 : 0;
        n_keep += keep[i] ? 1 : 0;
      }
      int keep_total;
      int pos = carry_keep + block_excl_scan(n_keep, wsum, &keep_total);
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        if (keep[i]) idx[pos++] = base + tid * kItems + i;
      }
      carry_eq += eq_total;
      carry_keep += keep_total;
    }
  }
  for (int t = tid; t < w_eff; t += kSelThreads) idx[k + t] = P + t;
  if (tid == 0) p.kept[unit] = m;
}

template <int ROWB>
__global__ __launch_bounds__(kCompThreads) void compact_kernel(SelectParams p) {
  constexpr int kSlices = ROWB / kSliceBytes;
  constexpr int kPerUnit = 2 * kSlices;             // (K or V) x slice workgroups of one unit
  // XCD-aware order: consecutive workgroup ids go to the eight XCDs in turn,
  // so ids are laid out in groups of 8 units x kPerUnit with every workgroup
  // of a unit at the same id mod 8: they share one XCD's L2 and the unit's
  // kept list is fetched from HBM once.  Padding workgroups return at once.
  const int grp8 = static_cast<int>(blockIdx.x) / (8 * kPerUnit);
  const int r8 = static_cast<int>(blockIdx.x) - grp8 * 8 * kPerUnit;
  const int unit = grp8 * 8 + (r8 & 7);
  const int job = r8 >> 3;
  const int slice = job % kSlices;
  const int tensor = job / kSlices;
  if (unit >= p.n_layers * p.batch * p.hkv) return;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const int m = p.kept[unit];
  if (m < 0) return;
  const int32_t *idx = p.idx + static_cast<size_t>(unit) * p.cap;
  unsigned char *base = reinterpret_cast<unsigned char *>(tensor == 0 ? p.k : p.v) +
                        cunit * static_cast<size_t>(p.cap) * ROWB + slice * kSliceBytes;
  const int sub = (threadIdx.x % kLanesPerRow) * 16;
  const int rrow = threadIdx.x / kLanesPerRow;

  for (int c0 = 0; c0 < m; c0 += kChunkRows) {
    // One 128-bit register per row of the chunk; the whole chunk stays in
    // registers across the barrier.  Rows that do not move (or lie past m)
    // read row 0 of the unit, which is always in bounds.
    typedef unsigned int u32x32 __attribute__((ext_vector_type(4 * kRowsPerThread)));
    u32x32 v;
    unsigned mv = 0;
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const int pdst = c0 + i * kRowsPerPass + rrow;
      const int s = idx[min(pdst, m - 1)];
      const bool move = pdst < m && s != pdst;
      mv |= (move ? 1u : 0u) << i;
      const uint4 x = *reinterpret_cast<const uint4 *>(base + static_cast<size_t>(move ? s : 0) * ROWB + sub);
      v[4 * i + 0] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
    __syncthreads();   // every read of this chunk has returned before any row of it is overwritten
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const int pdst = c0 + i * kRowsPerPass + rrow;
      if (mv & (1u << i))
        *reinterpret_cast<uint4 *>(base + static_cast<size_t>(pdst) * ROWB + sub) =
            make_uint4(v[4 * i + 0], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    }
  }
  if (tensor == 0 && slice == 0 && threadIdx.x == 0) p.len[cunit] = m;
}

}  // namespace

size_t select_workspace_bytes(int units, int capacity, bool need_idx) {
  size_t bytes = (static_cast<size_t>(units) * sizeof(int32_t) + 255) / 256 * 256;
  if (need_idx) bytes += static_cast<size_t>(units) * capacity * sizeof(int32_t);
  return bytes;
}

hipError_t launch_select_compact(const SelectParams &p, int dtype, int head_dim, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  hipLaunchKernelGGL(select_kernel, dim3(units), dim3(kSelThreads), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rowb = head_dim * (dtype == 0 ? 4 : 2);
  switch (rowb) {
    case 128:
      hipLaunchKernelGGL(compact_kernel<128>, dim3((units + 7) / 8 * 8 * 2 * 1), dim3(kCompThreads), 0, s, p);
      break;
    case 256:
      hipLaunchKernelGGL(compact_kernel<256>, dim3((units + 7) / 8 * 8 * 2 * 2), dim3(kCompThreads), 0, s, p);
      break;
    default:
      hipLaunchKernelGGL(compact_kernel<512>, dim3((units + 7) / 8 * 8 * 2 * 4), dim3(kCompThreads), 0, s, p);
      break;
  }
  return hipGetLastError();
}

}  // namespace reco
