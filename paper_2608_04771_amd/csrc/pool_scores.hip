// Score pooling before the top-k (gfx950): a policy variant on the scoring
// and selection kernels, the clustering idea of the eviction methods cited in
// Section 1.  Per unit with L = len and prefix P = L - min(w, L), prefix
// position j takes the max (mode 0) or the mean (mode 1) of the scores at the
// prefix positions within kernel / 2 of j; window positions keep their own
// score.  One 256-thread workgroup per (unit, 2048-position chunk) stages the
// chunk and its halo in LDS; means are summed in fp64 in index order and
// rounded once.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

namespace reco {

namespace {

constexpr int kPoolThreads = 256;
constexpr int kPoolChunk = 2048;
constexpr int kPoolMaxHalf = kPoolMaxKernel / 2;

__global__ __launch_bounds__(kPoolThreads) void pool_scores_kernel(PoolParams p) {
  __shared__ float s_tile[kPoolChunk + 2 * kPoolMaxHalf];
  const int chunk = blockIdx.x;
  const int unit = blockIdx.y;
  const int per_layer = p.batch * p.hkv;
  const int lc = unit / per_layer;
  const int b = (unit % per_layer) / p.hkv;
  const int h = unit % p.hkv;
  const size_t cunit = (static_cast<size_t>(p.layer0 + lc) * p.batch + b) * p.hkv + h;
  const int L = p.len[cunit];
  if (L < 0 || L > p.cap) {
    if (chunk == 0 && threadIdx.x == 0) report(p.dev_err, 5 /*RECO_DEV_BAD_LENGTH*/);
    return;
  }
  const int c0 = chunk * kPoolChunk;
  if (c0 >= L) return;                                   // uniform over the workgroup
  const int P = L - min(p.w, L);
  const int half = p.kernel / 2;
  const float *src = p.scores + static_cast<size_t>(unit) * p.cap;
  float *dst = p.pooled + static_cast<size_t>(unit) * p.cap;
  // Stage prefix scores [c0 - half, c0 + kPoolChunk + half) clipped to [0, P).
  const int t0 = c0 - half;
  const int tn = kPoolChunk + 2 * half;
  for (int i = threadIdx.x; i < tn; i += kPoolThreads) {
    const int j = t0 + i;
    s_tile[i] = (j >= 0 && j < P) ? src[j] : 0.f;
  }
  __syncthreads();
  const int c1 = min(L, c0 + kPoolChunk);
  for (int j = c0 + threadIdx.x; j < c1; j += kPoolThreads) {
    float out;
    if (j >= P) {
      out = src[j];                                      // window: own score
    } else {
      const int lo = max(0, j - half), hi = min(P - 1, j + half);
      if (p.mode == 0) {
        float m = s_tile[lo - t0];
        for (int i = lo + 1; i <= hi; ++i) m = fmaxf(m, s_tile[i - t0]);
        out = m;
      } else {
        double acc = 0.0;
        for (int i = lo; i <= hi; ++i) acc += static_cast<double>(s_tile[i - t0]);
        out = static_cast<float>(acc / static_cast<double>(hi - lo + 1));
      }
    }
    dst[j] = out;
  }
}

}  // namespace

hipError_t launch_pool_scores(const PoolParams &p, hipStream_t s) {
  const int units = p.n_layers * p.batch * p.hkv;
  const int chunks = (p.cap + kPoolChunk - 1) / kPoolChunk;
  hipLaunchKernelGGL(pool_scores_kernel, dim3(chunks, units), dim3(kPoolThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace reco
