// Generation-side kernels of Section 3.3 (gfx950):
//   reflection-token penalty, Eq. 3 (reward band) and Eq. 4 (subtract beta);
//   the same penalty fused with drawing the next token from softmax(z~ / T);
//   answer perplexity, Eq. 5, and the stop rule, Eq. 6.
#include "reco_device.hpp"
#include "reco_kernels.hpp"

#include <math.h>

namespace reco {

namespace {

constexpr int kPenThreads = 256;
constexpr int kMaxIds = 4096;

__global__ __launch_bounds__(kPenThreads) void logit_penalty_kernel(float *logits, int vocab, int64_t ld,
                                                                    const int32_t *ids, int n_ids,
                                                                    const float *reward, float tau_lo,
                                                                    float tau_hi, float b_lo, float b_mid,
                                                                    float b_hi, int32_t *dev_err) {
  __shared__ int32_t s_ids[kMaxIds];
  const int row = blockIdx.x;
  for (int i = threadIdx.x; i < n_ids; i += kPenThreads) s_ids[i] = ids[i];
  __syncthreads();
  const float v = reward[row];
  // Eq. 3 exactly as written: v <= tau_lo, tau_lo < v < tau_hi, v >= tau_hi.
  const float beta = (v <= tau_lo) ? b_lo : ((v >= tau_hi) ? b_hi : b_mid);
  float *z = logits + static_cast<int64_t>(row) * ld;
  for (int i = threadIdx.x; i < n_ids; i += kPenThreads) {
    const int u = s_ids[i];
    if (u < 0 || u >= vocab) {
      report(dev_err, 4 /*RECO_DEV_BAD_TOKEN_ID*/);
      continue;
    }
    bool first = true;  // R is a set: only the first occurrence of an id subtracts
    for (int j = 0; j < i; ++j) first = first && (s_ids[j] != u);
    if (first) z[u] = z[u] - beta;
  }
}

// ---- fused penalty + sampling ------------------------------------------------
//
// One pass over each logit row: Eq. 3 picks beta from the row's reward, Eq. 4
// subtracts it from the reflection ids (written back in place, as the plain
// penalty does), and the next token is the argmax of z~ (T = 0) or, for
// T > 0, the Gumbel-max draw argmax(z~ / T + G), which is an exact sample of
// softmax(z~ / T).  G = -log(-log U) with U from Philox4x32-10.  Workgroups
// take 1024-element chunks of a row (one Philox block of four per thread) and
// leave (best value, index) partials; a one-wave-per-row kernel merges them.  Ties and equal partials go to the
// lowest index; NaN values never win.

constexpr int kSmpThreads = 256;
constexpr int kSmpChunk = kSmpThreads * 4;   // logits per workgroup: one Philox block of 4 per thread
constexpr int kSmpBitWords = kSmpChunk / 32;

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror and Shaw, SC 2011): each
// round multiplies counter words 0 and 2 by the two round constants, crosses
// the 64-bit products' halves with words 1 and 3 and the key, and the key
// advances by the Weyl increments between rounds.
__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t a = c[0], b = c[2];
    const uint32_t lo0 = 0xD2511F53u * a, hi0 = __umulhi(0xD2511F53u, a);
    const uint32_t lo1 = 0xCD9E8D57u * b, hi1 = __umulhi(0xCD9E8D57u, b);
    c[0] = hi1 ^ c[1] ^ k0;
    c[1] = lo1;
    c[2] = hi0 ^ c[3] ^ k1;
    c[3] = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// Midpoint of one of 2^23 equal cells of (0, 1): exact in fp32, never 0 or 1.
__device__ __forceinline__ float unit_open(uint32_t x) {
  return static_cast<float>(x >> 9) * 0x1.0p-23f + 0x1.0p-24f;
}

__device__ __forceinline__ void arg_better(float &v, int &i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

__device__ __forceinline__ void wave_argmax(float &v, int &i) {
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    const float v2 = __shfl_xor(v, m, kWave);
    const int i2 = __shfl_xor(i, m, kWave);
    arg_better(v, i, v2, i2);
  }
}

struct SamplePart {
  float v;
  int32_t i;
};

__global__ __launch_bounds__(kSmpThreads) void penalty_sample_partial_kernel(
    float *logits, int vocab, int64_t ld, const int32_t *ids, int n_ids, const float *reward, float tau_lo,
    float tau_hi, float b_lo, float b_mid, float b_hi, float temperature, uint32_t seed_lo, uint32_t seed_hi,
    uint32_t off_lo, uint32_t off_hi, int chunks, SamplePart *part, int32_t *dev_err) {
  __shared__ uint32_t s_bits[kSmpBitWords];
  __shared__ SamplePart s_red[kSmpThreads / kWave];
  const int chunk = blockIdx.x;
  const int row = blockIdx.y;
  const int c0 = chunk * kSmpChunk;
  const int r0 = threadIdx.x * 4;                    // chunk-relative, multiple of 4
  const int j0 = c0 + r0;
  float *z = logits + static_cast<int64_t>(row) * ld;
  // Issue every global load before the first barrier so their latencies overlap.
  float x[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = (j0 + e < vocab) ? z[j0 + e] : -INFINITY;
  const float v = reward[row];
  const int my_id = (static_cast<int>(threadIdx.x) < n_ids) ? ids[threadIdx.x] : -1;
  if (threadIdx.x < kSmpBitWords) s_bits[threadIdx.x] = 0u;
  __syncthreads();
  // Mark the reflection ids that fall in this chunk; a set, so duplicates merge.
  for (int i = threadIdx.x; i < n_ids; i += kSmpThreads) {
    const int u = (i == static_cast<int>(threadIdx.x)) ? my_id : ids[i];
    if (u < 0 || u >= vocab) {
      if (chunk == 0) report(dev_err, 4 /*RECO_DEV_BAD_TOKEN_ID*/);
      continue;
    }
    const int r = u - c0;
    if (r >= 0 && r < kSmpChunk) atomicOr(&s_bits[r >> 5], 1u << (r & 31));
  }
  __syncthreads();
  const float beta = (v <= tau_lo) ? b_lo : ((v >= tau_hi) ? b_hi : b_mid);   // Eq. 3 as written

  float best = -INFINITY;
  int best_i = 0x7fffffff;
  if (j0 < vocab) {
    const uint32_t bits = (s_bits[r0 >> 5] >> (r0 & 31)) & 0xFu;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if ((bits >> e) & 1u) {                        // Eq. 4, one fp32 subtraction
        x[e] = x[e] - beta;
        z[j0 + e] = x[e];
      }
    if (temperature == 0.f) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j0 + e < vocab) arg_better(best, best_i, x[e], j0 + e);
    } else {
      uint32_t c[4] = {static_cast<uint32_t>(j0 >> 2), static_cast<uint32_t>(row), off_lo, off_hi};
      philox4x32_10(c, seed_lo, seed_hi);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float g = -logf(-logf(unit_open(c[e])));
        const float y = x[e] / temperature + g;
        if (j0 + e < vocab) arg_better(best, best_i, y, j0 + e);
      }
    }
  }
  wave_argmax(best, best_i);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  if (lane == 0) s_red[wave] = SamplePart{best, best_i};
  __syncthreads();
  if (threadIdx.x == 0) {
    SamplePart r = s_red[0];
#pragma unroll
    for (int w = 1; w < kSmpThreads / kWave; ++w) arg_better(r.v, r.i, s_red[w].v, s_red[w].i);
    part[static_cast<size_t>(row) * chunks + chunk] = r;
  }
}

// One wave per row: merge the chunk partials into the row's token.
__global__ __launch_bounds__(kSmpThreads) void penalty_sample_final_kernel(const SamplePart *part, int rows,
                                                                           int chunks, int32_t *tokens,
                                                                           int32_t *dev_err) {
  const int row = blockIdx.x * (kSmpThreads / kWave) + threadIdx.x / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  if (row >= rows) return;
  float best = -INFINITY;
  int best_i = 0x7fffffff;
  for (int c = lane; c < chunks; c += kWave) {
    const SamplePart q = part[static_cast<size_t>(row) * chunks + c];
    arg_better(best, best_i, q.v, q.i);
  }
  wave_argmax(best, best_i);
  if (lane == 0) {
    if (best_i == 0x7fffffff) {             // every value of the row was NaN
      report(dev_err, 6 /*RECO_DEV_BAD_LOGIT*/);
      best_i = -1;
    }
    tokens[row] = best_i;
  }
}

constexpr int kPplThreads = 256;
constexpr int kPplChunk = 16384;   // logits per workgroup

// Per (row, chunk): the chunk's max and sum of exp(z - max), natural log domain.
// Each thread holds its logits of the chunk in registers (all requested in
// one round trip, as 16-byte non-temporal loads where the rows allow), so
// the max and the sum need a single read of the chunk.
template <bool VEC>
__global__ __launch_bounds__(kPplThreads) void ppl_partial_kernel(const float *logits, int vocab, int chunks,
                                                                  float *part) {
  constexpr int kPer = kPplChunk / kPplThreads;
  __shared__ float red[kPplThreads / kWave];
  const int chunk = blockIdx.x;
  const size_t row = blockIdx.y;
  const int c0 = chunk * kPplChunk;
  const int c1 = min(vocab, c0 + kPplChunk);
  const float *z = logits + row * static_cast<size_t>(vocab);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;

  float x[kPer];
  if constexpr (VEC) {
#pragma unroll
    for (int i = 0; i < kPer / 4; ++i) {
      const int j = c0 + (i * kPplThreads + static_cast<int>(threadIdx.x)) * 4;   // c1 - j is a multiple of 4
      const uint4 u = j < c1 ? nt_load_u4(z + j) : make_uint4(0xff800000u, 0xff800000u, 0xff800000u, 0xff800000u);
      x[4 * i + 0] = __uint_as_float(u.x);
      x[4 * i + 1] = __uint_as_float(u.y);
      x[4 * i + 2] = __uint_as_float(u.z);
      x[4 * i + 3] = __uint_as_float(u.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int j = c0 + i * kPplThreads + static_cast<int>(threadIdx.x);
      x[i] = j < c1 ? z[j] : -INFINITY;
    }
  }
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kPer; ++i) m = fmaxf(m, x[i]);
  m = wave_max(m);
  if (lane == 0) red[wave] = m;
  __syncthreads();
  float M = red[0];
#pragma unroll
  for (int w = 1; w < kPplThreads / kWave; ++w) M = fmaxf(M, red[w]);
  __syncthreads();
  float s = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) s += expf(x[i] - M);     // x = -inf (past the row) adds 0
  }
  s = wave_sum(s);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float S = 0.f;
#pragma unroll
    for (int w = 0; w < kPplThreads / kWave; ++w) S += red[w];
    part[(row * chunks + chunk) * 2 + 0] = M;
    part[(row * chunks + chunk) * 2 + 1] = S;
  }
}

// Per sequence: LSE of every answer position (fp64 merge of the chunk
// partials), the mean negative log-likelihood, PPL and the stop flag.
__global__ __launch_bounds__(kPplThreads) void ppl_final_kernel(const float *logits, const int32_t *tokens, int n,
                                                                int vocab, int chunks, const float *part,
                                                                float tau_p, float *ppl, int32_t *stop,
                                                                int32_t *dev_err) {
  __shared__ double red[kPplThreads];
  const int b = blockIdx.x;
  double nll = 0.0;
  bool bad = false;
  for (int t = threadIdx.x; t < n; t += kPplThreads) {
    const size_t row = static_cast<size_t>(b) * n + t;
    const float *pr = part + row * chunks * 2;
    float M = -INFINITY;
    for (int c = 0; c < chunks; ++c) M = fmaxf(M, pr[2 * c]);
    double S = 0.0;
    for (int c = 0; c < chunks; ++c)
      if (pr[2 * c] != -INFINITY) S += static_cast<double>(pr[2 * c + 1]) * exp(static_cast<double>(pr[2 * c]) - M);
    const double lse = static_cast<double>(M) + log(S);
    const int x = tokens[row];
    if (x < 0 || x >= vocab) {
      bad = true;
      continue;
    }
    nll += lse - static_cast<double>(logits[row * vocab + x]);
  }
  red[threadIdx.x] = bad ? NAN : nll;
  __syncthreads();
  for (int s = kPplThreads / 2; s > 0; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double total = red[0];
    if (isnan(total)) report(dev_err, 4 /*RECO_DEV_BAD_TOKEN_ID*/);
    const double pp = exp(total / n);
    ppl[b] = static_cast<float>(pp);
    if (stop) stop[b] = (pp <= static_cast<double>(tau_p)) ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_logit_penalty(float *logits, int rows, int vocab, int64_t ld, const int32_t *ids, int n_ids,
                                const float *reward, float tau_lo, float tau_hi, float b_lo, float b_mid,
                                float b_hi, int32_t *dev_err, hipStream_t s) {
  hipLaunchKernelGGL(logit_penalty_kernel, dim3(rows), dim3(kPenThreads), 0, s, logits, vocab, ld, ids, n_ids,
                     reward, tau_lo, tau_hi, b_lo, b_mid, b_hi, dev_err);
  return hipGetLastError();
}

size_t penalty_sample_workspace_bytes(int rows, int vocab) {
  const size_t chunks = static_cast<size_t>((static_cast<int64_t>(vocab) + kSmpChunk - 1) / kSmpChunk);
  return static_cast<size_t>(rows) * chunks * sizeof(SamplePart);
}

hipError_t launch_penalty_sample(float *logits, int rows, int vocab, int64_t ld, const int32_t *ids, int n_ids,
                                 const float *reward, float tau_lo, float tau_hi, float b_lo, float b_mid,
                                 float b_hi, float temperature, uint64_t seed, uint64_t offset, int32_t *tokens,
                                 void *ws, int32_t *dev_err, hipStream_t s) {
  const int chunks = static_cast<int>((static_cast<int64_t>(vocab) + kSmpChunk - 1) / kSmpChunk);
  SamplePart *part = reinterpret_cast<SamplePart *>(ws);
  hipLaunchKernelGGL(penalty_sample_partial_kernel, dim3(chunks, rows), dim3(kSmpThreads), 0, s, logits, vocab, ld,
                     ids, n_ids, reward, tau_lo, tau_hi, b_lo, b_mid, b_hi, temperature,
                     static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), static_cast<uint32_t>(offset),
                     static_cast<uint32_t>(offset >> 32), chunks, part, dev_err);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int per_wg = kSmpThreads / kWave;
  hipLaunchKernelGGL(penalty_sample_final_kernel, dim3((rows + per_wg - 1) / per_wg), dim3(kSmpThreads), 0, s, part,
                     rows, chunks, tokens, dev_err);
  return hipGetLastError();
}

size_t ppl_workspace_bytes(int batch, int n, int vocab) {
  const size_t chunks = static_cast<size_t>((static_cast<int64_t>(vocab) + kPplChunk - 1) / kPplChunk);
  return static_cast<size_t>(batch) * n * chunks * 2 * sizeof(float);
}

hipError_t launch_answer_ppl(const float *logits, const int32_t *tokens, int batch, int n, int vocab, float tau_p,
                             float *ppl, int32_t *stop, void *ws, int32_t *dev_err, hipStream_t s) {
  const int chunks = static_cast<int>((static_cast<int64_t>(vocab) + kPplChunk - 1) / kPplChunk);
  float *part = reinterpret_cast<float *>(ws);
  const bool vec = vocab % 4 == 0 && reinterpret_cast<uintptr_t>(logits) % 16 == 0;
  if (vec)
    hipLaunchKernelGGL(ppl_partial_kernel<true>, dim3(chunks, batch * n), dim3(kPplThreads), 0, s, logits, vocab,
                       chunks, part);
  else
    hipLaunchKernelGGL(ppl_partial_kernel<false>, dim3(chunks, batch * n), dim3(kPplThreads), 0, s, logits, vocab,
                       chunks, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ppl_final_kernel, dim3(batch), dim3(kPplThreads), 0, s, logits, tokens, n, vocab, chunks, part,
                     tau_p, ppl, stop, dev_err);
  return hipGetLastError();
}

}  // namespace reco
