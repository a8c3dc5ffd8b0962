// Generation-side kernels of Section 3.3 (gfx950):
//   reflection-token penalty, Eq. 3 (reward band) and Eq. 4 (subtract beta);
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

constexpr int kPplThreads = 256;
constexpr int kPplChunk = 16384;   // logits per workgroup

// Per (row, chunk): the chunk's max and sum of exp(z - max), natural log domain.
__global__ __launch_bounds__(kPplThreads) void ppl_partial_kernel(const float *logits, int vocab, int chunks,
                                                                  float *part) {
  __shared__ float red[kPplThreads / kWave];
  const int chunk = blockIdx.x;
  const size_t row = blockIdx.y;
  const int c0 = chunk * kPplChunk;
  const int c1 = min(vocab, c0 + kPplChunk);
  const float *z = logits + row * static_cast<size_t>(vocab);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;

  float m = -INFINITY;
  for (int j = c0 + threadIdx.x; j < c1; j += kPplThreads) m = fmaxf(m, z[j]);
  m = wave_max(m);
  if (lane == 0) red[wave] = m;
  __syncthreads();
  float M = red[0];
#pragma unroll
  for (int w = 1; w < kPplThreads / kWave; ++w) M = fmaxf(M, red[w]);
  __syncthreads();
  float s = 0.f;
  if (M != -INFINITY)
    for (int j = c0 + threadIdx.x; j < c1; j += kPplThreads) s += expf(z[j] - M);
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
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
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

size_t ppl_workspace_bytes(int batch, int n, int vocab) {
  const size_t chunks = static_cast<size_t>((vocab + kPplChunk - 1) / kPplChunk);
  return static_cast<size_t>(batch) * n * chunks * 2 * sizeof(float);
}

hipError_t launch_answer_ppl(const float *logits, const int32_t *tokens, int batch, int n, int vocab, float tau_p,
                             float *ppl, int32_t *stop, void *ws, int32_t *dev_err, hipStream_t s) {
  const int chunks = (vocab + kPplChunk - 1) / kPplChunk;
  float *part = reinterpret_cast<float *>(ws);
  hipLaunchKernelGGL(ppl_partial_kernel, dim3(chunks, batch * n), dim3(kPplThreads), 0, s, logits, vocab, chunks,
                     part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ppl_final_kernel, dim3(batch), dim3(kPplThreads), 0, s, logits, tokens, n, vocab, chunks, part,
                     tau_p, ppl, stop, dev_err);
  return hipGetLastError();
}

}  // namespace reco
