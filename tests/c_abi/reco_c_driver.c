/*
 * Plain C11 client of libreco.so: one compression (Eq. 2 scoring, then
 * reward-budgeted selection and in-place compaction, Section 3.2) followed by
 * decode steps that append their token, then the banded reflection penalty on
 * a block of logit rows (Eq. 3-4) and the answer perplexity with its stop
 * flag (Eq. 5-6): all five calls driven only through the C ABI in reco.h with
 * memory from the HIP runtime (no Python, no torch).
 *
 * Usage: reco_c_driver <input file> <output file>
 *
 * Input (little-endian, written by tests/test_gpu_c_abi.py):
 *   int32  NL, B, H, Hq, D, cap, w, dtype (0 fp32, 1 bf16), nsteps
 *   float  scale
 *   double retention[B]
 *   int32  len[NL][B][H]
 *   elem   K[NL][B][H][cap][D], V[NL][B][H][cap][D]
 *   elem   q_win[NL][B][Hq][w][D]
 *   elem   q[nsteps][NL][B][Hq][D], k_new[nsteps][NL][B][H][D], v_new[nsteps][NL][B][H][D]
 *   int32  rows, vocab, n_refl
 *   float  tau_lo, tau_hi, beta_lo, beta_mid, beta_hi
 *   float  logits[rows][vocab];  int32 refl_ids[n_refl];  float reward[rows]
 *   int32  pb, pn, pv;  float tau_p
 *   float  answer_logits[pb][pn][pv];  int32 answer_tokens[pb][pn]
 * (elem = 4-byte float for fp32, the 2-byte bf16 pattern for bf16)
 *
 * Output:
 *   int32  dev_err
 *   float  scores[NL][B][H][cap]        (as scored, before compaction)
 *   int32  kept[NL][B][H][cap]          (first m entries of each unit valid)
 *   int32  len[NL][B][H]                (after the decode steps)
 *   elem   out[nsteps][NL][B][Hq][D]
 *   float  lse[nsteps][NL][B][Hq]
 *   float  logits[rows][vocab]          (after the penalty, in place)
 *   float  ppl[pb];  int32 stop[pb]
 *
 * Every HIP and library status is checked; any failure prints a message and
 * exits with status 1 before the output file is written.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "reco.h"

#define HIP_CHECK(x)                                                                  \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      fprintf(stderr, "%s:%d: %s failed: %s\n", __FILE__, __LINE__, #x,               \
              hipGetErrorString(e_));                                                 \
      exit(1);                                                                        \
    }                                                                                 \
  } while (0)

#define RECO_CHECK(x)                                                                 \
  do {                                                                                \
    reco_status_t s_ = (x);                                                           \
    if (s_ != RECO_OK) {                                                              \
      fprintf(stderr, "%s:%d: %s failed: %s\n", __FILE__, __LINE__, #x,               \
              reco_status_str(s_));                                                   \
      exit(1);                                                                        \
    }                                                                                 \
  } while (0)

static void read_exact(FILE *f, void *dst, size_t bytes, const char *what) {
  if (bytes && fread(dst, 1, bytes, f) != bytes) {
    fprintf(stderr, "short read: %s (%zu bytes)\n", what, bytes);
    exit(1);
  }
}

static void write_exact(FILE *f, const void *src, size_t bytes) {
  if (bytes && fwrite(src, 1, bytes, f) != bytes) {
    fprintf(stderr, "short write (%zu bytes)\n", bytes);
    exit(1);
  }
}

/* Host buffer of `bytes` read from the input, copied to a new device buffer. */
static void *upload(FILE *f, size_t bytes, const char *what) {
  void *h = malloc(bytes ? bytes : 1), *d = NULL;
  if (!h) {
    fprintf(stderr, "out of host memory (%s)\n", what);
    exit(1);
  }
  read_exact(f, h, bytes, what);
  HIP_CHECK(hipMalloc(&d, bytes ? bytes : 1));
  HIP_CHECK(hipMemcpy(d, h, bytes, hipMemcpyHostToDevice));
  free(h);
  return d;
}

/* Device buffer of `bytes` copied back and appended to the output. */
static void download(FILE *f, const void *d, size_t bytes) {
  void *h = malloc(bytes ? bytes : 1);
  if (!h) {
    fprintf(stderr, "out of host memory\n");
    exit(1);
  }
  HIP_CHECK(hipMemcpy(h, d, bytes, hipMemcpyDeviceToHost));
  write_exact(f, h, bytes);
  free(h);
}

int main(int argc, char **argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s <input> <output>\n", argv[0]);
    return 2;
  }
  if (reco_abi_version() != RECO_ABI_VERSION) {
    fprintf(stderr, "library ABI %d, header ABI %d\n", reco_abi_version(), RECO_ABI_VERSION);
    return 1;
  }
  FILE *in = fopen(argv[1], "rb");
  if (!in) {
    perror(argv[1]);
    return 1;
  }
  int32_t hdr[9];
  read_exact(in, hdr, sizeof hdr, "header");
  const int32_t NL = hdr[0], B = hdr[1], H = hdr[2], Hq = hdr[3], D = hdr[4], cap = hdr[5], w = hdr[6];
  const int32_t dtype = hdr[7], nsteps = hdr[8];
  if (NL < 1 || B < 1 || H < 1 || Hq < H || D < 1 || cap < 1 || w < 1 || nsteps < 0 || (dtype != 0 && dtype != 1)) {
    fprintf(stderr, "bad header\n");
    return 1;
  }
  float scale;
  read_exact(in, &scale, sizeof scale, "scale");
  const size_t e = dtype == 0 ? 4 : 2;
  const size_t units = (size_t)NL * B * H;
  const size_t qrows = (size_t)NL * B * Hq;

  void *d_ret = upload(in, sizeof(double) * B, "retention");
  int32_t *d_len = (int32_t *)upload(in, sizeof(int32_t) * units, "len");
  void *d_k = upload(in, units * cap * D * e, "K");
  void *d_v = upload(in, units * cap * D * e, "V");
  void *d_qwin = upload(in, qrows * w * D * e, "q_win");
  void *d_q = upload(in, (size_t)nsteps * qrows * D * e, "q");
  void *d_kn = upload(in, (size_t)nsteps * units * D * e, "k_new");
  void *d_vn = upload(in, (size_t)nsteps * units * D * e, "v_new");
  int32_t phdr[3];
  float pen[5];
  read_exact(in, phdr, sizeof phdr, "penalty header");
  read_exact(in, pen, sizeof pen, "penalty bands");
  const int32_t rows = phdr[0], vocab = phdr[1], n_refl = phdr[2];
  if (rows < 1 || vocab < 1 || n_refl < 0) {
    fprintf(stderr, "bad penalty header\n");
    return 1;
  }
  float *d_logits = (float *)upload(in, (size_t)rows * vocab * sizeof(float), "logits");
  int32_t *d_refl = (int32_t *)upload(in, (size_t)n_refl * sizeof(int32_t), "refl_ids");
  float *d_reward = (float *)upload(in, (size_t)rows * sizeof(float), "reward");
  int32_t ahdr[3];
  float tau_p;
  read_exact(in, ahdr, sizeof ahdr, "answer header");
  read_exact(in, &tau_p, sizeof tau_p, "tau_p");
  const int32_t pb = ahdr[0], pn = ahdr[1], pv = ahdr[2];
  if (pb < 1 || pn < 1 || pv < 1) {
    fprintf(stderr, "bad answer header\n");
    return 1;
  }
  float *d_alog = (float *)upload(in, (size_t)pb * pn * pv * sizeof(float), "answer logits");
  int32_t *d_atok = (int32_t *)upload(in, (size_t)pb * pn * sizeof(int32_t), "answer tokens");
  fclose(in);

  reco_kv_cache_t cache;
  cache.k = d_k;
  cache.v = d_v;
  cache.len = d_len;
  cache.n_layers = NL;
  cache.batch = B;
  cache.n_kv_heads = H;
  cache.capacity = cap;
  cache.head_dim = D;
  cache.dtype = dtype == 0 ? RECO_F32 : RECO_BF16;

  hipStream_t stream;
  HIP_CHECK(hipStreamCreate(&stream));
  int32_t *d_err = NULL;
  float *d_scores = NULL, *d_lse = NULL;
  int32_t *d_kept = NULL;
  void *d_out = NULL;
  HIP_CHECK(hipMalloc((void **)&d_err, sizeof(int32_t)));
  HIP_CHECK(hipMemsetAsync(d_err, 0, sizeof(int32_t), stream));
  HIP_CHECK(hipMalloc((void **)&d_scores, units * cap * sizeof(float)));
  HIP_CHECK(hipMemsetAsync(d_scores, 0, units * cap * sizeof(float), stream));
  HIP_CHECK(hipMalloc((void **)&d_kept, units * cap * sizeof(int32_t)));
  HIP_CHECK(hipMemsetAsync(d_kept, 0xff, units * cap * sizeof(int32_t), stream));
  HIP_CHECK(hipMalloc(&d_out, (size_t)(nsteps ? nsteps : 1) * qrows * D * e));
  HIP_CHECK(hipMalloc((void **)&d_lse, (size_t)(nsteps ? nsteps : 1) * qrows * sizeof(float)));

  /* Workspaces: sized by the library, owned here, one per entry point. */
  const size_t ws_score_bytes = reco_score_workspace_size(&cache, NL, Hq, w);
  const size_t ws_sel_bytes = reco_select_compact_workspace_size(&cache, NL);
  const size_t ws_dec_bytes = reco_decode_attn_workspace_size(&cache, NL, Hq);
  if (!ws_score_bytes || !ws_sel_bytes || !ws_dec_bytes) {
    fprintf(stderr, "a workspace size query refused the shape\n");
    return 1;
  }
  void *ws_score = NULL, *ws_sel = NULL, *ws_dec = NULL;
  HIP_CHECK(hipMalloc(&ws_score, ws_score_bytes));
  HIP_CHECK(hipMalloc(&ws_sel, ws_sel_bytes));
  HIP_CHECK(hipMalloc(&ws_dec, ws_dec_bytes));

  /* Compression: score (causal window), then select + compact in place. */
  RECO_CHECK(reco_score(&cache, 0, NL, d_qwin, Hq, w, scale, RECO_SCORE_CAUSAL, NULL, d_scores, ws_score,
                        ws_score_bytes, d_err, stream));
  RECO_CHECK(reco_select_compact(&cache, 0, NL, d_scores, (const double *)d_ret, 0, w, d_kept, ws_sel,
                                 ws_sel_bytes, d_err, stream));
  /* Decode steps over all layers, each appending its token. */
  for (int32_t s = 0; s < nsteps; ++s) {
    const char *q = (const char *)d_q + (size_t)s * qrows * D * e;
    const char *kn = (const char *)d_kn + (size_t)s * units * D * e;
    const char *vn = (const char *)d_vn + (size_t)s * units * D * e;
    char *out = (char *)d_out + (size_t)s * qrows * D * e;
    float *lse = d_lse + (size_t)s * qrows;
    RECO_CHECK(reco_decode_attn(&cache, 0, NL, q, Hq, scale, kn, vn, out, lse, NULL, ws_dec, ws_dec_bytes, d_err,
                                stream));
  }
  /* Eq. 3-4 on the logit rows (in place), then Eq. 5-6 on the answer probe. */
  RECO_CHECK(reco_logit_penalty(d_logits, rows, vocab, vocab, d_refl, n_refl, d_reward, pen[0], pen[1], pen[2],
                                pen[3], pen[4], d_err, stream));
  float *d_ppl = NULL;
  int32_t *d_stop = NULL;
  HIP_CHECK(hipMalloc((void **)&d_ppl, (size_t)pb * sizeof(float)));
  HIP_CHECK(hipMalloc((void **)&d_stop, (size_t)pb * sizeof(int32_t)));
  const size_t ws_ppl_bytes = reco_answer_ppl_workspace_size(pb, pn, pv);
  if (!ws_ppl_bytes) {
    fprintf(stderr, "the answer-ppl workspace query refused the shape\n");
    return 1;
  }
  void *ws_ppl = NULL;
  HIP_CHECK(hipMalloc(&ws_ppl, ws_ppl_bytes));
  RECO_CHECK(reco_answer_ppl(d_alog, d_atok, pb, pn, pv, tau_p, d_ppl, d_stop, ws_ppl, ws_ppl_bytes, d_err,
                             stream));
  HIP_CHECK(hipStreamSynchronize(stream));

  FILE *outf = fopen(argv[2], "wb");
  if (!outf) {
    perror(argv[2]);
    return 1;
  }
  download(outf, d_err, sizeof(int32_t));
  download(outf, d_scores, units * cap * sizeof(float));
  download(outf, d_kept, units * cap * sizeof(int32_t));
  download(outf, d_len, units * sizeof(int32_t));
  download(outf, d_out, (size_t)nsteps * qrows * D * e);
  download(outf, d_lse, (size_t)nsteps * qrows * sizeof(float));
  download(outf, d_logits, (size_t)rows * vocab * sizeof(float));
  download(outf, d_ppl, (size_t)pb * sizeof(float));
  download(outf, d_stop, (size_t)pb * sizeof(int32_t));
  if (fclose(outf) != 0) {
    perror(argv[2]);
    return 1;
  }

  void *bufs[] = {d_ret, d_len, d_k, d_v, d_qwin, d_q, d_kn, d_vn, d_err, d_scores, d_kept, d_out, d_lse,
                  ws_score, ws_sel, ws_dec, d_logits, d_refl, d_reward, d_alog, d_atok, d_ppl, d_stop, ws_ppl};
  for (size_t i = 0; i < sizeof bufs / sizeof bufs[0]; ++i) HIP_CHECK(hipFree(bufs[i]));
  HIP_CHECK(hipStreamDestroy(stream));
  return 0;
}
