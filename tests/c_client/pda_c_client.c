/*
 * A plain C client of the paged decode-attention library: no Python and no
 * PyTorch, only include/pda.h, the HIP runtime for device memory, and the
 * fp64 oracle (test infrastructure) for the expected values.
 *
 * It builds one small seeded decode step (ragged contexts including an
 * empty and a one-token one, blocks placed at random in a pool whose unused
 * slots hold NaN), runs pda_decode with several partition sizes (the
 * library's own among them), compares each output element with the
 * oracle (max-abs 8e-3, mean-abs 1e-3), checks that a reused work order
 * (pda_work_order + pda_decode_reusing_order) and the entry point without
 * allocation (pda_decode_noalloc) give bitwise the same output, and that
 * invalid arguments come back as status codes.  Then 40 new tokens per
 * sequence on the same cache (workgroups of 8 wavefronts, two 16-row tiles
 * each) against the oracle's multi-token attention, and token
 * log-probabilities and entropies of seeded bf16 logits (a small batch,
 * rows split over workgroups through the workspace) against the oracle's.
 * Exit status 0 means every check passed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pda.h"

/* The oracle's entry points (oracle/pda_oracle.c), in fp64: single-query
   and multi-token attention, token log-probabilities and entropies. */
int pda_oracle_decode(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                      const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                      const int32_t *block_table, const int32_t *context_lens, double scale, double *out,
                      int num_threads);
int pda_oracle_decode_multi(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                            const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                            const int32_t *block_table, const int32_t *context_lens, double scale, int n,
                            double *out, int num_threads);
int pda_oracle_logprob(int B, int V, int64_t row_stride, const void *logits, int logits_are_f32,
                       const int32_t *tokens, double inv_temperature, double *logprob, double *entropy);

#define CHECK_HIP(x)                                                              \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
      exit(2);                                                                    \
    }                                                                             \
  } while (0)

static uint64_t rng_state;
static uint64_t next_u64(void) { /* splitmix64 */
  uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
static double uniform(void) { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }
static float normalish(void) { /* four uniforms, centred and scaled to unit variance */
  return (float)((uniform() + uniform() + uniform() + uniform() - 2.0) * 1.7320508075688772);
}
static uint16_t to_bf16(float f) { /* round to nearest even (finite inputs) */
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static int failures = 0;
static void expect(int ok, const char *what) {
  printf("%s: %s\n", ok ? "ok  " : "FAIL", what);
  if (!ok) ++failures;
}

/* max-abs and mean-abs of got (float) against ref (double); 0 when any got is not finite */
static int within(const float *got, const double *ref, size_t n, double max_bar, double mean_bar, const char *what) {
  double max_err = 0.0, sum_err = 0.0;
  int finite = 1;
  for (size_t i = 0; i < n; ++i) {
    if (!isfinite(got[i])) finite = 0;
    const double e = fabs((double)got[i] - ref[i]);
    if (e > max_err) max_err = e;
    sum_err += e;
  }
  printf("%s: max-abs %.3e, mean-abs %.3e over %zu values\n", what, max_err, sum_err / (double)n, n);
  return finite && max_err <= max_bar && sum_err / (double)n <= mean_bar;
}

int main(void) {
  enum { B = 6, HQ = 8, HKV = 2, D = 128, BS = 16 };
  const int32_t lens[B] = {0, 1, 17, 300, 1024, 2049};
  int max_len = 0, used = 0;
  for (int b = 0; b < B; ++b) {
    if (lens[b] > max_len) max_len = lens[b];
    used += (lens[b] + BS - 1) / BS;
  }
  const int MB = (max_len + BS - 1) / BS;
  const int NB = used + used / 8 + 3; /* some blocks belong to nobody */
  rng_state = 20240517u;

  /* random placement: a permutation of the pool, handed out in order */
  int32_t *perm = malloc(sizeof(int32_t) * NB);
  for (int i = 0; i < NB; ++i) perm[i] = i;
  for (int i = NB - 1; i > 0; --i) {
    int j = (int)(next_u64() % (uint64_t)(i + 1));
    int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
  }
  int32_t *bt = malloc(sizeof(int32_t) * B * MB);
  int next = 0;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < MB; ++j) bt[b * MB + j] = j < (lens[b] + BS - 1) / BS ? perm[next++] : -1;

  const size_t nq = (size_t)B * HQ * D, nkv = (size_t)NB * HKV * BS * D;
  uint16_t *q = malloc(nq * 2), *k = malloc(nkv * 2), *v = malloc(nkv * 2);
  for (size_t i = 0; i < nq; ++i) q[i] = to_bf16(normalish());
  for (size_t i = 0; i < nkv; ++i) { k[i] = 0x7fc0u; v[i] = 0x7fc0u; } /* NaN where no token lives */
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < lens[b]; ++t) {
      const int p = bt[b * MB + t / BS], o = t % BS;
      for (int g = 0; g < HKV; ++g)
        for (int d = 0; d < D; ++d) {
          k[((((size_t)p * HKV + g) * (D / 8) + d / 8) * BS + o) * 8 + d % 8] = to_bf16(normalish());
          v[(((size_t)p * HKV + g) * BS + o) * D + d] = to_bf16(normalish());
        }
    }
  const double scale = 1.0 / sqrt((double)D);

  double *ref = malloc(sizeof(double) * nq);
  if (pda_oracle_decode(B, HQ, HKV, D, BS, NB, MB, q, k, v, bt, lens, scale, ref, 1) != 0) {
    fprintf(stderr, "oracle rejected the problem\n");
    return 2;
  }

  void *dq, *dk, *dv, *dbt, *dlens, *dout, *dout2;
  CHECK_HIP(hipMalloc(&dq, nq * 2));
  CHECK_HIP(hipMalloc(&dk, nkv * 2));
  CHECK_HIP(hipMalloc(&dv, nkv * 2));
  CHECK_HIP(hipMalloc(&dbt, sizeof(int32_t) * B * MB));
  CHECK_HIP(hipMalloc(&dlens, sizeof(int32_t) * B));
  CHECK_HIP(hipMalloc(&dout, sizeof(float) * nq));
  CHECK_HIP(hipMalloc(&dout2, sizeof(float) * nq));
  CHECK_HIP(hipMemcpy(dq, q, nq * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dk, k, nkv * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dv, v, nkv * 2, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dbt, bt, sizeof(int32_t) * B * MB, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dlens, lens, sizeof(int32_t) * B, hipMemcpyHostToDevice));
  hipStream_t stream;
  CHECK_HIP(hipStreamCreate(&stream));
  float *out = malloc(sizeof(float) * nq), *out2 = malloc(sizeof(float) * nq);

  /* 129 one-block partitions (more work items than the GPU runs at once, so
     the step takes a work order), 9 partitions, the library's choice, and one
     partition (no merge pass) */
  const int partitions[4] = {16, 256, 0, 2064};
  for (int c = 0; c < 4; ++c) {
    pda_problem prob = {B, HQ, HKV, D, BS, NB, MB, max_len, partitions[c], 1};
    pda_plan_info plan;
    expect(pda_plan(&prob, &plan) == PDA_OK, "pda_plan");
    size_t ws_bytes = 0;
    expect(pda_workspace_bytes(&prob, &ws_bytes) == PDA_OK && ws_bytes == plan.workspace_bytes,
           "pda_workspace_bytes agrees with the plan");
    void *ws;
    CHECK_HIP(hipMalloc(&ws, ws_bytes));
    expect(pda_decode(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout, ws, ws_bytes, stream) == PDA_OK,
           "pda_decode");
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(out, dout, sizeof(float) * nq, hipMemcpyDeviceToHost));
    double max_err = 0.0, sum_err = 0.0;
    int finite = 1;
    for (size_t i = 0; i < nq; ++i) {
      if (!isfinite(out[i])) finite = 0;
      const double e = fabs((double)out[i] - ref[i]);
      if (e > max_err) max_err = e;
      sum_err += e;
    }
    printf("partition_tokens %d (plan: %d tokens, %d partitions): max-abs %.3e, mean-abs %.3e\n",
           partitions[c], plan.partition_tokens, plan.num_partitions, max_err, sum_err / (double)nq);
    expect(finite && max_err <= 8e-3 && sum_err / (double)nq <= 1e-3, "pda_decode matches the oracle");

    /* the work order once, then a decode that reuses it */
    expect(pda_work_order(&prob, dlens, ws, ws_bytes, stream) == PDA_OK, "pda_work_order");
    expect(pda_decode_reusing_order(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout2, ws, ws_bytes, stream) ==
               PDA_OK,
           "pda_decode_reusing_order");
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(out2, dout2, sizeof(float) * nq, hipMemcpyDeviceToHost));
    expect(memcmp(out, out2, sizeof(float) * nq) == 0, "reused work order: bitwise the same output");

    /* errors are status codes, returned before anything is launched */
    expect(pda_decode(&prob, NULL, dk, dv, dbt, dlens, (float)scale, dout, ws, ws_bytes, stream) == PDA_ERR_NULL,
           "NULL q -> PDA_ERR_NULL");
    expect(pda_decode(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout, ws, ws_bytes - 1, stream) ==
               PDA_ERR_WORKSPACE,
           "short workspace -> PDA_ERR_WORKSPACE");
    expect(pda_decode(&prob, dq, dk, dv, dbt, dlens, NAN, dout, ws, ws_bytes, stream) == PDA_ERR_VALUE,
           "NaN scale -> PDA_ERR_VALUE");
    CHECK_HIP(hipFree(ws));
  }
  expect(strlen(pda_status_string(PDA_ERR_SHAPE)) > 0, "pda_status_string");

  /* the entry point without allocation: the library's own scratch as workspace */
  {
    pda_problem prob = {B, HQ, HKV, D, BS, NB, MB, max_len, 0, 1};
    size_t ws_bytes = 0;
    expect(pda_workspace_bytes(&prob, &ws_bytes) == PDA_OK, "pda_workspace_bytes");
    void *ws;
    CHECK_HIP(hipMalloc(&ws, ws_bytes > 0 ? ws_bytes : 16));
    expect(pda_decode(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout, ws, ws_bytes, stream) == PDA_OK,
           "pda_decode");
    expect(pda_decode_noalloc(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout2, stream) == PDA_OK,
           "pda_decode_noalloc");
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(out, dout, sizeof(float) * nq, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(out2, dout2, sizeof(float) * nq, hipMemcpyDeviceToHost));
    expect(memcmp(out, out2, sizeof(float) * nq) == 0, "pda_decode_noalloc: bitwise pda_decode's output");
    CHECK_HIP(hipFree(ws));
  }

  /* 40 new tokens per sequence over the same cache: the last 40 tokens of each
     context are the new ones (rows of a shorter context see nothing) */
  {
    enum { N = 40 };
    const size_t nqm = (size_t)B * N * HQ * D;
    uint16_t *qm = malloc(nqm * 2);
    for (size_t i = 0; i < nqm; ++i) qm[i] = to_bf16(normalish());
    double *refm = malloc(sizeof(double) * nqm);
    expect(pda_oracle_decode_multi(B, HQ, HKV, D, BS, NB, MB, qm, k, v, bt, lens, scale, N, refm, 1) == 0,
           "oracle (40 new tokens)");
    void *dqm, *doutm;
    CHECK_HIP(hipMalloc(&dqm, nqm * 2));
    CHECK_HIP(hipMalloc(&doutm, sizeof(float) * nqm));
    CHECK_HIP(hipMemcpy(dqm, qm, nqm * 2, hipMemcpyHostToDevice));
    pda_problem prob = {B, HQ, HKV, D, BS, NB, MB, max_len, 0, N};
    size_t ws_bytes = 0;
    expect(pda_workspace_bytes(&prob, &ws_bytes) == PDA_OK, "pda_workspace_bytes (40 new tokens)");
    void *ws;
    CHECK_HIP(hipMalloc(&ws, ws_bytes > 0 ? ws_bytes : 16));
    expect(pda_decode(&prob, dqm, dk, dv, dbt, dlens, (float)scale, (float *)doutm, ws, ws_bytes, stream) == PDA_OK,
           "pda_decode (40 new tokens)");
    CHECK_HIP(hipStreamSynchronize(stream));
    float *outm = malloc(sizeof(float) * nqm);
    CHECK_HIP(hipMemcpy(outm, doutm, sizeof(float) * nqm, hipMemcpyDeviceToHost));
    expect(within(outm, refm, nqm, 8e-3, 1e-3, "40 new tokens"), "40 new tokens match the oracle");
    CHECK_HIP(hipFree(ws));
    hipFree(dqm); hipFree(doutm);
    free(qm); free(refm); free(outm);
  }

  /* token log-probabilities and entropies: 12 rows of a 40000-token
     vocabulary (bf16, rows padded to 40008), each row split over 4
     workgroups through the workspace */
  {
    enum { R = 12, V = 40000, STRIDE = 40008 };
    uint16_t *lg = malloc(sizeof(uint16_t) * R * STRIDE);
    int32_t tok[R];
    for (int r = 0; r < R; ++r) {
      for (int j = 0; j < STRIDE; ++j) lg[(size_t)r * STRIDE + j] = to_bf16(2.0f * normalish());
      for (int x = 0; x < 8; ++x) /* a few likely tokens */
        lg[(size_t)r * STRIDE + (next_u64() % V)] = to_bf16(8.0f + 4.0f * (float)uniform());
      tok[r] = (int32_t)(next_u64() % V);
    }
    double ref_lp[R], ref_ent[R];
    expect(pda_oracle_logprob(R, V, STRIDE, lg, 0, tok, 1.0, ref_lp, ref_ent) == 0, "oracle log-probabilities");
    void *dlg, *dtok, *dlp, *dent, *ws;
    CHECK_HIP(hipMalloc(&dlg, sizeof(uint16_t) * R * STRIDE));
    CHECK_HIP(hipMalloc(&dtok, sizeof(tok)));
    CHECK_HIP(hipMalloc(&dlp, sizeof(float) * R));
    CHECK_HIP(hipMalloc(&dent, sizeof(float) * R));
    CHECK_HIP(hipMemcpy(dlg, lg, sizeof(uint16_t) * R * STRIDE, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dtok, tok, sizeof(tok), hipMemcpyHostToDevice));
    size_t ws_bytes = 0;
    expect(pda_logprob_workspace_bytes(R, V, PDA_DTYPE_BF16, &ws_bytes) == PDA_OK && ws_bytes > 0,
           "pda_logprob_workspace_bytes: a small batch splits its rows");
    CHECK_HIP(hipMalloc(&ws, ws_bytes));
    expect(pda_token_logprobs(R, V, STRIDE, PDA_DTYPE_BF16, dlg, (const int32_t *)dtok, 1.0f, (float *)dlp,
                              (float *)dent, ws, ws_bytes, stream) == PDA_OK,
           "pda_token_logprobs");
    CHECK_HIP(hipStreamSynchronize(stream));
    float lp[R], ent[R];
    CHECK_HIP(hipMemcpy(lp, dlp, sizeof(lp), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(ent, dent, sizeof(ent), hipMemcpyDeviceToHost));
    expect(within(lp, ref_lp, R, 1e-4, 1e-4, "log-probabilities"), "log-probabilities match the oracle");
    expect(within(ent, ref_ent, R, 1e-4, 1e-4, "entropies"), "entropies match the oracle");
    hipFree(dlg); hipFree(dtok); hipFree(dlp); hipFree(dent); hipFree(ws);
    free(lg);
  }

  CHECK_HIP(hipStreamDestroy(stream));
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dbt); hipFree(dlens); hipFree(dout); hipFree(dout2);
  free(perm); free(bt); free(q); free(k); free(v); free(ref); free(out); free(out2);
  printf("%s\n", failures ? "C client: FAILED" : "C client: all checks passed");
  return failures ? 1 : 0;
}
