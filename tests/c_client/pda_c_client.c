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
 * (pda_work_order + pda_decode_reusing_order, or pass 1 alone on it with
 * pda_partition_attention_reusing_order + pda_merge_partitions) and the
 * entry point without
 * allocation (pda_decode_noalloc) give bitwise the same output, and that
 * invalid arguments come back as status codes.  Then 40 new tokens per
 * sequence on the same cache (workgroups of 8 wavefronts, two 16-row tiles
 * each) against the oracle's multi-token attention, and token
 * log-probabilities and entropies of seeded bf16 logits (a small batch,
 * rows split over workgroups through the workspace) against the oracle's.
 * Last, a shared-prefix group of 20 samples (more than one prefix item's
 * members) with one and with three new tokens per sequence, against the
 * oracle's plain attention over the same block tables.
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
    /* pass 1 alone on the same order, then the merge: the same bits */
    CHECK_HIP(hipMemset(dout2, 0, sizeof(float) * nq));
    expect(pda_partition_attention_reusing_order(&prob, dq, dk, dv, dbt, dlens, (float)scale, dout2, ws, ws_bytes,
                                                 stream) == PDA_OK,
           "pda_partition_attention_reusing_order");
    expect(pda_merge_partitions(&prob, dlens, dout2, ws, ws_bytes, stream) == PDA_OK, "pda_merge_partitions");
    CHECK_HIP(hipStreamSynchronize(stream));
    CHECK_HIP(hipMemcpy(out2, dout2, sizeof(float) * nq, hipMemcpyDeviceToHost));
    expect(memcmp(out, out2, sizeof(float) * nq) == 0, "pass 1 on the reused order + merge: bitwise the same output");

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

  /* shared-prefix groups (parallel sampling): 20 samples of one prompt whose
     block tables start with the same 4 prefix blocks (64 tokens), one sample
     with no tokens of its own, two sequences in no group.  The prefix is
     attended once per row group: 16 samples at one new token (G = 4), 5 at
     three.  Expected: the oracle's plain attention over the same tables. */
  {
    enum { M = 20, LONERS = 2, B2 = M + LONERS, PL = 64, PB = PL / BS };
    int32_t lens2[B2];
    for (int b = 0; b < B2; ++b) lens2[b] = b < M ? PL + 1 + (int)(next_u64() % 300) : 50 + 200 * (b - M);
    lens2[3] = PL; /* its last token (the new one, or the three new ones) lies in the prefix */
    int ml = 0, used2 = PB;
    for (int b = 0; b < B2; ++b) {
      if (lens2[b] > ml) ml = lens2[b];
      used2 += (lens2[b] + BS - 1) / BS - (b < M ? PB : 0);
    }
    const int MB2 = (ml + BS - 1) / BS, NB2 = used2 + 7;
    int32_t *perm2 = malloc(sizeof(int32_t) * NB2);
    for (int i = 0; i < NB2; ++i) perm2[i] = i;
    for (int i = NB2 - 1; i > 0; --i) {
      int j = (int)(next_u64() % (uint64_t)(i + 1));
      int32_t t = perm2[i]; perm2[i] = perm2[j]; perm2[j] = t;
    }
    int32_t *bt2 = malloc(sizeof(int32_t) * B2 * MB2);
    int nxt = PB; /* perm2[0 .. PB-1] are the prefix blocks */
    for (int b = 0; b < B2; ++b)
      for (int j = 0; j < MB2; ++j)
        bt2[b * MB2 + j] = j >= (lens2[b] + BS - 1) / BS ? -1 : (b < M && j < PB) ? perm2[j] : perm2[nxt++];
    const size_t nkv2 = (size_t)NB2 * HKV * BS * D;
    uint16_t *k2 = malloc(nkv2 * 2), *v2 = malloc(nkv2 * 2);
    for (size_t i = 0; i < nkv2; ++i) { k2[i] = 0x7fc0u; v2[i] = 0x7fc0u; } /* unused blocks: NaN */
    for (int i = 0; i < nxt; ++i) /* every slot of a used block, so shared slots hold one value */
      for (size_t e = 0; e < (size_t)HKV * BS * D; ++e) {
        k2[(size_t)perm2[i] * HKV * BS * D + e] = to_bf16(normalish());
        v2[(size_t)perm2[i] * HKV * BS * D + e] = to_bf16(normalish());
      }
    const int32_t gstart[2] = {0, M}, gprefix[1] = {PL};
    void *dk2, *dv2, *dbt2, *dlens2, *dgs, *dgp;
    CHECK_HIP(hipMalloc(&dk2, nkv2 * 2));
    CHECK_HIP(hipMalloc(&dv2, nkv2 * 2));
    CHECK_HIP(hipMalloc(&dbt2, sizeof(int32_t) * B2 * MB2));
    CHECK_HIP(hipMalloc(&dlens2, sizeof(lens2)));
    CHECK_HIP(hipMalloc(&dgs, sizeof(gstart)));
    CHECK_HIP(hipMalloc(&dgp, sizeof(gprefix)));
    CHECK_HIP(hipMemcpy(dk2, k2, nkv2 * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dv2, v2, nkv2 * 2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dbt2, bt2, sizeof(int32_t) * B2 * MB2, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dlens2, lens2, sizeof(lens2), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dgs, gstart, sizeof(gstart), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dgp, gprefix, sizeof(gprefix), hipMemcpyHostToDevice));
    const pda_prefix_groups groups = {1, M, PL, (const int32_t *)dgs, (const int32_t *)dgp};
    for (int n = 1; n <= 3; n += 2) {
      const size_t nq2 = (size_t)B2 * n * HQ * D;
      uint16_t *q2 = malloc(nq2 * 2);
      for (size_t i = 0; i < nq2; ++i) q2[i] = to_bf16(normalish());
      double *ref2 = malloc(sizeof(double) * nq2);
      expect(pda_oracle_decode_multi(B2, HQ, HKV, D, BS, NB2, MB2, q2, k2, v2, bt2, lens2, scale, n, ref2, 1) == 0,
             "oracle (shared prefix)");
      void *dq2, *dout3;
      CHECK_HIP(hipMalloc(&dq2, nq2 * 2));
      CHECK_HIP(hipMalloc(&dout3, sizeof(float) * nq2));
      CHECK_HIP(hipMemcpy(dq2, q2, nq2 * 2, hipMemcpyHostToDevice));
      pda_problem prob = {B2, HQ, HKV, D, BS, NB2, MB2, ml, 0, n};
      pda_plan_info plan;
      expect(pda_plan_shared_prefix(&prob, &groups, &plan) == PDA_OK, "pda_plan_shared_prefix");
      void *ws;
      CHECK_HIP(hipMalloc(&ws, plan.workspace_bytes));
      expect(pda_decode_shared_prefix(&prob, &groups, dq2, dk2, dv2, (const int32_t *)dbt2, (const int32_t *)dlens2,
                                      (float)scale, (float *)dout3, ws, plan.workspace_bytes, stream) == PDA_OK,
             "pda_decode_shared_prefix");
      CHECK_HIP(hipStreamSynchronize(stream));
      float *out3 = malloc(sizeof(float) * nq2);
      CHECK_HIP(hipMemcpy(out3, dout3, sizeof(float) * nq2, hipMemcpyDeviceToHost));
      expect(within(out3, ref2, nq2, 8e-3, 1e-3, n == 1 ? "shared prefix, 20 samples" : "shared prefix, 3 new tokens"),
             "shared-prefix step matches the oracle");
      expect(pda_decode_shared_prefix(&prob, &groups, dq2, dk2, dv2, (const int32_t *)dbt2, (const int32_t *)dlens2,
                                      (float)scale, (float *)dout3, ws, plan.workspace_bytes - 1, stream) ==
                 PDA_ERR_WORKSPACE,
             "short workspace -> PDA_ERR_WORKSPACE");
      CHECK_HIP(hipFree(ws));
      hipFree(dq2); hipFree(dout3);
      free(q2); free(ref2); free(out3);
    }
    hipFree(dk2); hipFree(dv2); hipFree(dbt2); hipFree(dlens2); hipFree(dgs); hipFree(dgp);
    free(perm2); free(bt2); free(k2); free(v2);
  }

  CHECK_HIP(hipStreamDestroy(stream));
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dbt); hipFree(dlens); hipFree(dout); hipFree(dout2);
  free(perm); free(bt); free(q); free(k); free(v); free(ref); free(out); free(out2);
  printf("%s\n", failures ? "C client: FAILED" : "C client: all checks passed");
  return failures ? 1 : 0;
}
