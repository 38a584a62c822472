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
 * (pda_work_order + pda_decode_reusing_order) gives bitwise the same output,
 * and that invalid arguments come back as status codes.  Exit status 0 means
 * every check passed.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pda.h"

/* The oracle's entry point (oracle/pda_oracle.c): single-query attention in fp64. */
int pda_oracle_decode(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                      const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                      const int32_t *block_table, const int32_t *context_lens, double scale, double *out,
                      int num_threads);

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

  CHECK_HIP(hipStreamDestroy(stream));
  hipFree(dq); hipFree(dk); hipFree(dv); hipFree(dbt); hipFree(dlens); hipFree(dout); hipFree(dout2);
  free(perm); free(bt); free(q); free(k); free(v); free(ref); free(out); free(out2);
  printf("%s\n", failures ? "C client: FAILED" : "C client: all checks passed");
  return failures ? 1 : 0;
}
