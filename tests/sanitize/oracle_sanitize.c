/*
 * Sanitizer driver for the CPU oracle (test infrastructure).  Built together
 * with oracle/pda_oracle.c under AddressSanitizer + UndefinedBehaviorSanitizer
 * or ThreadSanitizer, it calls every oracle entry point on small seeded
 * problems -- ragged and empty contexts, partial last blocks, shuffled block
 * tables, several query tokens, all thread counts from 1 to 8 -- and checks
 * that the multi-threaded results are bitwise those of one thread.  Any
 * out-of-bounds access, undefined operation or data race aborts the run
 * through the sanitizer; a result mismatch returns a nonzero status.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int pda_oracle_decode(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                      const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                      const int32_t *block_table, const int32_t *context_lens, double scale, double *out,
                      int num_threads);
int pda_oracle_decode_multi(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                            const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                            const int32_t *block_table, const int32_t *context_lens, double scale, int n,
                            double *out, int num_threads);
int pda_oracle_decode_rows(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                           const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                           const int32_t *block_table, const int32_t *context_lens, double scale, int n,
                           const int32_t *rows, int n_rows, double *out, int num_threads);
int pda_oracle_weights(int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                       const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,
                       const int32_t *block_table, const int32_t *context_lens, double scale, int b, int h,
                       double *w);
int pda_oracle_append(int B, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq, int n,
                      const uint16_t *k_new, const uint16_t *v_new, const int32_t *block_table,
                      const int32_t *context_lens, uint16_t *k_cache, uint16_t *v_cache);
int pda_oracle_logprob(int B, int V, int64_t row_stride, const void *logits, int logits_are_f32,
                       const int32_t *tokens, double inv_temperature, double *logprob, double *entropy);

static uint64_t state = 2405;
static uint32_t next_u32(void) { /* xorshift64* */
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 2685821657736338717ull) >> 32);
}
/* a bf16 pattern of a value in about [-4, 4] (exponent 0x7c..0x80) */
static uint16_t small_bf16(void) {
  const uint32_t r = next_u32();
  return (uint16_t)(((r & 1u) << 15) | ((0x7cu + (r >> 1) % 5u) << 7) | ((r >> 4) & 0x7fu));
}

static int fails = 0;
static void expect_same(const double *a, const double *b, size_t n, const char *what) {
  if (memcmp(a, b, n * sizeof(double)) != 0) {
    fprintf(stderr, "mismatch: %s\n", what);
    ++fails;
  }
}

static void attention_case(int B, int Hq, int Hkv, int D, int nq, const int32_t *lens_in) {
  const int BS = 16;
  int max_len = 1;
  for (int b = 0; b < B; ++b) max_len = lens_in[b] > max_len ? lens_in[b] : max_len;
  const int mbps = (max_len + BS - 1) / BS + 1;
  const int nblocks = B * mbps + 3;
  uint16_t *q = malloc(sizeof(uint16_t) * (size_t)B * nq * Hq * D);
  uint16_t *k = malloc(sizeof(uint16_t) * (size_t)nblocks * Hkv * D * BS);
  uint16_t *v = malloc(sizeof(uint16_t) * (size_t)nblocks * Hkv * D * BS);
  int32_t *bt = malloc(sizeof(int32_t) * (size_t)B * mbps);
  int32_t *lens = malloc(sizeof(int32_t) * (size_t)B);
  int32_t *perm = malloc(sizeof(int32_t) * (size_t)nblocks);
  for (size_t i = 0; i < (size_t)B * nq * Hq * D; ++i) q[i] = small_bf16();
  for (size_t i = 0; i < (size_t)nblocks * Hkv * D * BS; ++i) {
    k[i] = small_bf16();
    v[i] = small_bf16();
  }
  for (int i = 0; i < nblocks; ++i) perm[i] = i;
  for (int i = nblocks - 1; i > 0; --i) { /* Fisher-Yates */
    const int j = (int)(next_u32() % (uint32_t)(i + 1));
    const int32_t t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  for (int b = 0; b < B; ++b) {
    lens[b] = lens_in[b];
    for (int j = 0; j < mbps; ++j) bt[b * mbps + j] = perm[b * mbps + j];
  }
  const size_t rows = (size_t)B * nq * Hq;
  double *o1 = malloc(sizeof(double) * rows * D), *o8 = malloc(sizeof(double) * rows * D);
  const double scale = 1.0 / sqrt((double)D);
  for (int threads = 1; threads <= 8; ++threads) {
    double *dst = threads == 1 ? o1 : o8;
    int rc = nq == 1 ? pda_oracle_decode(B, Hq, Hkv, D, BS, nblocks, mbps, q, k, v, bt, lens, scale, dst, threads)
                     : pda_oracle_decode_multi(B, Hq, Hkv, D, BS, nblocks, mbps, q, k, v, bt, lens, scale, nq, dst,
                                               threads);
    if (rc != 0) {
      fprintf(stderr, "attention rc %d\n", rc);
      ++fails;
    }
    if (threads > 1) expect_same(o1, o8, rows * D, "threads");
  }
  /* a few rows one by one */
  int32_t trip[3 * 5];
  for (int r = 0; r < 5; ++r) {
    trip[3 * r] = (int32_t)(next_u32() % (uint32_t)B);
    trip[3 * r + 1] = (int32_t)(next_u32() % (uint32_t)nq);
    trip[3 * r + 2] = (int32_t)(next_u32() % (uint32_t)Hq);
  }
  double *orow = malloc(sizeof(double) * 5 * D);
  if (pda_oracle_decode_rows(B, Hq, Hkv, D, BS, nblocks, mbps, q, k, v, bt, lens, scale, nq, trip, 5, orow, 3) != 0)
    ++fails;
  for (int r = 0; r < 5; ++r) {
    const size_t row = ((size_t)trip[3 * r] * nq + trip[3 * r + 1]) * Hq + trip[3 * r + 2];
    expect_same(orow + (size_t)r * D, o1 + row * D, (size_t)D, "rows");
  }
  if (nq == 1) {
    double *w = malloc(sizeof(double) * (size_t)(max_len > 0 ? max_len : 1));
    for (int b = 0; b < B; ++b)
      if (pda_oracle_weights(B, Hq, Hkv, D, BS, nblocks, mbps, q, k, v, bt, lens, scale, b, Hq - 1, w) < 0) ++fails;
    free(w);
  }
  /* append nq new tokens per sequence into copies of the pools */
  uint16_t *kn = malloc(sizeof(uint16_t) * (size_t)B * nq * Hkv * D);
  uint16_t *vn = malloc(sizeof(uint16_t) * (size_t)B * nq * Hkv * D);
  for (size_t i = 0; i < (size_t)B * nq * Hkv * D; ++i) {
    kn[i] = small_bf16();
    vn[i] = small_bf16();
  }
  if (pda_oracle_append(B, Hkv, D, BS, nblocks, mbps, nq, kn, vn, bt, lens, k, v) != 0) ++fails;
  free(kn);
  free(vn);
  free(orow);
  free(o1);
  free(o8);
  free(q);
  free(k);
  free(v);
  free(bt);
  free(lens);
  free(perm);
}

static void logprob_case(int B, int V) {
  uint16_t *xb = malloc(sizeof(uint16_t) * (size_t)B * V);
  float *xf = malloc(sizeof(float) * (size_t)B * V);
  int32_t *tok = malloc(sizeof(int32_t) * (size_t)B);
  double *lp = malloc(sizeof(double) * (size_t)B), *ent = malloc(sizeof(double) * (size_t)B);
  for (size_t i = 0; i < (size_t)B * V; ++i) {
    xb[i] = small_bf16();
    xf[i] = (float)((int32_t)next_u32() % 1000) / 100.f;
  }
  xb[0] = 0xff80; /* -inf */
  for (int b = 0; b < B; ++b) tok[b] = (int32_t)(next_u32() % (uint32_t)V);
  if (pda_oracle_logprob(B, V, V, xb, 0, tok, 1.0, lp, ent) != 0) ++fails;
  if (pda_oracle_logprob(B, V, V, xf, 1, tok, 0.5, lp, NULL) != 0) ++fails;
  free(xb);
  free(xf);
  free(tok);
  free(lp);
  free(ent);
}

int main(void) {
  const int32_t lens_a[] = {1, 15, 16, 17, 0, 300, -3, 64};
  attention_case(8, 8, 2, 64, 1, lens_a);
  attention_case(8, 32, 8, 128, 1, lens_a);
  const int32_t lens_b[] = {7, 40, 129, 5};
  attention_case(4, 12, 4, 64, 6, lens_b);
  attention_case(4, 8, 1, 128, 3, lens_b);
  logprob_case(3, 1000);
  if (fails) {
    fprintf(stderr, "%d check(s) failed\n", fails);
    return 1;
  }
  printf("oracle sanitizer driver: all checks passed\n");
  return 0;
}
