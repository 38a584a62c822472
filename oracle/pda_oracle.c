/*
 * pda_oracle.c -- reference (oracle) for paged decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, obviously correct
 * CPU definition that the GPU library is checked against.  Only the test
 * suite, the package smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no source, header, table or helper with the HIP
 * library, and the HIP library never calls it.
 *
 * What it computes (the paper's rollout hot path):
 *   The paper puts the rollout (generation) phase at over 90% of RLHF/RLVR
 *   runtime (Section 1) and runs it on vLLM, whose central technique is
 *   PagedAttention: the key/value memory of every sequence lives in
 *   fixed-size blocks reached through a per-sequence block table
 *   (Section 3.2, "Accelerated CoT Inference with vLLM"; Appendix C,
 *   stage 1 "Rollout Generation", which names KV-cache management and
 *   PagedAttention).  In every autoregressive step each sequence contributes
 *   one new query token, which attends over its whole cached context.
 *   Paging changes where K/V rows live, never the value computed, so the
 *   oracle is the plain definition of single-query scaled dot-product
 *   attention, written out in fp64:
 *
 *     for every sequence b and query head h:
 *       g   = floor(h / G),  G = Hq / Hkv           (grouped-query heads)
 *       L   = context_lens[b]; if L <= 0 the output row is all zeros
 *       for t in [0, L):
 *         p   = block_table[b][floor(t / BS)],  o = t mod BS
 *         k_t = K[p][g][:][o],  v_t = V[p][g][o][:]  (bf16 widened exactly)
 *         s_t = scale * sum_d q[b][h][d] * k_t[d]
 *       m   = max_t s_t
 *       e_t = exp(s_t - m),  Z = sum_t e_t           (two passes, t ascending)
 *       out[b][h][d] = sum_t (e_t / Z) * v_t[d]
 *
 *   Layouts (all row-major, element counts):
 *     q            bf16  [B][Hq][D]
 *     k_cache      bf16  [num_blocks][Hkv][D/8][BS][8]   key d of slot o sits at
 *                        [p][g][d/8][o][d%8]: each block's keys are stored as
 *                        D/8 chunks of BS rows of 8 consecutive elements
 *     v_cache      bf16  [num_blocks][Hkv][BS][D]
 *     block_table  int32 [B][max_blocks_per_seq]
 *     context_lens int32 [B]
 *     out          fp64  [B][Hq][D]
 *   bf16 values are passed as their raw 16-bit patterns.
 *
 * Every entry point returns 0 on success and a negative value when an
 * argument is out of range (including a block id outside [0, num_blocks) or a
 * context length beyond the block table); on error nothing is written.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int B, Hq, Hkv, D, BS, num_blocks, max_blocks_per_seq;
  const uint16_t *q, *k, *v;
  const int32_t *block_table, *context_lens;
  double scale;
} problem_t;

/* bf16 is the upper half of an IEEE binary32: widening is a 16-bit shift. */
static double bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

static int check_problem(const problem_t *P) {
  if (P->B < 0 || P->Hq <= 0 || P->Hkv <= 0 || P->D <= 0 || P->BS <= 0 ||
      P->num_blocks <= 0 || P->max_blocks_per_seq <= 0)
    return -1;
  if (P->Hq % P->Hkv != 0 || P->D % 8 != 0) return -2;
  if (P->B > 0 && (!P->q || !P->k || !P->v || !P->block_table || !P->context_lens))
    return -3;
  for (int b = 0; b < P->B; ++b) {
    int L = P->context_lens[b];
    if (L <= 0) continue;
    int nblk = (L + P->BS - 1) / P->BS;
    if (nblk > P->max_blocks_per_seq) return -4;
    for (int j = 0; j < nblk; ++j) {
      int32_t p = P->block_table[(size_t)b * P->max_blocks_per_seq + j];
      if (p < 0 || p >= P->num_blocks) return -5;
    }
  }
  return 0;
}

/* Element d of key slot o, block p, KV head g: [p][g][d/8][o][d%8]. */
static size_t k_elem(const problem_t *P, int32_t p, int g, int o, int d) {
  return ((((size_t)p * P->Hkv + g) * (P->D / 8) + d / 8) * P->BS + o) * 8 + d % 8;
}

/* Start of value slot o of block p, KV head g: [p][g][o][0]. */
static size_t v_row(const problem_t *P, int32_t p, int g, int o) {
  return (((size_t)p * P->Hkv + g) * P->BS + o) * P->D;
}

/* The softmax weights w_t = e_t / Z of (b, h), t in [0, L); returns L.
 * `scores` must hold max(L, 1) doubles. */
static int row_weights(const problem_t *P, int b, int h, double *scores) {
  int L = P->context_lens[b];
  if (L <= 0) return 0;
  int G = P->Hq / P->Hkv;
  int g = h / G;
  const uint16_t *qrow = P->q + ((size_t)b * P->Hq + h) * P->D;
  const int32_t *bt = P->block_table + (size_t)b * P->max_blocks_per_seq;
  /* pass 1: scores and their maximum */
  double m = -INFINITY;
  for (int t = 0; t < L; ++t) {
    const int32_t p = bt[t / P->BS];
    const int o = t % P->BS;
    double dot = 0.0;
    for (int d = 0; d < P->D; ++d)
      dot += bf16_to_double(qrow[d]) * bf16_to_double(P->k[k_elem(P, p, g, o, d)]);
    scores[t] = P->scale * dot;
    if (scores[t] > m) m = scores[t];
  }
  /* pass 2: exponentials and their sum, t ascending */
  double Z = 0.0;
  for (int t = 0; t < L; ++t) {
    scores[t] = exp(scores[t] - m);
    Z += scores[t];
  }
  for (int t = 0; t < L; ++t) scores[t] /= Z;
  return L;
}

static void row_output(const problem_t *P, int b, int h, double *w, double *out_row) {
  for (int d = 0; d < P->D; ++d) out_row[d] = 0.0;
  int L = row_weights(P, b, h, w);
  if (L == 0) return;
  int G = P->Hq / P->Hkv;
  int g = h / G;
  const int32_t *bt = P->block_table + (size_t)b * P->max_blocks_per_seq;
  for (int t = 0; t < L; ++t) {
    const uint16_t *vrow = P->v + v_row(P, bt[t / P->BS], g, t % P->BS);
    for (int d = 0; d < P->D; ++d) out_row[d] += w[t] * bf16_to_double(vrow[d]);
  }
}

/* ---- work split over host threads: rows r = tid, tid + T, tid + 2T, ... ---- */
typedef struct {
  const problem_t *P;
  const int32_t *rows; /* (b, h) pairs, or NULL for all rows in order */
  int n_rows, tid, nthreads, max_len;
  double *out;
  int failed;
} job_t;

static void *worker(void *arg) {
  job_t *J = (job_t *)arg;
  double *w = (double *)malloc(sizeof(double) * (size_t)(J->max_len > 0 ? J->max_len : 1));
  if (!w) { J->failed = 1; return NULL; }
  for (int r = J->tid; r < J->n_rows; r += J->nthreads) {
    int b, h;
    if (J->rows) { b = J->rows[2 * r]; h = J->rows[2 * r + 1]; }
    else { b = r / J->P->Hq; h = r % J->P->Hq; }
    row_output(J->P, b, h, w, J->out + (size_t)r * J->P->D);
  }
  free(w);
  return NULL;
}

static int run_rows(const problem_t *P, const int32_t *rows, int n_rows, double *out, int nthreads) {
  int rc = check_problem(P);
  if (rc) return rc;
  if (rows)
    for (int r = 0; r < n_rows; ++r)
      if (rows[2 * r] < 0 || rows[2 * r] >= P->B || rows[2 * r + 1] < 0 || rows[2 * r + 1] >= P->Hq)
        return -6;
  if (n_rows <= 0) return 0;
  int max_len = 1;
  for (int b = 0; b < P->B; ++b)
    if (P->context_lens[b] > max_len) max_len = P->context_lens[b];
  if (nthreads < 1) nthreads = 1;
  if (nthreads > n_rows) nthreads = n_rows;
  job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
  pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return -7; }
  int failed = 0;
  for (int i = 0; i < nthreads; ++i) {
    jobs[i] = (job_t){P, rows, n_rows, i, nthreads, max_len, out, 0};
    if (i > 0 && pthread_create(&th[i], NULL, worker, &jobs[i]) != 0) { failed = 1; nthreads = i; break; }
  }
  if (!failed) worker(&jobs[0]);
  for (int i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
  for (int i = 0; i < nthreads; ++i) failed |= jobs[i].failed;
  free(jobs);
  free(th);
  return failed ? -7 : 0;
}

#define PROBLEM_ARGS                                                                 \
  int B, int Hq, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq, \
      const uint16_t *q, const uint16_t *k_cache, const uint16_t *v_cache,           \
      const int32_t *block_table, const int32_t *context_lens, double scale
#define PROBLEM_INIT                                                                  \
  problem_t P = {B, Hq, Hkv, D, block_size, num_blocks, max_blocks_per_seq, q, k_cache, \
                 v_cache, block_table, context_lens, scale}

/* All B*Hq rows; out is fp64 [B][Hq][D]. */
int pda_oracle_decode(PROBLEM_ARGS, double *out, int num_threads) {
  PROBLEM_INIT;
  return run_rows(&P, NULL, B * Hq, out, num_threads);
}

/* Only the listed (b, h) pairs (rows[2r], rows[2r+1]); out is fp64 [n_rows][D]. */
int pda_oracle_decode_rows(PROBLEM_ARGS, const int32_t *rows, int n_rows, double *out,
                           int num_threads) {
  PROBLEM_INIT;
  if (n_rows > 0 && !rows) return -3;
  return run_rows(&P, rows, n_rows, out, num_threads);
}

/* The L softmax weights of (b, h) into w[0..L); returns L (>= 0) or an error. */
int pda_oracle_weights(PROBLEM_ARGS, int b, int h, double *w) {
  PROBLEM_INIT;
  int rc = check_problem(&P);
  if (rc) return rc;
  if (b < 0 || b >= B || h < 0 || h >= Hq) return -6;
  return row_weights(&P, b, h, w);
}
