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
 * Several new query tokens per sequence (pda_oracle_decode_multi).  When a
 * sequence brings n new tokens at once -- the draft tokens of speculative
 * decoding, or a chunk of a prompt in chunked prefill, both of which the
 * paper lists among vLLM's features (Section 3.2) -- their keys and values
 * are already in the cache as the last n of its L positions, and new token i
 * (0 <= i < n, in sequence order) sits at position L - n + i.  It attends to
 * every position up to and including its own (causal attention), i.e. to the
 * first L - n + 1 + i tokens; with n = 1 this is the decode step above.
 *   q, out  [B][n][Hq][D]
 *
 * KV-cache append (pda_oracle_append).  Before attention runs, the step
 * stores the new tokens' keys and values in the cache (the KV-cache
 * management of the rollout stage, Appendix C): new token i of sequence b
 * goes to position t = L - n + i, i.e. block block_table[b][t / BS], slot
 * t mod BS, in the layouts above.  context_lens already counts the new
 * tokens.  Positions t < 0 (L < n) are skipped; nothing else is written.
 *   k_new, v_new  bf16 [B][n][Hkv][D]
 *
 * Token log-probabilities (pda_oracle_logprob).  After the LM head, the
 * rollout records the log-probability of each sampled token (Appendix C),
 * and the policy loss uses the entropy of the same distribution (Appendix C,
 * the entropy bonus).  With x_j = logits[b][j] * inv_temperature over the
 * vocabulary j in [0, V):
 *   lse        = log sum_j exp(x_j)       (computed as m + log sum_j exp(x_j - m))
 *   logprob[b] = x_{tokens[b]} - lse
 *   entropy[b] = lse - sum_j softmax(x)_j * x_j
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
  int nq; /* new query tokens per sequence (1: decode) */
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
      P->num_blocks <= 0 || P->max_blocks_per_seq <= 0 || P->nq <= 0)
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

/* Tokens that new query token i of sequence b attends to: positions
 * [0, L - nq + 1 + i), none when that is empty or L <= 0. */
static int visible_len(const problem_t *P, int b, int i) {
  int L = P->context_lens[b];
  if (L <= 0) return 0;
  int n = L - P->nq + 1 + i;
  return n > 0 ? n : 0;
}

/* The softmax weights w_t = e_t / Z of query row (b, i, h), t in [0, L) with
 * L its visible length; returns L.  `scores` must hold max(L, 1) doubles. */
static int row_weights(const problem_t *P, int b, int i, int h, double *scores) {
  int L = visible_len(P, b, i);
  if (L <= 0) return 0;
  int G = P->Hq / P->Hkv;
  int g = h / G;
  const uint16_t *qrow = P->q + (((size_t)b * P->nq + i) * P->Hq + h) * P->D;
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

static void row_output(const problem_t *P, int b, int i, int h, double *w, double *out_row) {
  for (int d = 0; d < P->D; ++d) out_row[d] = 0.0;
  int L = row_weights(P, b, i, h, w);
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
  const int32_t *rows; /* (b, i, h) triples, or NULL for all rows in order */
  int n_rows, tid, nthreads, max_len;
  double *out;
  int failed;
} job_t;

static void *worker(void *arg) {
  job_t *J = (job_t *)arg;
  double *w = (double *)malloc(sizeof(double) * (size_t)(J->max_len > 0 ? J->max_len : 1));
  if (!w) { J->failed = 1; return NULL; }
  for (int r = J->tid; r < J->n_rows; r += J->nthreads) {
    int b, i, h;
    if (J->rows) { b = J->rows[3 * r]; i = J->rows[3 * r + 1]; h = J->rows[3 * r + 2]; }
    else { b = r / (J->P->nq * J->P->Hq); i = (r / J->P->Hq) % J->P->nq; h = r % J->P->Hq; }
    row_output(J->P, b, i, h, w, J->out + (size_t)r * J->P->D);
  }
  free(w);
  return NULL;
}

static int run_rows(const problem_t *P, const int32_t *rows, int n_rows, double *out, int nthreads) {
  int rc = check_problem(P);
  if (rc) return rc;
  if (rows)
    for (int r = 0; r < n_rows; ++r)
      if (rows[3 * r] < 0 || rows[3 * r] >= P->B || rows[3 * r + 1] < 0 || rows[3 * r + 1] >= P->nq ||
          rows[3 * r + 2] < 0 || rows[3 * r + 2] >= P->Hq)
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
#define PROBLEM_INIT(NQ)                                                              \
  problem_t P = {B, Hq, Hkv, D, block_size, num_blocks, max_blocks_per_seq, q, k_cache, \
                 v_cache, block_table, context_lens, scale, NQ}

/* All B*Hq rows of a decode step; out is fp64 [B][Hq][D]. */
int pda_oracle_decode(PROBLEM_ARGS, double *out, int num_threads) {
  PROBLEM_INIT(1);
  return run_rows(&P, NULL, B * Hq, out, num_threads);
}

/* All B*n*Hq rows with n new query tokens per sequence; q and out are
 * [B][n][Hq][D] (out fp64). */
int pda_oracle_decode_multi(PROBLEM_ARGS, int n, double *out, int num_threads) {
  PROBLEM_INIT(n);
  if (n <= 0) return -1;
  return run_rows(&P, NULL, B * n * Hq, out, num_threads);
}

/* Only the listed (b, i, h) triples (rows[3r..3r+2]) with n new query tokens
 * per sequence (n = 1: a decode step); out is fp64 [n_rows][D]. */
int pda_oracle_decode_rows(PROBLEM_ARGS, int n, const int32_t *rows, int n_rows, double *out,
                           int num_threads) {
  PROBLEM_INIT(n);
  if (n_rows > 0 && !rows) return -3;
  return run_rows(&P, rows, n_rows, out, num_threads);
}

/* The softmax weights of decode row (b, h) into w[0..L); returns L (>= 0) or
 * an error. */
int pda_oracle_weights(PROBLEM_ARGS, int b, int h, double *w) {
  PROBLEM_INIT(1);
  int rc = check_problem(&P);
  if (rc) return rc;
  if (b < 0 || b >= B || h < 0 || h >= Hq) return -6;
  return row_weights(&P, b, 0, h, w);
}

/* ---- KV-cache append ---- */

/* Store the n new tokens of every sequence in the cache (in place).  All
 * target block ids are checked before anything is written. */
int pda_oracle_append(int B, int Hkv, int D, int block_size, int num_blocks, int max_blocks_per_seq,
                      int n, const uint16_t *k_new, const uint16_t *v_new, const int32_t *block_table,
                      const int32_t *context_lens, uint16_t *k_cache, uint16_t *v_cache) {
  problem_t P = {B, Hkv, Hkv, D, block_size, num_blocks, max_blocks_per_seq, NULL, k_cache,
                 v_cache, block_table, context_lens, 0.0, n};
  if (B < 0 || Hkv <= 0 || D <= 0 || D % 8 != 0 || block_size <= 0 || num_blocks <= 0 ||
      max_blocks_per_seq <= 0 || n <= 0)
    return -1;
  if (B > 0 && (!k_new || !v_new || !block_table || !context_lens || !k_cache || !v_cache)) return -3;
  for (int b = 0; b < B; ++b) {
    const int L = context_lens[b];
    for (int i = 0; i < n; ++i) {
      const int t = L - n + i;
      if (t < 0) continue;
      if (t / block_size >= max_blocks_per_seq) return -4;
      const int32_t p = block_table[(size_t)b * max_blocks_per_seq + t / block_size];
      if (p < 0 || p >= num_blocks) return -5;
    }
  }
  for (int b = 0; b < B; ++b) {
    const int L = context_lens[b];
    const int32_t *bt = block_table + (size_t)b * max_blocks_per_seq;
    for (int i = 0; i < n; ++i) {
      const int t = L - n + i;
      if (t < 0) continue;
      const int32_t p = bt[t / block_size];
      const int o = t % block_size;
      for (int g = 0; g < Hkv; ++g) {
        const size_t src = (((size_t)b * n + i) * Hkv + g) * D;
        for (int d = 0; d < D; ++d) {
          k_cache[k_elem(&P, p, g, o, d)] = k_new[src + d];
          v_cache[v_row(&P, p, g, o) + d] = v_new[src + d];
        }
      }
    }
  }
  return 0;
}

/* ---- token log-probabilities and entropy ---- */

/* logits: B rows of V values, row r starting at element r * row_stride; bf16
 * bit patterns when logits_are_f32 == 0, IEEE binary32 otherwise.  Writes
 * logprob[b] and, when `entropy` is not NULL, entropy[b] (both fp64). */
int pda_oracle_logprob(int B, int V, int64_t row_stride, const void *logits, int logits_are_f32,
                       const int32_t *tokens, double inv_temperature, double *logprob, double *entropy) {
  if (B < 0 || V <= 0 || row_stride < V) return -1;
  if (B > 0 && (!logits || !tokens || !logprob)) return -3;
  for (int b = 0; b < B; ++b)
    if (tokens[b] < 0 || tokens[b] >= V) return -6;
  for (int b = 0; b < B; ++b) {
    const size_t base = (size_t)b * (size_t)row_stride;
    double *x = (double *)malloc(sizeof(double) * (size_t)V);
    if (!x) return -7;
    for (int j = 0; j < V; ++j) {
      double raw;
      if (logits_are_f32) {
        float f;
        memcpy(&f, (const char *)logits + (base + j) * 4, 4);
        raw = (double)f;
      } else {
        raw = bf16_to_double(((const uint16_t *)logits)[base + j]);
      }
      x[j] = raw * inv_temperature;
    }
    double m = -INFINITY;
    for (int j = 0; j < V; ++j)
      if (x[j] > m) m = x[j];
    double Z = 0.0;
    for (int j = 0; j < V; ++j) Z += exp(x[j] - m);
    const double lse = m + log(Z);
    logprob[b] = x[tokens[b]] - lse;
    if (entropy) {
      double mean_x = 0.0; /* sum_j softmax_j * x_j */
      for (int j = 0; j < V; ++j) {
        const double e = exp(x[j] - m);
        if (e > 0.0) mean_x += e / Z * x[j]; /* a term of probability 0 adds 0, also at x = -inf */
      }
      entropy[b] = lse - mean_x;
    }
    free(x);
  }
  return 0;
}
