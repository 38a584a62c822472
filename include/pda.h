/*
 * pda.h -- paged decode attention for AMD MI355X (gfx950).
 *
 * The operation.  The paper (OpenRLHF) puts the rollout generation phase at
 * over 90% of RLHF/RLVR runtime (Section 1) and runs it on vLLM, whose key
 * technique is PagedAttention: every sequence's attention key and value
 * memory lives in fixed-size blocks of a shared pool, reached through a
 * per-sequence block table, with blocks shareable between sequences for
 * parallel sampling (Section 3.2, "Accelerated CoT Inference with vLLM";
 * Appendix C, stage 1 "Rollout Generation", KV-cache management and
 * PagedAttention).  Each autoregressive step gives every sequence one new
 * query token that attends over its cached context.  This library computes
 * that step for a whole batch, with grouped-query heads:
 *
 *   for sequence b, query head h:   g = floor(h / G),  G = Hq / Hkv
 *     L = context_lens[b]  (clamped to [0, max_context_len]); L == 0 gives 0
 *     token t in [0, L) lives in block p = block_table[b][t / 16], slot o = t % 16
 *     s_t = scale * sum_d q[b][h][d] * K[p][g][d / 8][o][d % 8]
 *     out[b][h] = sum_t softmax(s)_t * V[p][g][o][:]
 *
 * Several new tokens per sequence.  vLLM's speculative decoding and chunked
 * prefill (Section 3.2) bring n > 1 new tokens of a sequence in one step.
 * With num_query_tokens = n, q and out hold n rows per sequence; new token i
 * (0 <= i < n) sits at position L - n + i of the context (L counts the new
 * tokens) and attends causally, to tokens t < L - n + 1 + i.  n = 1 is the
 * decode step above.
 *
 * Layouts (row-major; all pointers below are DEVICE pointers):
 *   q            bf16  [num_seqs][n][num_q_heads][head_dim]
 *   k_cache      bf16  [num_blocks][num_kv_heads][head_dim/8][block_size][8]
 *                       each block's keys as head_dim/8 chunks of 16 slots x 8
 *                       consecutive elements (key element d of slot o at
 *                       [d/8][o][d%8]); a 16-byte load of lane l at offset 16*l
 *                       is then exactly the MFMA operand fragment it needs
 *   v_cache      bf16  [num_blocks][num_kv_heads][block_size][head_dim]
 *   block_table  int32 [num_seqs][max_blocks_per_seq]  (entries past
 *                       ceil(L/16) are never read and may hold anything)
 *   context_lens int32 [num_seqs]
 *   out          fp32  [num_seqs][n][num_q_heads][head_dim]
 *   k_new, v_new bf16  [num_seqs][n][num_kv_heads][head_dim]  (pda_append_kv)
 *   workspace    opaque, pda_workspace_bytes() bytes
 * Pool slots past a sequence's context (the tail of its last block) and pool
 * blocks no sequence references are never used, whatever they hold.  K and V
 * inside a context are expected to be finite: a NaN or infinite element makes
 * the outputs of the rows that see its token non-finite (and, in a chunk of
 * several new tokens, possibly rows of that chunk that do not).
 *
 * Long contexts are split into partitions of `partition_tokens` tokens that
 * are processed independently; a second pass merges the partial softmax
 * states.  Pass 1 runs one workgroup per (partition, sequence, KV head,
 * group of up to 4 chunks of at most 16 / G new tokens each; up to 8 when
 * there are more than 4 chunks, up to 16 when there are more than 8), largest
 * partition first (a small kernel sorts the items by size on the GPU; it is
 * skipped when every item runs at once).  The partition size depends
 * only on the problem descriptor and the arithmetic of an item only on its
 * data, never on physical block ids, timing or the order the items run in,
 * so for a given descriptor the output is bit-for-bit reproducible and
 * independent of where blocks sit in the pool.
 *
 * Ownership and errors.  The caller owns every buffer; the per-step entry
 * points allocate nothing and keep no state, so concurrent calls (with
 * separate workspaces) are safe.  Only pda_step_graph_create allocates: the
 * HIP graph objects it returns, freed by pda_step_graph_destroy.
 * Every entry point validates its scalar arguments and pointers on the host
 * and returns a pda_status without touching the GPU when they are invalid.
 * Work is enqueued asynchronously on `stream` (NULL = the null stream); a
 * failed launch returns PDA_ERR_HIP.  Device-resident contents are the
 * caller's contract (block ids in [0, num_blocks), lengths at most
 * max_context_len); the kernels clamp lengths to [0, max_context_len] and
 * never read or write outside the pool: a (b, kv head) whose block table
 * holds an out-of-range id gets NaN output rows, and the append skips that
 * token.  pda_validate_host() checks host copies of the contents.
 */
#ifndef PDA_H
#define PDA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum pda_status {
  PDA_OK = 0,
  PDA_ERR_NULL = 1,        /* a required pointer is NULL */
  PDA_ERR_SHAPE = 2,       /* a size is negative, zero where it must not be, too large, or inconsistent */
  PDA_ERR_UNSUPPORTED = 3, /* valid but not built: head_dim not 64/128, block_size not 16, G > 16;
                              shared-prefix groups with n G > 64; pda_decode_append with n > 1 */
  PDA_ERR_WORKSPACE = 4,   /* workspace NULL or smaller than pda_workspace_bytes() */
  PDA_ERR_ALIGNMENT = 5,   /* q, k_cache, v_cache, k_new, v_new, out or workspace not 16-byte aligned */
  PDA_ERR_VALUE = 6,       /* non-finite scale, or a host-side content check failed */
  PDA_ERR_HIP = 7,         /* a HIP call failed (launch, graph capture or instantiation) */
  PDA_ERR_SCRATCH = 8      /* pda_decode_noalloc: the step needs more than PDA_NOALLOC_SCRATCH_BYTES */
};

/* Sizes of one step.  All fields are plain host integers. */
typedef struct pda_problem {
  int32_t num_seqs;           /* B >= 0 */
  int32_t num_q_heads;        /* Hq >= 1 */
  int32_t num_kv_heads;       /* Hkv >= 1, divides Hq; G = Hq / Hkv must be <= 16 */
  int32_t head_dim;           /* D: 64 or 128 */
  int32_t block_size;         /* tokens per KV block: must be 16 */
  int32_t num_blocks;         /* rows of k_cache / v_cache, >= 1 */
  int32_t max_blocks_per_seq; /* row stride of block_table, >= 1 */
  int32_t max_context_len;    /* host-known bound on context_lens[]; 0 <= it <= 16*max_blocks_per_seq
                                 and <= 2^28 */
  int32_t partition_tokens;   /* split-K partition size: 0 lets the library choose, otherwise a
                                 positive multiple of 16 (a size beyond max_context_len acts as
                                 max_context_len rounded up to a multiple of 16: one partition) */
  int32_t num_query_tokens;   /* n, new tokens per sequence: 0 or 1 = a decode step */
} pda_problem;

/* What pda_decode will do for a descriptor. */
typedef struct pda_plan_info {
  int32_t partition_tokens;   /* tokens per partition */
  int32_t num_partitions;     /* partitions of the longest context */
  size_t workspace_bytes;     /* workspace the step needs: the work order (4 bytes per item) and,
                                 when a context spans several partitions, the partial states;
                                 0 only for an empty batch */
} pda_plan_info;

/* Plan `prob`.  Returns PDA_OK or the validation error of the descriptor. */
int pda_plan(const pda_problem *prob, pda_plan_info *plan);

/* Workspace bytes pda_decode needs for `prob` (0 only for an empty batch). */
int pda_workspace_bytes(const pda_problem *prob, size_t *bytes);

/* One attention step for the whole batch: pda_partition_attention followed
 * by pda_merge_partitions on the same stream.  `scale` is the softmax scale
 * (usually 1/sqrt(head_dim)); it must be finite.  `workspace` (any contents)
 * must hold pda_workspace_bytes() bytes; it may be NULL for an empty batch.
 * Calls that overlap on the GPU need separate workspaces. */
int pda_decode(const pda_problem *prob, const void *q, const void *k_cache, const void *v_cache,
               const int32_t *block_table, const int32_t *context_lens, float scale, float *out,
               void *workspace, size_t workspace_bytes, hipStream_t stream);

/* pda_decode for callers that cannot allocate: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation.  There is no
 * workspace argument: the step's workspace (work order and partial softmax
 * states) lives in a static device array of PDA_NOALLOC_SCRATCH_BYTES that
 * the library holds on each GPU it runs on until the process ends; its
 * address is looked up once per device, on the first call made with that
 * device current.  The call allocates nothing.  Arguments, layouts, results
 * (bitwise those of pda_decode) and errors are pda_decode's, plus
 * PDA_ERR_SCRATCH, returned without touching the GPU, when
 * pda_workspace_bytes() of the descriptor exceeds PDA_NOALLOC_SCRATCH_BYTES
 * (decode steps of the named Llama-3 shapes need at most a few MB; many new
 * tokens per sequence with split contexts can need more).  Nothing in the
 * scratch needs clearing: each call writes every entry it reads.  All calls
 * on one GPU share its scratch, so calls that overlap on the GPU (on
 * different streams, or from several host threads) race: the caller orders
 * them, e.g. on one stream. */
#define PDA_NOALLOC_SCRATCH_BYTES (64u << 20)
int pda_decode_noalloc(const pda_problem *prob, const void *q, const void *k_cache, const void *v_cache,
                       const int32_t *block_table, const int32_t *context_lens, float scale, float *out,
                       hipStream_t stream);

/* Pass 1 alone (the work-order kernel when needed, then one workgroup per
 * work item):
 * rows that see a single partition, and rows that see no token, are final
 * in `out` after this pass; the others are left as partial softmax states in
 * `workspace`. */
int pda_partition_attention(const pda_problem *prob, const void *q, const void *k_cache,
                            const void *v_cache, const int32_t *block_table,
                            const int32_t *context_lens, float scale, float *out,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Pass 2 alone: merge the partial states that pass 1 left in `workspace` into
 * `out` for every row that sees more than one partition, in ascending
 * partition order.  Must follow pass 1 for the same descriptor and lengths. */
int pda_merge_partitions(const pda_problem *prob, const int32_t *context_lens, float *out,
                         const void *workspace, size_t workspace_bytes, hipStream_t stream);

/* The work order of one step's pass 1 (largest item first, placed for the
 * XCDs), written into `workspace`: every layer of a model's decode step
 * attends over the same lengths and block tables, so the order can be
 * computed once per step and reused by each layer's
 * pda_decode_reusing_order.  pda_decode leaves the same order in its
 * workspace.  Nothing is launched when the step needs no order (all its
 * items run at once).  Only the lengths are read; the order is a
 * permutation of the step's work items whatever they were, so a stale one
 * (lengths changed since) costs schedule quality, never correctness.
 * `context_lens` is device int32 [num_seqs]; `workspace` (16 B aligned, at
 * least pda_workspace_bytes) is caller-owned.  Errors as pda_decode's:
 * PDA_ERR_NULL for a NULL length array, _WORKSPACE, _ALIGNMENT, and the
 * descriptor checks; an empty batch returns PDA_OK and reads nothing. */
int pda_work_order(const pda_problem *prob, const int32_t *context_lens, void *workspace,
                   size_t workspace_bytes, hipStream_t stream);

/* pda_decode without the work-order kernel: pass 1 takes its items in the
 * order already in `workspace`, which a pda_work_order or pda_decode call for
 * the same descriptor (and workspace) must have written; the partial states
 * of the workspace are rewritten as in pda_decode.  With any other contents
 * the kernels stay memory-safe (item indices are bounds-checked) but the
 * output is undefined. */
int pda_decode_reusing_order(const pda_problem *prob, const void *q, const void *k_cache,
                             const void *v_cache, const int32_t *block_table,
                             const int32_t *context_lens, float scale, float *out,
                             void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Pass 1 alone with the order already in `workspace` (pda_partition_attention
 * without its work-order kernel; the order's contract is that of
 * pda_decode_reusing_order): a caller that keeps the partial states before
 * merging them -- e.g. to combine them with states computed elsewhere -- or
 * that times the attention kernel by itself.  pda_merge_partitions completes
 * the step. */
int pda_partition_attention_reusing_order(const pda_problem *prob, const void *q, const void *k_cache,
                                          const void *v_cache, const int32_t *block_table,
                                          const int32_t *context_lens, float scale, float *out,
                                          void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Shared-prefix groups for parallel sampling (Section 3.2: PagedAttention
 * lets the samples of one prompt share the prompt's KV blocks).  The members
 * of group i are the sequences [group_start[i], group_start[i+1]) -- a
 * prompt's samples sit next to each other in the batch -- and their first
 * group_prefix_len[i] tokens (a multiple of 16, at most every member's
 * context length) live in the same physical blocks, i.e. entries
 * 0 .. group_prefix_len[i]/16 - 1 of their block-table rows are equal.
 * Sequences in no group attend as in pda_decode.  The host bounds size the
 * launch; the two arrays are device data (their contents are clamped to the
 * bounds, never trusted for memory safety). */
typedef struct pda_prefix_groups {
  int32_t num_groups;               /* >= 0 */
  int32_t max_group_size;           /* bound on members per group, >= 1 (members past it attend as sequences
                                       in no group: the whole context through their own work items) */
  int32_t max_prefix_len;           /* bound on group_prefix_len[]: a multiple of 16, <= max_context_len */
  const int32_t *group_start;       /* device int32 [num_groups + 1], non-decreasing, within [0, num_seqs] */
  const int32_t *group_prefix_len;  /* device int32 [num_groups] */
} pda_prefix_groups;

/* Plan of pda_decode_shared_prefix (the workspace is larger than pda_decode's);
 * only the host bounds of `groups` are read. */
int pda_plan_shared_prefix(const pda_problem *prob, const pda_prefix_groups *groups, pda_plan_info *plan);

/* The step of pda_decode (one new token per sequence, or n = num_query_tokens
 * with q and out [B][n][Hq][D]) with each group's shared prefix attended once
 * per row group of its members: the members are taken 64 / (n G) at a time
 * (16 at n = 1, G = 4), and a work item reads the prefix blocks and computes
 * all members x n x G query rows of a KV head (at most 64) of one row group on
 * 16-row MFMA tiles, each row seeing the prefix tokens before its own
 * position; every member row then merges the prefix's partial softmax state
 * with those of its own tokens.  One member's rows must fit an item: n G <= 64,
 * else PDA_ERR_UNSUPPORTED.  The result is the same attention as pda_decode
 * (up to rounding).  `workspace` must hold pda_plan_shared_prefix()'s
 * workspace_bytes. */
int pda_decode_shared_prefix(const pda_problem *prob, const pda_prefix_groups *groups, const void *q,
                             const void *k_cache, const void *v_cache, const int32_t *block_table,
                             const int32_t *context_lens, float scale, float *out, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* KV-cache append, the step before attention (Appendix C: the rollout stage's
 * KV-cache management): store the keys and values of the n new tokens of
 * every sequence in the cache.  New token i of sequence b goes to position
 * t = L - n + i (L = context_lens[b], clamped to [0, max_context_len], already
 * counting the new tokens): block block_table[b][t / 16], slot t % 16, in the
 * k_cache / v_cache layouts above.  Positions t < 0 are skipped, and so is a
 * token whose block id is outside [0, num_blocks).  Nothing else in the
 * cache changes.  k_new and v_new are 16-byte aligned device buffers of
 * [B][n][Hkv][D] bf16; k_cache and v_cache are written in place. */
int pda_append_kv(const pda_problem *prob, const void *k_new, const void *v_new,
                  const int32_t *block_table, const int32_t *context_lens, void *k_cache,
                  void *v_cache, hipStream_t stream);

/* pda_append_kv followed by pda_decode, for one new token per sequence
 * (num_query_tokens 0 or 1; the KV-cache management and attention of one
 * rollout step, Section 3.2 and Appendix C).  When every pass-1 work item of
 * the step runs at once (a small batch, where each launch is a large part of
 * the step), the append is folded into pass 1: the wavefront that reads
 * position L - 1 of a (sequence, KV head) first stores the new token's K and
 * V rows there, and the step needs no append launch.  Larger steps run the
 * append kernel first.  Arguments are those of pda_append_kv and pda_decode;
 * the caches and the output (bitwise those of the two calls) are written in
 * place.  PDA_ERR_UNSUPPORTED for num_query_tokens > 1. */
int pda_decode_append(const pda_problem *prob, const void *q, const void *k_new, const void *v_new,
                      void *k_cache, void *v_cache, const int32_t *block_table, const int32_t *context_lens,
                      float scale, float *out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* A whole step captured once as a HIP graph: pda_append_kv, then pda_decode,
 * with the pointers given here (vLLM runs its decode steps as captured
 * graphs, Section 3.2).  Each pda_step_graph_launch replays the step on
 * `stream` and reads the buffers' CURRENT contents (new tokens, queries,
 * block table, lengths), so a caller refills them and relaunches; the
 * descriptor, in particular max_context_len, is fixed at creation.  The
 * arguments are validated as for pda_append_kv and pda_decode.  Launches of
 * one graph must not overlap on the GPU (they share the workspace).
 * pda_step_graph_create allocates the graph objects; pda_step_graph_destroy
 * frees them (NULL is accepted). */
typedef struct pda_step_graph pda_step_graph;
int pda_step_graph_create(const pda_problem *prob, const void *q, const void *k_new,
                          const void *v_new, void *k_cache, void *v_cache,
                          const int32_t *block_table, const int32_t *context_lens, float scale,
                          float *out, void *workspace, size_t workspace_bytes,
                          pda_step_graph **graph);
int pda_step_graph_launch(pda_step_graph *graph, hipStream_t stream);

/* A whole decode step of a model as one HIP graph: for each of num_layers
 * layers, the append of its new tokens' K/V into its own cache and its
 * attention step, with the work order (the lengths and block tables are the
 * same in every layer) computed once, in the first layer.  This is the
 * per-token loop a rollout engine replays (vLLM runs its decode steps as
 * captured graphs, Section 3.2): one graph launch stands for num_layers x 1-4
 * kernel launches (with one new token per sequence and a small batch, each
 * layer's append is folded into its pass 1, as in pda_decode_append).  Every layer has its own q, k_new, v_new, caches and out
 * (the layouts of pda_append_kv / pda_decode); the descriptor, block table,
 * lengths, scale and workspace are shared.  Launch and destroy the result
 * with pda_step_graph_launch / pda_step_graph_destroy; launches of one graph
 * must not overlap on the GPU.  Every layer is validated as pda_append_kv and
 * pda_decode validate their arguments before anything is captured;
 * num_layers < 1 is PDA_ERR_SHAPE.  pda_step_graph_create is this with one
 * layer. */
typedef struct pda_layer_buffers {
  const void *q;      /* bf16 [B][n][Hq][D] */
  const void *k_new;  /* bf16 [B][n][Hkv][D] */
  const void *v_new;  /* bf16 [B][n][Hkv][D] */
  void *k_cache;      /* bf16 [num_blocks][Hkv][D/8][16][8] */
  void *v_cache;      /* bf16 [num_blocks][Hkv][16][D] */
  float *out;         /* fp32 [B][n][Hq][D] */
} pda_layer_buffers;
int pda_model_step_graph_create(const pda_problem *prob, int32_t num_layers, const pda_layer_buffers *layers,
                                const int32_t *block_table, const int32_t *context_lens, float scale,
                                void *workspace, size_t workspace_bytes, pda_step_graph **graph);
int pda_step_graph_destroy(pda_step_graph *graph);

/* Token log-probabilities and entropies of one step's LM-head logits: the
 * rollout records the log-probability of every sampled token, and the policy
 * loss uses the entropy of the same distribution (Appendix C).  With
 * x_j = logits[r][j] * inv_temperature over j in [0, vocab):
 *   logprobs[r]  = x_{tokens[r]} - log sum_j exp(x_j)
 *   entropies[r] = -sum_j p_j log p_j,  p = softmax(x)      (skipped if NULL:
 *   a leaner kernel then runs, with bitwise the same log-probabilities)
 * in natural-log units.  logits: device rows of `vocab` values (bf16 for
 * PDA_DTYPE_BF16, fp32 for PDA_DTYPE_F32), row r starting at element
 * r * row_stride (row_stride >= vocab); the buffer holds num_rows * row_stride
 * elements and every row must be 16-byte aligned.  -inf logits have probability 0; a token id outside
 * [0, vocab) gives a NaN log-probability.  inv_temperature must be finite
 * and >= 0 (0: the uniform distribution).
 *
 * `workspace` may be NULL: one workgroup then streams each row.  Given a
 * workspace of at least pda_logprob_workspace_bytes() bytes (16-byte
 * aligned, any contents; 0 bytes when the batch has at least as many rows as
 * the GPU has compute units), a smaller batch has its rows split over
 * several workgroups whose partial states a second, small kernel merges in a
 * fixed order; results are reproducible for a given (num_rows, vocab, dtype)
 * and agree with the one-workgroup results to fp32 rounding.  Calls that
 * share a workspace must not overlap on the GPU.  PDA_ERR_WORKSPACE: smaller
 * than pda_logprob_workspace_bytes(). */
enum pda_dtype { PDA_DTYPE_BF16 = 0, PDA_DTYPE_F32 = 1 };
int pda_logprob_workspace_bytes(int32_t num_rows, int32_t vocab, int32_t logits_dtype, size_t *bytes);
int pda_token_logprobs(int32_t num_rows, int32_t vocab, int64_t row_stride, int32_t logits_dtype,
                       const void *logits, const int32_t *tokens, float inv_temperature,
                       float *logprobs, float *entropies, void *workspace, size_t workspace_bytes,
                       hipStream_t stream);

/* Host-side check of device contents, on HOST copies: every context length
 * is at most max_context_len and every block id a sequence reads is in
 * [0, num_blocks).  Returns PDA_OK or PDA_ERR_VALUE; on error *first_bad (if
 * not NULL) receives the flat index of the first offending entry, in
 * context_lens for a length and in block_table for a block id. */
int pda_validate_host(const pda_problem *prob, const int32_t *block_table,
                      const int32_t *context_lens, int64_t *first_bad);

/* A static, human-readable name for a pda_status value. */
const char *pda_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* PDA_H */
