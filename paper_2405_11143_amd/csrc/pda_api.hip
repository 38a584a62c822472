// C ABI of the paged decode-attention library (declared in include/pda.h):
// host-side validation, the plan (partition size, query chunks, workspace),
// the launches, and the captured step graph.  Apart from the graph objects
// that pda_step_graph_create returns, nothing here allocates memory or keeps
// state between calls.
#include <math.h>

#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <new>

#include "pda.h"
#include "pda_internal.h"

namespace {

// Partition size when the caller leaves it to the library.  Pass 1 runs its
// items largest first, a greedy schedule that ends at most one item's
// duration after the ideal one, so an item should be short next to the work
// each of the kConcurrentItems workgroups the GPU runs at once has to do;
// longer items amortise each workgroup's start-up (order, length, block ids,
// q) and its partial state over more streamed tiles.  With only
// max_context_len on the host, the work is estimated as B * Hkv * chunk
// groups * max_context_len / 2 tokens (the mean of contexts spread up to the
// maximum), and the share is that over kConcurrentItems.  Items of 16 or more
// query rows (several new tokens per sequence) take kRowsShareNum /
// kRowsShareDen of it: on MI355X the 70B TP=8 shard with 2, 4 and 8 new
// tokens ran 1%, 8% and 6% faster at 3584 tokens than at the plain share
// (2816), while the one-token step is flat between 2816 and 4096.  A share
// above kMaxPartitionTokens splits the longest context into the fewest equal
// partitions of at most that size (9216 -> 2 x 4608, 16384 -> 4 x 4096).
// Items of kWideItemRows or more query rows (tens of new tokens per
// sequence) skip that cap: each partition beyond the first costs a partial
// state per row written and read back, which for them is as large as the
// partition's K/V bytes (2 MB per 4096 tokens of one KV head against 2 MB of
// states for 2048 rows); on MI355X the chunked-prefill step (32 sequences,
// 512 or 256 new tokens, contexts up to 8192) ran 2% and 4.5% faster in one
// partition than in two of 4096.
// The result is rounded up to kPartitionQuantum tokens, at least
// kMinPartitionTokens and never longer than the longest context (then there
// is one partition and no merge pass).
// Longest context a descriptor may announce: keeps every token sum of the
// kernels (a position plus a partition size) far inside int32.
constexpr int32_t kMaxContextTokens = 1 << 28;
constexpr int kMaxPartitionTokens = 4608;
constexpr int64_t kWideItemRows = 64;
constexpr int64_t kRowsShareNum = 13, kRowsShareDen = 10;
constexpr int kMinPartitionTokens = 256;
constexpr int kPartitionQuantum = 256;
constexpr int64_t kConcurrentItems = 768;  // 256 compute units x 3 workgroups of 4 wavefronts
constexpr int64_t kPrefixItemRows = 64;    // query rows of one prefix item: 4 tiles of 16

int query_tokens(const pda_problem* p) { return p->num_query_tokens > 0 ? p->num_query_tokens : 1; }

int check_problem(const pda_problem* p) {
  if (!p) return PDA_ERR_NULL;
  if (p->num_seqs < 0 || p->num_q_heads < 1 || p->num_kv_heads < 1 || p->num_blocks < 1 ||
      p->max_blocks_per_seq < 1 || p->max_context_len < 0 || p->partition_tokens < 0 || p->num_query_tokens < 0)
    return PDA_ERR_SHAPE;
  if (p->num_q_heads % p->num_kv_heads != 0) return PDA_ERR_SHAPE;
  if (p->partition_tokens % pda::kBlockTokens != 0) return PDA_ERR_SHAPE;
  if ((int64_t)p->max_context_len > (int64_t)pda::kBlockTokens * p->max_blocks_per_seq) return PDA_ERR_SHAPE;
  if (p->max_context_len > kMaxContextTokens) return PDA_ERR_SHAPE;
  // output rows B * n * Hq must fit an int (two factors at a time: three int32 factors can overflow int64)
  const int64_t rows_per_seq = (int64_t)query_tokens(p) * p->num_q_heads;
  if (rows_per_seq > 0x7fffffff || (int64_t)p->num_seqs * rows_per_seq > 0x7fffffff) return PDA_ERR_SHAPE;
  if (p->block_size != pda::kBlockTokens) return PDA_ERR_UNSUPPORTED;
  if (p->head_dim != 64 && p->head_dim != 128) return PDA_ERR_UNSUPPORTED;
  if (p->num_q_heads / p->num_kv_heads > pda::kMaxGroup) return PDA_ERR_UNSUPPORTED;
  return PDA_OK;
}

struct Plan {
  pda_plan_info info;
  int query_chunk;        // new tokens per work item: min(n, 16 / G)
  int num_query_chunks;   // ceil(n / query_chunk)
  int chunks_per_group;   // 4; 8 with more than 4 chunks (two 16-row tiles per wavefront); 16 with more than 8
  int num_chunk_groups;   // ceil(chunks / chunks_per_group): chunks per work item share its tiles
  int prefix_partitions;  // Pp: partitions of the longest shared prefix (0 without groups)
  int members_per_row_group;  // MR: members whose query rows (n G each) fill one prefix item of 64 rows
  int prefix_row_groups;      // RG: prefix items per group, partition and KV head
  size_t regular_items;   // P * B * Hkv * chunk groups (pass-1 workgroups of the sequences' own tokens)
  size_t items;           // regular items + num_groups * Pp * RG * Hkv prefix items
  size_t slots;           // partial states: (Pp + P) per output row; 0 when nothing is split
};

// Workgroups the GPU runs at once in a step's pass-1 variant: 3 per compute
// unit for items of up to 4 query chunks, 2 for the wide variant (243
// VGPRs at D = 128), 1 for its 8-wavefront form.
int64_t concurrent_items(const Plan& plan) {
  if (plan.chunks_per_group > pda::kWideChunks) return kConcurrentItems / 3;
  if (plan.chunks_per_group > pda::kWaves) return kConcurrentItems * 2 / 3;
  return kConcurrentItems;
}

// Shared-prefix groups: host bounds checked here (the plan needs no more);
// the arrays are device data, required by the step itself.
int check_groups(const pda_problem* p, const pda_prefix_groups* g) {
  if (!g) return PDA_ERR_NULL;
  if (g->num_groups < 0 || g->max_group_size < 1 || g->max_prefix_len < 0 ||
      g->max_prefix_len % pda::kBlockTokens != 0 || g->max_prefix_len > p->max_context_len)
    return PDA_ERR_SHAPE;
  // one member's rows (new tokens x G) fit the 4 tiles of a prefix item; a
  // group's members are split into row groups of 64 rows at most
  if ((int64_t)query_tokens(p) * (p->num_q_heads / p->num_kv_heads) > kPrefixItemRows) return PDA_ERR_UNSUPPORTED;
  return PDA_OK;
}

// a * b for non-negative factors, saturated far above any accepted count
int64_t mul_sat(int64_t a, int64_t b) {
  constexpr int64_t kSat = int64_t(1) << 40;
  if (a == 0 || b == 0) return 0;
  return a > kSat / b ? kSat : std::min(kSat, a * b);
}

int make_plan(const pda_problem* p, const pda_prefix_groups* groups, Plan* plan) {
  int rc = check_problem(p);
  if (rc != PDA_OK) return rc;
  if (groups && (rc = check_groups(p, groups)) != PDA_OK) return rc;
  const int n = query_tokens(p);
  const int G = p->num_q_heads / p->num_kv_heads;
  const int qc = std::min(n, pda::kMaxGroup / G);
  const int nqc = (n + qc - 1) / qc;
  const int cpg = nqc > pda::kWideChunks ? pda::kWide16Chunks
                  : nqc > pda::kWaves    ? pda::kWideChunks
                                         : pda::kWaves;  // chunks per work item
  const int ncg = (nqc + cpg - 1) / cpg;
  // the work order counts Hkv items per pair of either kind: with groups a
  // work item holds every query chunk of a sequence (n G <= 64 means at most 7)
  if (groups && ncg != 1) return PDA_ERR_UNSUPPORTED;
  const int64_t units = (int64_t)p->num_seqs * p->num_kv_heads * ncg;
  int tp = p->partition_tokens;
  if (tp == 0) {
    const int64_t len = p->max_context_len > 0 ? p->max_context_len : 1;
    // (a product that would overflow only means: as long as allowed)
    // items of more than 8 chunks (one 8-wavefront workgroup per compute
    // unit) count 512 at once: long enough to amortise their start-up,
    // short enough that ragged contexts still balance
    const int64_t slots = cpg > pda::kWideChunks ? kConcurrentItems * 2 / 3 : kConcurrentItems;
    int64_t share = units > (INT64_MAX / 4) / len ? INT64_MAX / 4 : (units * len / 2 + slots - 1) / slots;
    const int64_t item_rows = (int64_t)std::min(nqc, cpg) * qc * G;
    if (item_rows >= pda::kMaxGroup) share = share * kRowsShareNum / kRowsShareDen;
    const int64_t cap = item_rows >= kWideItemRows ? kMaxContextTokens : kMaxPartitionTokens;
    if (share > cap) {
      const int64_t pieces = (len + cap - 1) / cap;
      share = (len + pieces - 1) / pieces;
    }
    const int64_t quanta = (share + kPartitionQuantum - 1) / kPartitionQuantum;
    tp = (int)std::min<int64_t>(cap, std::max<int64_t>(kMinPartitionTokens, quanta * kPartitionQuantum));
    const int64_t rounded = (len + pda::kBlockTokens - 1) / pda::kBlockTokens * pda::kBlockTokens;
    if (rounded < tp) tp = (int)rounded;  // the whole context fits one partition
  } else {
    // a forced size beyond the longest context means one partition: the same
    // step as with that context's length rounded up to a whole block
    const int64_t whole = std::max<int64_t>(pda::kBlockTokens, ((int64_t)p->max_context_len + pda::kBlockTokens - 1) /
                                                                   pda::kBlockTokens * pda::kBlockTokens);
    if (tp > whole) tp = (int)whole;
  }
  const int64_t parts = p->max_context_len > 0 ? ((int64_t)p->max_context_len + tp - 1) / tp : 1;
  const int num_groups = groups ? groups->num_groups : 0;
  const int64_t pparts = num_groups > 0 ? ((int64_t)groups->max_prefix_len + tp - 1) / tp : 0;
  // members per prefix item, and prefix items per (group, partition, KV head):
  // a group has at most min(max_group_size, B) members
  const int mr = (int)(kPrefixItemRows / ((int64_t)n * G));
  const int64_t group_members = groups ? std::min<int64_t>(groups->max_group_size, std::max(p->num_seqs, 1)) : 0;
  const int64_t rgroups = num_groups > 0 ? (group_members + mr - 1) / mr : 0;
  const int64_t prefix_pairs = mul_sat(mul_sat(num_groups, pparts), rgroups);
  const int64_t prefix_items = mul_sat(prefix_pairs, p->num_kv_heads);
  if (mul_sat(parts, units) + prefix_items > 0x7fffffff || mul_sat(parts, p->num_seqs) + prefix_pairs > 0x7fffffff)
    return PDA_ERR_SHAPE;
  *plan = Plan{};
  plan->info.partition_tokens = tp;
  plan->info.num_partitions = (int32_t)parts;
  plan->query_chunk = qc;
  plan->num_query_chunks = nqc;
  plan->chunks_per_group = cpg;
  plan->num_chunk_groups = ncg;
  plan->prefix_partitions = (int)pparts;
  plan->members_per_row_group = num_groups > 0 ? mr : 0;
  plan->prefix_row_groups = (int)rgroups;
  if (p->num_seqs > 0) {
    plan->regular_items = (size_t)(parts * units);
    plan->items = plan->regular_items + (size_t)prefix_items;
    // with groups every member row is merged from its prefix and own partitions
    const bool split = parts > 1 || groups != nullptr;
    plan->slots = split ? (size_t)p->num_seqs * n * p->num_q_heads * (size_t)(pparts + parts) : 0;
    // partial states (O, m, l), then the work order, then (with groups) the
    // per-sequence prefix lengths
    plan->info.workspace_bytes = plan->slots * (p->head_dim + 2) * sizeof(float) + plan->items * sizeof(int32_t) +
                                 (groups ? (size_t)p->num_seqs * sizeof(int32_t) : 0);
  }
  return PDA_OK;
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

// Sizes and workspace carving shared by every launch.
void fill_args(const pda_problem* p, const Plan* plan, void* ws, pda::StepArgs* args) {
  *args = pda::StepArgs{};
  float* wsf = static_cast<float*>(ws);
  if (plan->info.workspace_bytes > 0 && ws) {
    if (plan->slots > 0) {
      args->part_o = wsf;
      args->part_m = wsf + plan->slots * p->head_dim;
      args->part_l = wsf + plan->slots * (p->head_dim + 1);
    }
    args->order = reinterpret_cast<int32_t*>(wsf + plan->slots * (p->head_dim + 2));
  }
  args->slots_per_row = plan->prefix_partitions + plan->info.num_partitions;
  args->prefix_partitions = plan->prefix_partitions;
  args->members_per_row_group = plan->members_per_row_group;
  args->prefix_row_groups = plan->prefix_row_groups;
  args->num_regular_items = (int32_t)plan->regular_items;
  args->num_prefix_items = (int32_t)(plan->items - plan->regular_items);
  args->num_seqs = p->num_seqs;
  args->num_q_heads = p->num_q_heads;
  args->num_kv_heads = p->num_kv_heads;
  args->group = p->num_q_heads / p->num_kv_heads;
  args->num_blocks = p->num_blocks;
  args->max_blocks_per_seq = p->max_blocks_per_seq;
  args->max_context_len = p->max_context_len;
  args->num_query_tokens = query_tokens(p);
  args->query_chunk = plan->query_chunk;
  args->num_query_chunks = plan->num_query_chunks;
  args->chunks_per_group = plan->chunks_per_group;
  args->num_chunk_groups = plan->num_chunk_groups;
  args->partition_tokens = plan->info.partition_tokens;
  args->num_partitions = plan->info.num_partitions;
}

// Validation shared by the entry points that launch pass 1; fills `args`.
int prepare_step(const pda_problem* p, const pda_prefix_groups* groups, const void* q, const void* k, const void* v,
                 const int32_t* bt, const int32_t* lens, float scale, float* out, void* ws, size_t ws_bytes,
                 Plan* plan, pda::StepArgs* args) {
  int rc = check_problem(p);
  if (rc != PDA_OK) return rc;
  if (p->num_seqs > 0 && (!q || !k || !v || !bt || !lens || !out)) return PDA_ERR_NULL;
  if (!isfinite(scale)) return PDA_ERR_VALUE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16)) return PDA_ERR_ALIGNMENT;
  rc = make_plan(p, groups, plan);
  if (rc != PDA_OK) return rc;
  if (plan->info.workspace_bytes > 0) {
    if (!ws || ws_bytes < plan->info.workspace_bytes) return PDA_ERR_WORKSPACE;
    if (!aligned(ws, 16)) return PDA_ERR_ALIGNMENT;
  }
  if (groups && groups->num_groups > 0 && p->num_seqs > 0 && (!groups->group_start || !groups->group_prefix_len))
    return PDA_ERR_NULL;
  fill_args(p, plan, ws, args);
  // When the GPU runs every item at once the order is irrelevant: the step
  // skips the work-order kernel (one dependent launch less) and item i is
  // workgroup i.  Shared-prefix groups still need it for the prefix table.
  if (plan->items <= (size_t)concurrent_items(*plan) && !(groups && groups->num_groups > 0)) args->order = nullptr;
  if (groups && groups->num_groups > 0 && p->num_seqs > 0) {
    args->group_start = groups->group_start;
    args->group_prefix_len = groups->group_prefix_len;
    args->num_groups = groups->num_groups;
    args->max_group_size = groups->max_group_size;
    args->max_prefix_len = groups->max_prefix_len;
    args->seq_prefix = args->order + plan->items;
  }
  args->q = static_cast<const uint16_t*>(q);
  args->k = static_cast<const uint16_t*>(k);
  args->v = static_cast<const uint16_t*>(v);
  args->table = bt;
  args->lens = lens;
  args->out = out;
  args->scale_log2 = scale * 1.4426950408889634f;
  return PDA_OK;
}

// Validation of an append; fills `args` (no workspace is involved).
int prepare_append(const pda_problem* p, const void* k_new, const void* v_new, const int32_t* bt,
                   const int32_t* lens, void* k_cache, void* v_cache, pda::StepArgs* args) {
  int rc = check_problem(p);
  if (rc != PDA_OK) return rc;
  if (p->num_seqs > 0 && (!k_new || !v_new || !bt || !lens || !k_cache || !v_cache)) return PDA_ERR_NULL;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
    return PDA_ERR_ALIGNMENT;
  Plan plan;
  rc = make_plan(p, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  fill_args(p, &plan, nullptr, args);
  args->table = bt;
  args->lens = lens;
  return PDA_OK;
}

// The launches of one attention step (work order, pass 1, merge).
int launch_attention(const pda_problem* p, const Plan& plan, const pda::StepArgs& args, hipStream_t stream) {
  if (p->num_seqs == 0) return PDA_OK;
  if (args.order && pda::launch_order(args, stream) != hipSuccess) return PDA_ERR_HIP;
  if (pda::launch_partition(args, p->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  if (plan.slots > 0 && pda::launch_merge(args, p->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  return PDA_OK;
}

hipError_t launch_append_of(const pda_problem* p, const pda::StepArgs& args, const void* k_new, const void* v_new,
                            void* k_cache, void* v_cache, hipStream_t stream) {
  return pda::launch_append(args, static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                            static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), p->head_dim, stream);
}

// Whether a step folds its KV append into pass 1: one new token per
// sequence, and every work item runs at once (a small batch, where the
// append's own launch is a large part of the step: the 32-layer step of a
// 4-sequence batch ran 1.6x faster as one graph with the appends folded).
// In larger steps each item's wavefront that stores the new rows waits for
// its stores before it streams, and on MI355X that cost the Llama-3-8B step
// 3%, more than the separate append kernel (3.4 us), so there the append
// keeps its own launch.
bool folds_append(const pda_problem* p, const Plan& plan) {
  return query_tokens(p) == 1 && plan.items <= (size_t)concurrent_items(plan);
}

// Let pass 1 store the step's new K/V rows (one new token per sequence, no
// shared-prefix groups) instead of a separate append launch.
void fold_append(pda::StepArgs* args, const void* k_new, const void* v_new, void* k_cache, void* v_cache) {
  args->k_new = static_cast<const uint16_t*>(k_new);
  args->v_new = static_cast<const uint16_t*>(v_new);
  args->k_store = static_cast<uint16_t*>(k_cache);
  args->v_store = static_cast<uint16_t*>(v_cache);
}

}  // namespace

// The scratch of pda_decode_noalloc: the workspace of a step (work order and
// partial softmax states) for callers that cannot allocate.  Each GPU the
// library runs on holds its own copy of this array from the code object's
// load until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: the device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static __device__ __align__(256) unsigned char scratch[PDA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices];  // device address of `scratch` on each device (null: not yet looked up)

// The current device's scratch address (looked up on its first use), or null
// when the device cannot be named or the lookup fails.
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    scratch_ptr[dev] = ptr;
  }
  return scratch_ptr[dev];
}

}  // namespace

struct pda_step_graph {
  hipGraph_t graph;
  hipGraphExec_t exec;
  bool empty;  // an empty batch: nothing to launch
};

extern "C" {

int pda_plan(const pda_problem* prob, pda_plan_info* info) {
  if (!info) return PDA_ERR_NULL;
  Plan plan;
  int rc = make_plan(prob, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  *info = plan.info;
  return PDA_OK;
}

int pda_workspace_bytes(const pda_problem* prob, size_t* bytes) {
  if (!bytes) return PDA_ERR_NULL;
  Plan plan;
  int rc = make_plan(prob, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  *bytes = plan.info.workspace_bytes;
  return PDA_OK;
}

int pda_partition_attention(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
                            const int32_t* block_table, const int32_t* context_lens, float scale, float* out,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Plan plan;
  pda::StepArgs args;
  int rc = prepare_step(prob, nullptr, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                        workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  if (args.order && pda::launch_order(args, stream) != hipSuccess) return PDA_ERR_HIP;
  if (pda::launch_partition(args, prob->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  return PDA_OK;
}

int pda_work_order(const pda_problem* prob, const int32_t* context_lens, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
  int rc = check_problem(prob);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  if (!context_lens) return PDA_ERR_NULL;
  Plan plan;
  rc = make_plan(prob, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  if (!workspace || workspace_bytes < plan.info.workspace_bytes) return PDA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return PDA_ERR_ALIGNMENT;
  if (plan.items <= (size_t)concurrent_items(plan)) return PDA_OK;  // the step runs without an order
  pda::StepArgs args;
  fill_args(prob, &plan, workspace, &args);
  args.lens = context_lens;
  return pda::launch_order(args, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_decode_reusing_order(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
                             const int32_t* block_table, const int32_t* context_lens, float scale, float* out,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Plan plan;
  pda::StepArgs args;
  int rc = prepare_step(prob, nullptr, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                        workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  if (pda::launch_partition(args, prob->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  if (plan.slots > 0 && pda::launch_merge(args, prob->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  return PDA_OK;
}

int pda_partition_attention_reusing_order(const pda_problem* prob, const void* q, const void* k_cache,
                                          const void* v_cache, const int32_t* block_table,
                                          const int32_t* context_lens, float scale, float* out, void* workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
  Plan plan;
  pda::StepArgs args;
  int rc = prepare_step(prob, nullptr, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                        workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  return pda::launch_partition(args, prob->head_dim, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_merge_partitions(const pda_problem* prob, const int32_t* context_lens, float* out, const void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  int rc = check_problem(prob);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  if (!context_lens || !out) return PDA_ERR_NULL;
  if (!aligned(workspace, 16) || !aligned(out, 16)) return PDA_ERR_ALIGNMENT;
  Plan plan;
  rc = make_plan(prob, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  if (plan.slots == 0) return PDA_OK;  // nothing was split
  if (!workspace || workspace_bytes < plan.info.workspace_bytes) return PDA_ERR_WORKSPACE;
  pda::StepArgs args;
  fill_args(prob, &plan, const_cast<void*>(workspace), &args);
  args.lens = context_lens;
  args.out = out;
  return pda::launch_merge(args, prob->head_dim, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_decode(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
               const int32_t* block_table, const int32_t* context_lens, float scale, float* out, void* workspace,
               size_t workspace_bytes, hipStream_t stream) {
  int rc = pda_partition_attention(prob, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                                   workspace_bytes, stream);
  if (rc != PDA_OK) return rc;
  return pda_merge_partitions(prob, context_lens, out, workspace, workspace_bytes, stream);
}

int pda_decode_noalloc(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
                       const int32_t* block_table, const int32_t* context_lens, float scale, float* out,
                       hipStream_t stream) {
  Plan plan;
  int rc = make_plan(prob, nullptr, &plan);
  if (rc != PDA_OK) return rc;
  if (plan.info.workspace_bytes > (size_t)PDA_NOALLOC_SCRATCH_BYTES) return PDA_ERR_SCRATCH;
  void* ws = nullptr;
  if (prob->num_seqs > 0 && !(ws = device_scratch())) return PDA_ERR_HIP;
  pda::StepArgs args;
  rc = prepare_step(prob, nullptr, q, k_cache, v_cache, block_table, context_lens, scale, out, ws,
                    PDA_NOALLOC_SCRATCH_BYTES, &plan, &args);
  if (rc != PDA_OK) return rc;
  return launch_attention(prob, plan, args, stream);
}

int pda_decode_append(const pda_problem* prob, const void* q, const void* k_new, const void* v_new, void* k_cache,
                      void* v_cache, const int32_t* block_table, const int32_t* context_lens, float scale, float* out,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  pda::StepArgs append_args, args;
  Plan plan;
  int rc = prepare_append(prob, k_new, v_new, block_table, context_lens, k_cache, v_cache, &append_args);
  if (rc != PDA_OK) return rc;
  rc = prepare_step(prob, nullptr, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                    workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  if (query_tokens(prob) != 1) return PDA_ERR_UNSUPPORTED;  // one new token per sequence
  if (prob->num_seqs == 0) return PDA_OK;
  if (folds_append(prob, plan))
    fold_append(&args, k_new, v_new, k_cache, v_cache);
  else if (launch_append_of(prob, append_args, k_new, v_new, k_cache, v_cache, stream) != hipSuccess)
    return PDA_ERR_HIP;
  return launch_attention(prob, plan, args, stream);
}

int pda_append_kv(const pda_problem* prob, const void* k_new, const void* v_new, const int32_t* block_table,
                  const int32_t* context_lens, void* k_cache, void* v_cache, hipStream_t stream) {
  pda::StepArgs args;
  int rc = prepare_append(prob, k_new, v_new, block_table, context_lens, k_cache, v_cache, &args);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  return launch_append_of(prob, args, k_new, v_new, k_cache, v_cache, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_step_graph_create(const pda_problem* prob, const void* q, const void* k_new, const void* v_new,
                          void* k_cache, void* v_cache, const int32_t* block_table, const int32_t* context_lens,
                          float scale, float* out, void* workspace, size_t workspace_bytes,
                          pda_step_graph** graph) {
  pda_layer_buffers layer = {q, k_new, v_new, k_cache, v_cache, out};
  return pda_model_step_graph_create(prob, 1, &layer, block_table, context_lens, scale, workspace, workspace_bytes,
                                     graph);
}

int pda_model_step_graph_create(const pda_problem* prob, int32_t num_layers, const pda_layer_buffers* layers,
                                const int32_t* block_table, const int32_t* context_lens, float scale,
                                void* workspace, size_t workspace_bytes, pda_step_graph** graph) {
  if (!graph) return PDA_ERR_NULL;
  *graph = nullptr;
  if (num_layers < 1) return PDA_ERR_SHAPE;
  if (!layers) return PDA_ERR_NULL;
  // validate every layer before capturing anything
  Plan plan;
  for (int32_t l = 0; l < num_layers; ++l) {
    const pda_layer_buffers& L = layers[l];
    pda::StepArgs append_args, args;
    int rc = prepare_append(prob, L.k_new, L.v_new, block_table, context_lens, L.k_cache, L.v_cache, &append_args);
    if (rc != PDA_OK) return rc;
    rc = prepare_step(prob, nullptr, L.q, L.k_cache, L.v_cache, block_table, context_lens, scale, L.out, workspace,
                      workspace_bytes, &plan, &args);
    if (rc != PDA_OK) return rc;
  }
  pda_step_graph* g = new (std::nothrow) pda_step_graph{nullptr, nullptr, prob->num_seqs == 0};
  if (!g) return PDA_ERR_HIP;
  if (g->empty) {
    *graph = g;
    return PDA_OK;
  }
  hipStream_t s = nullptr;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) {
    delete g;
    return PDA_ERR_HIP;
  }
  int rc = PDA_OK;
  if (hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) != hipSuccess) {
    rc = PDA_ERR_HIP;
  } else {
    // the launches of pda_append_kv + pda_decode for each layer, with the
    // work order (the lengths are the same in every layer) computed once
    for (int32_t l = 0; l < num_layers && rc == PDA_OK; ++l) {
      const pda_layer_buffers& L = layers[l];
      pda::StepArgs append_args, args;
      prepare_append(prob, L.k_new, L.v_new, block_table, context_lens, L.k_cache, L.v_cache, &append_args);
      prepare_step(prob, nullptr, L.q, L.k_cache, L.v_cache, block_table, context_lens, scale, L.out, workspace,
                   workspace_bytes, &plan, &args);
      // a small step with one new token per sequence: pass 1 stores it (one launch less per layer)
      const bool fold = folds_append(prob, plan);
      if (fold) fold_append(&args, L.k_new, L.v_new, L.k_cache, L.v_cache);
      if ((!fold && launch_append_of(prob, append_args, L.k_new, L.v_new, L.k_cache, L.v_cache, s) != hipSuccess) ||
          (l == 0 && args.order && pda::launch_order(args, s) != hipSuccess) ||
          pda::launch_partition(args, prob->head_dim, s) != hipSuccess ||
          (plan.slots > 0 && pda::launch_merge(args, prob->head_dim, s) != hipSuccess))
        rc = PDA_ERR_HIP;
    }
    hipGraph_t captured = nullptr;
    const hipError_t end = hipStreamEndCapture(s, &captured);  // always ends the capture
    g->graph = captured;
    if (rc == PDA_OK && (end != hipSuccess || !captured)) rc = PDA_ERR_HIP;
    if (rc == PDA_OK && hipGraphInstantiate(&g->exec, captured, nullptr, nullptr, 0) != hipSuccess) rc = PDA_ERR_HIP;
  }
  (void)hipStreamDestroy(s);
  if (rc != PDA_OK) {
    pda_step_graph_destroy(g);
    return rc;
  }
  *graph = g;
  return PDA_OK;
}

int pda_step_graph_launch(pda_step_graph* graph, hipStream_t stream) {
  if (!graph) return PDA_ERR_NULL;
  if (graph->empty) return PDA_OK;
  return hipGraphLaunch(graph->exec, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_step_graph_destroy(pda_step_graph* graph) {
  if (!graph) return PDA_OK;
  int rc = PDA_OK;
  if (graph->exec && hipGraphExecDestroy(graph->exec) != hipSuccess) rc = PDA_ERR_HIP;
  if (graph->graph && hipGraphDestroy(graph->graph) != hipSuccess) rc = PDA_ERR_HIP;
  delete graph;
  return rc;
}

int pda_plan_shared_prefix(const pda_problem* prob, const pda_prefix_groups* groups, pda_plan_info* info) {
  if (!info) return PDA_ERR_NULL;
  Plan plan;
  int rc = make_plan(prob, groups, &plan);
  if (rc != PDA_OK) return rc;
  *info = plan.info;
  return PDA_OK;
}

int pda_decode_shared_prefix(const pda_problem* prob, const pda_prefix_groups* groups, const void* q,
                             const void* k_cache, const void* v_cache, const int32_t* block_table,
                             const int32_t* context_lens, float scale, float* out, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!groups) return PDA_ERR_NULL;
  Plan plan;
  pda::StepArgs args;
  int rc = prepare_step(prob, groups, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                        workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  return launch_attention(prob, plan, args, stream);
}

int pda_logprob_workspace_bytes(int32_t num_rows, int32_t vocab, int32_t logits_dtype, size_t* bytes) {
  if (!bytes) return PDA_ERR_NULL;
  if (num_rows < 0 || vocab < 1) return PDA_ERR_SHAPE;
  if (logits_dtype != PDA_DTYPE_BF16 && logits_dtype != PDA_DTYPE_F32) return PDA_ERR_UNSUPPORTED;
  const int S = pda::logprob_slices(num_rows, vocab, logits_dtype == PDA_DTYPE_BF16 ? 2 : 4);
  *bytes = S > 1 ? (size_t)num_rows * S * 16 : 0;  // S partial states of 16 bytes per row
  return PDA_OK;
}

int pda_token_logprobs(int32_t num_rows, int32_t vocab, int64_t row_stride, int32_t logits_dtype, const void* logits,
                       const int32_t* tokens, float inv_temperature, float* logprobs, float* entropies,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (num_rows < 0 || vocab < 1 || row_stride < vocab) return PDA_ERR_SHAPE;
  if (logits_dtype != PDA_DTYPE_BF16 && logits_dtype != PDA_DTYPE_F32) return PDA_ERR_UNSUPPORTED;
  const int esize = logits_dtype == PDA_DTYPE_BF16 ? 2 : 4;
  if ((int64_t)vocab * esize + 64 > 0x7fffffff) return PDA_ERR_SHAPE;  // one row must fit a buffer descriptor
  if ((int64_t)num_rows * pda::kLpMaxSlices > 0x7fffffff) return PDA_ERR_SHAPE;  // the grid
  if (num_rows == 0) return PDA_OK;
  if (!logits || !tokens || !logprobs) return PDA_ERR_NULL;
  if (!isfinite(inv_temperature) || inv_temperature < 0.f) return PDA_ERR_VALUE;
  if (!aligned(logits, 16) || (row_stride * esize) % 16 != 0 || !aligned(logprobs, 4) || !aligned(entropies, 4))
    return PDA_ERR_ALIGNMENT;
  pda::LogprobArgs a;
  a.logits = logits;
  a.tokens = tokens;
  a.logprobs = logprobs;
  a.entropies = entropies;
  a.inv_temperature = inv_temperature;
  a.num_rows = num_rows;
  a.vocab = vocab;
  a.row_stride = row_stride;
  a.elem_bytes = esize;
  a.slices = 1;
  a.part = nullptr;
  if (workspace) {
    size_t need = 0;
    pda_logprob_workspace_bytes(num_rows, vocab, logits_dtype, &need);
    if (workspace_bytes < need) return PDA_ERR_WORKSPACE;
    if (!aligned(workspace, 16)) return PDA_ERR_ALIGNMENT;
    if (need > 0) {
      a.slices = pda::logprob_slices(num_rows, vocab, esize);
      a.part = static_cast<float*>(workspace);
    }
  }
  return pda::launch_logprob(a, stream) == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_validate_host(const pda_problem* prob, const int32_t* block_table, const int32_t* context_lens,
                      int64_t* first_bad) {
  int rc = check_problem(prob);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs > 0 && (!block_table || !context_lens)) return PDA_ERR_NULL;
  for (int32_t b = 0; b < prob->num_seqs; ++b) {
    const int32_t L = context_lens[b];
    if (L > prob->max_context_len) {
      if (first_bad) *first_bad = b;
      return PDA_ERR_VALUE;
    }
    const int32_t nblk = L > 0 ? (L + pda::kBlockTokens - 1) / pda::kBlockTokens : 0;
    for (int32_t j = 0; j < nblk; ++j) {
      const int64_t idx = (int64_t)b * prob->max_blocks_per_seq + j;
      const int32_t id = block_table[idx];
      if (id < 0 || id >= prob->num_blocks) {
        if (first_bad) *first_bad = idx;
        return PDA_ERR_VALUE;
      }
    }
  }
  return PDA_OK;
}

const char* pda_status_string(int status) {
  switch (status) {
    case PDA_OK: return "PDA_OK: success";
    case PDA_ERR_NULL: return "PDA_ERR_NULL: a required pointer is NULL";
    case PDA_ERR_SHAPE: return "PDA_ERR_SHAPE: sizes out of range or inconsistent";
    case PDA_ERR_UNSUPPORTED:
      return "PDA_ERR_UNSUPPORTED: head_dim must be 64 or 128, block_size 16, Hq/Hkv <= 16 (shared-prefix "
             "groups: n Hq/Hkv <= 64; pda_decode_append: one new token; logits bf16 or fp32)";
    case PDA_ERR_WORKSPACE: return "PDA_ERR_WORKSPACE: workspace missing or smaller than pda_workspace_bytes()";
    case PDA_ERR_ALIGNMENT:
      return "PDA_ERR_ALIGNMENT: q/k_cache/v_cache/k_new/v_new/out/workspace/logits need 16-byte alignment "
             "(log-prob outputs 4-byte)";
    case PDA_ERR_VALUE: return "PDA_ERR_VALUE: non-finite scale or invalid device contents";
    case PDA_ERR_HIP: return "PDA_ERR_HIP: a HIP launch, graph capture or instantiation failed";
    case PDA_ERR_SCRATCH:
      return "PDA_ERR_SCRATCH: the step needs more workspace than pda_decode_noalloc's static scratch holds";
    default: return "unknown pda status";
  }
}

}  // extern "C"
