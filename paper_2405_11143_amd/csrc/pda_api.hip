// C ABI of the paged decode-attention library (declared in include/pda.h):
// host-side validation, the split-K plan, and the two kernel launches.
// Nothing here allocates memory or keeps state between calls.
#include <math.h>

#include "pda.h"
#include "pda_internal.h"

namespace {

// Split-K policy: partitions of kMaxPartitionTokens, halved (down to
// kMinPartitionTokens) while the step would have fewer than kMinWorkItems
// (sequence, KV head, partition) items -- too few to keep 256 compute units
// busy -- and never longer than the longest context (then there is one
// partition and no merge pass).  Larger partitions amortise each workgroup's start-up
// (lengths, block ids, q) over more streamed tiles; on MI355X 2048 tokens
// measured fastest on all four Llama-3-shaped decode steps.
constexpr int kMaxPartitionTokens = 2048;
constexpr int kMinPartitionTokens = 256;
constexpr int64_t kMinWorkItems = 2048;

int check_problem(const pda_problem* p) {
  if (!p) return PDA_ERR_NULL;
  if (p->num_seqs < 0 || p->num_q_heads < 1 || p->num_kv_heads < 1 || p->num_blocks < 1 ||
      p->max_blocks_per_seq < 1 || p->max_context_len < 0 || p->partition_tokens < 0)
    return PDA_ERR_SHAPE;
  if (p->num_q_heads % p->num_kv_heads != 0) return PDA_ERR_SHAPE;
  if (p->partition_tokens % pda::kBlockTokens != 0) return PDA_ERR_SHAPE;
  if ((int64_t)p->max_context_len > (int64_t)pda::kBlockTokens * p->max_blocks_per_seq) return PDA_ERR_SHAPE;
  if (p->block_size != pda::kBlockTokens) return PDA_ERR_UNSUPPORTED;
  if (p->head_dim != 64 && p->head_dim != 128) return PDA_ERR_UNSUPPORTED;
  if (p->num_q_heads / p->num_kv_heads > pda::kMaxGroup) return PDA_ERR_UNSUPPORTED;
  return PDA_OK;
}

struct Plan {
  int32_t partition_tokens;
  int32_t num_partitions;  // partitions of the longest context, at least 1 (grid extent)
  size_t workspace_bytes;
  size_t part_o_floats;    // offset of part_m in floats
  size_t part_ml_floats;   // length of part_m (and of part_l) in floats
};

int make_plan(const pda_problem* p, Plan* plan) {
  int rc = check_problem(p);
  if (rc != PDA_OK) return rc;
  int tp = p->partition_tokens;
  if (tp == 0) {
    const int64_t units = (int64_t)p->num_seqs * p->num_kv_heads;
    const int64_t len = p->max_context_len > 0 ? p->max_context_len : 1;
    tp = kMaxPartitionTokens;
    while (tp > kMinPartitionTokens && units * ((len + tp - 1) / tp) < kMinWorkItems) tp /= 2;
    const int rounded = (int)((len + pda::kBlockTokens - 1) / pda::kBlockTokens * pda::kBlockTokens);
    if (rounded < tp) tp = rounded;  // the whole context fits one partition
  }
  const int64_t parts = p->max_context_len > 0 ? ((int64_t)p->max_context_len + tp - 1) / tp : 1;
  const int64_t grid = parts * p->num_seqs * p->num_kv_heads;
  if (grid > 0x7fffffff) return PDA_ERR_SHAPE;
  plan->partition_tokens = tp;
  plan->num_partitions = (int32_t)parts;
  if (parts > 1) {
    const size_t rows = (size_t)p->num_seqs * p->num_q_heads * (size_t)parts;
    plan->part_o_floats = rows * p->head_dim;
    plan->part_ml_floats = rows;
    plan->workspace_bytes = (plan->part_o_floats + 2 * rows) * sizeof(float);
  } else {
    plan->part_o_floats = plan->part_ml_floats = 0;
    plan->workspace_bytes = 0;
  }
  return PDA_OK;
}

bool aligned(const void* ptr, size_t a) { return ((uintptr_t)ptr % a) == 0; }

// Validation shared by the entry points that launch pass 1; fills `args`.
int prepare_step(const pda_problem* p, const void* q, const void* k, const void* v, const int32_t* bt,
                 const int32_t* lens, float scale, float* out, void* ws, size_t ws_bytes, Plan* plan,
                 pda::StepArgs* args) {
  int rc = make_plan(p, plan);
  if (rc != PDA_OK) return rc;
  if (p->num_seqs > 0 && (!q || !k || !v || !bt || !lens || !out)) return PDA_ERR_NULL;
  if (!isfinite(scale)) return PDA_ERR_VALUE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 4)) return PDA_ERR_ALIGNMENT;
  if (plan->workspace_bytes > 0) {
    if (!ws || ws_bytes < plan->workspace_bytes) return PDA_ERR_WORKSPACE;
    if (!aligned(ws, 16)) return PDA_ERR_ALIGNMENT;
  }
  float* wsf = static_cast<float*>(ws);
  *args = pda::StepArgs{static_cast<const uint16_t*>(q),
                        static_cast<const uint16_t*>(k),
                        static_cast<const uint16_t*>(v),
                        bt,
                        lens,
                        out,
                        plan->workspace_bytes ? wsf : nullptr,
                        plan->workspace_bytes ? wsf + plan->part_o_floats : nullptr,
                        plan->workspace_bytes ? wsf + plan->part_o_floats + plan->part_ml_floats : nullptr,
                        scale * 1.4426950408889634f,
                        p->num_seqs,
                        p->num_q_heads,
                        p->num_kv_heads,
                        p->num_blocks,
                        p->max_blocks_per_seq,
                        p->max_context_len,
                        plan->partition_tokens,
                        plan->num_partitions};
  return PDA_OK;
}

}  // namespace

extern "C" {

int pda_plan(const pda_problem* prob, int32_t* partition_tokens, int32_t* num_partitions,
             size_t* workspace_bytes) {
  Plan plan;
  int rc = make_plan(prob, &plan);
  if (rc != PDA_OK) return rc;
  if (partition_tokens) *partition_tokens = plan.partition_tokens;
  if (num_partitions) *num_partitions = plan.num_partitions;
  if (workspace_bytes) *workspace_bytes = plan.workspace_bytes;
  return PDA_OK;
}

int pda_workspace_bytes(const pda_problem* prob, size_t* bytes) {
  if (!bytes) return PDA_ERR_NULL;
  return pda_plan(prob, nullptr, nullptr, bytes);
}

int pda_partition_attention(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
                            const int32_t* block_table, const int32_t* context_lens, float scale, float* out,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  Plan plan;
  pda::StepArgs args;
  int rc = prepare_step(prob, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                        workspace_bytes, &plan, &args);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0) return PDA_OK;
  const int group = prob->num_q_heads / prob->num_kv_heads;
  if (pda::launch_partition(args, group, prob->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  return PDA_OK;
}

int pda_merge_partitions(const pda_problem* prob, const int32_t* context_lens, float* out, const void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  Plan plan;
  int rc = make_plan(prob, &plan);
  if (rc != PDA_OK) return rc;
  if (prob->num_seqs == 0 || plan.workspace_bytes == 0) return PDA_OK;  // nothing was split
  if (!context_lens || !out) return PDA_ERR_NULL;
  if (!workspace || workspace_bytes < plan.workspace_bytes) return PDA_ERR_WORKSPACE;
  if (!aligned(workspace, 16) || !aligned(out, 4)) return PDA_ERR_ALIGNMENT;
  const float* wsf = static_cast<const float*>(workspace);
  pda::StepArgs args{};
  args.lens = context_lens;
  args.out = out;
  args.part_o = const_cast<float*>(wsf);
  args.part_m = const_cast<float*>(wsf + plan.part_o_floats);
  args.part_l = const_cast<float*>(wsf + plan.part_o_floats + plan.part_ml_floats);
  args.num_seqs = prob->num_seqs;
  args.num_q_heads = prob->num_q_heads;
  args.num_kv_heads = prob->num_kv_heads;
  args.num_blocks = prob->num_blocks;
  args.max_blocks_per_seq = prob->max_blocks_per_seq;
  args.max_context_len = prob->max_context_len;
  args.partition_tokens = plan.partition_tokens;
  args.num_partitions = plan.num_partitions;
  if (pda::launch_merge(args, prob->head_dim, stream) != hipSuccess) return PDA_ERR_HIP;
  return PDA_OK;
}

int pda_decode(const pda_problem* prob, const void* q, const void* k_cache, const void* v_cache,
               const int32_t* block_table, const int32_t* context_lens, float scale, float* out, void* workspace,
               size_t workspace_bytes, hipStream_t stream) {
  int rc = pda_partition_attention(prob, q, k_cache, v_cache, block_table, context_lens, scale, out, workspace,
                                   workspace_bytes, stream);
  if (rc != PDA_OK) return rc;
  return pda_merge_partitions(prob, context_lens, out, workspace, workspace_bytes, stream);
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
    case PDA_ERR_UNSUPPORTED: return "PDA_ERR_UNSUPPORTED: head_dim must be 64 or 128, block_size 16, Hq/Hkv <= 16";
    case PDA_ERR_WORKSPACE: return "PDA_ERR_WORKSPACE: workspace missing or smaller than pda_workspace_bytes()";
    case PDA_ERR_ALIGNMENT: return "PDA_ERR_ALIGNMENT: q/k_cache/v_cache/workspace need 16-byte alignment, out 4-byte";
    case PDA_ERR_VALUE: return "PDA_ERR_VALUE: non-finite scale or invalid device contents";
    case PDA_ERR_HIP: return "PDA_ERR_HIP: a HIP kernel launch failed";
    default: return "unknown pda status";
  }
}

}  // extern "C"
