// Internal interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pda {

constexpr int kBlockTokens = 16;  // tokens per KV-cache block
constexpr int kWaveSize = 64;     // CDNA wavefront
constexpr int kWaves = 4;         // wavefronts per partition workgroup
constexpr int kMaxGroup = 16;     // query heads per KV head: one 16-row MFMA tile
constexpr int kWideChunks = 2 * kWaves;  // query chunks of a work item when each wavefront folds two
constexpr int kWide16Chunks = 4 * kWaves;  // the same with 8 wavefronts per workgroup (more than 8 chunks)
constexpr int kOrderThreads = 1024;  // the work-order kernel is one workgroup of this size
constexpr int kOrderBuckets = 256;   // size classes of its counting sort (partition blocks, capped)

// Kernel arguments for one step (passed by value).  n = num_query_tokens new
// tokens per sequence (1 for a decode step); new token i of sequence b sits at
// position L_b - n + i of its context.
struct StepArgs {
  const uint16_t* q;       // bf16 [B][n][Hq][D]
  const uint16_t* k;       // bf16 [num_blocks][Hkv][D/8][16][8]
  const uint16_t* v;       // bf16 [num_blocks][Hkv][16][D]
  const int32_t* table;    // int32 [B][max_blocks_per_seq]
  const int32_t* lens;     // int32 [B]
  float* out;              // fp32 [B][n][Hq][D]
  int32_t* order;          // int32 [items]: work item of each workgroup, largest partition first,
                           // placed for the XCDs (null: workgroup i runs item i)
  float* part_o;           // fp32 [B*n*Hq*slots_per_row][D]  unnormalised partition outputs
  float* part_m;           // fp32 [B*n*Hq*slots_per_row]     partition reference max, log2 domain
  float* part_l;           // fp32 [B*n*Hq*slots_per_row]     partition softmax denominators
  float scale_log2;        // softmax scale * log2(e)
  int32_t num_seqs;        // B
  int32_t num_q_heads;     // Hq
  int32_t num_kv_heads;    // Hkv
  int32_t group;           // G = Hq / Hkv
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t max_context_len;
  int32_t num_query_tokens;  // n
  int32_t query_chunk;       // new tokens per query chunk (one 16-row tile): min(n, 16 / G)
  int32_t num_query_chunks;  // NQC = ceil(n / query_chunk)
  int32_t chunks_per_group;  // CPG: 4; 8 when NQC > 4 (each wavefront then folds two tiles); 16 when NQC > 8
                             // (8 wavefronts of two tiles)
  int32_t num_chunk_groups;  // NCG = ceil(NQC / CPG): chunks of one work item share its K/V tiles
  int32_t partition_tokens;  // T_p, multiple of 16
  int32_t num_partitions;    // P = max(1, ceil(max_context_len / T_p))
  // Shared-prefix groups (num_groups == 0: none).  The members of group i are
  // sequences [group_start[i], group_start[i+1]); their first
  // group_prefix_len[i] tokens sit in the same blocks.
  const int32_t* group_start;       // int32 [num_groups + 1]
  const int32_t* group_prefix_len;  // int32 [num_groups], multiples of 16
  int32_t* seq_prefix;              // int32 [B] (workspace): prefix tokens of each sequence's group
  int32_t num_groups;
  int32_t max_group_size;           // bound on the members of one group
  int32_t max_prefix_len;           // bound on group_prefix_len, multiple of 16
  int32_t prefix_partitions;        // Pp = ceil(max_prefix_len / T_p)
  int32_t members_per_row_group;    // MR = 64 / (n G): members whose query rows fill one prefix item
  int32_t prefix_row_groups;        // RG = ceil(min(max_group_size, B) / MR): prefix items per group and partition
  int32_t slots_per_row;            // Pp + P partial states per output row (P when no groups)
  int32_t num_regular_items;        // items below this index are (partition, sequence, KV head, chunk group)
  int32_t num_prefix_items;         // num_groups * Pp * RG * Hkv items after them
  // The step's KV append folded into pass 1 (one new token per sequence, no
  // shared-prefix groups), or null: the item that reads position L - 1 of
  // (sequence, KV head) first stores that token's K and V rows there.
  const uint16_t* k_new;            // bf16 [B][Hkv][D]
  const uint16_t* v_new;            // bf16 [B][Hkv][D]
  uint16_t* k_store;                // the K cache (a.k, writable)
  uint16_t* v_store;                // the V cache (a.v, writable)
};

// Prefix tokens of sequence b's group (0 without groups); pass 1 and the
// merge treat tokens [0, prefix) as covered by the group's prefix items.
__device__ __forceinline__ int seq_prefix_len(const StepArgs& a, int b) {
  return a.seq_prefix ? a.seq_prefix[b] : 0;
}

// Tokens that the last row of query chunk `chunk` sees (<= 0: none).
__device__ __forceinline__ int chunk_visible(const StepArgs& a, int L, int chunk) {
  const int i0 = chunk * a.query_chunk;
  const int nv = min(a.query_chunk, a.num_query_tokens - i0);
  return L - a.num_query_tokens + i0 + nv;
}

// The token log-probability kernel: 1024-thread workgroups, one per row; a
// batch with fewer rows than compute units has its rows split into `slices`
// workgroups when the caller gives a workspace, so that every compute unit
// streams part of a row.
constexpr int kLpThreads = 1024;
constexpr int kLpTargetWorkgroups = 256;  // one per compute unit
constexpr int kLpMaxSlices = 16;

// Workgroups per row for a log-prob call with a workspace (1: none needed).
inline int logprob_slices(int rows, int vocab, int elem_bytes) {
  if (rows <= 0) return 1;
  const long chunks = (long)vocab * elem_bytes / 16;  // whole 16-byte chunks of a row
  long s = (kLpTargetWorkgroups + (long)rows - 1) / rows;
  if (s > kLpMaxSlices) s = kLpMaxSlices;
  if (s > chunks / kLpThreads) s = chunks / kLpThreads;  // at least a chunk per thread in each slice
  return s < 1 ? 1 : (int)s;
}

// Arguments of the token log-probability kernel (passed by value).
struct LogprobArgs {
  const void* logits;      // [num_rows][row_stride] bf16 or fp32, the first `vocab` of each row used
  const int32_t* tokens;   // int32 [num_rows]
  float* logprobs;         // fp32 [num_rows]
  float* entropies;        // fp32 [num_rows], or null
  float inv_temperature;   // 1 / T
  int32_t num_rows;
  int32_t vocab;
  int64_t row_stride;      // elements
  int32_t elem_bytes;      // 2 (bf16) or 4 (fp32)
  int32_t slices;          // workgroups per row (1: no workspace, or enough rows)
  float* part;             // [num_rows][slices][4] partial states (mk, s, t, -) when slices > 1
};

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Results are written with the non-temporal hint, 16 (or 8) bytes per lane:
// the outputs are read by the next layer, not by this step, and on MI355X
// plain 4-byte stores at the end of every work item cost the Llama-3-8B step
// 0.75% and a 4-new-token step 4%.
__device__ __forceinline__ void store_nt4(float* p, float x, float y, float z, float w) {
  __builtin_nontemporal_store(f32x4_t{x, y, z, w}, reinterpret_cast<f32x4_t*>(p));
}
__device__ __forceinline__ void store_nt2(float* p, float x, float y) {
  __builtin_nontemporal_store(f32x2_t{x, y}, reinterpret_cast<f32x2_t*>(p));
}

// Launchers (asynchronous; return the hipGetLastError() of the launch).
hipError_t launch_logprob(const LogprobArgs& a, hipStream_t stream);
hipError_t launch_append(const StepArgs& a, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                         uint16_t* v_cache, int head_dim, hipStream_t stream);
hipError_t launch_order(const StepArgs& a, hipStream_t stream);
hipError_t launch_partition(const StepArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_merge(const StepArgs& a, int head_dim, hipStream_t stream);

}  // namespace pda
