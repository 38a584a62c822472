// Sanitizer driver for the host side of the C ABI (test infrastructure).
// pda_api.hip is compiled for the host only, under AddressSanitizer and
// UndefinedBehaviorSanitizer, and linked with the launchers below, which
// stand in for the GPU kernels and report a failed launch.  The driver feeds
// the descriptor checks, the plan and the host validation seeded random and
// extreme descriptors (negative, zero, huge and wrapping sizes) and checks
// the invariants of the plan; any out-of-bounds access, signed overflow or
// other undefined operation aborts the run through the sanitizer.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "pda.h"
#include "pda_internal.h"

namespace pda {  // no GPU here: every launch reports failure
hipError_t launch_logprob(const LogprobArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_append(const StepArgs&, const uint16_t*, const uint16_t*, uint16_t*, uint16_t*, int, hipStream_t) {
  return hipErrorInvalidValue;
}
hipError_t launch_order(const StepArgs&, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_partition(const StepArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_merge(const StepArgs&, int, hipStream_t) { return hipErrorInvalidValue; }
}  // namespace pda

static uint64_t state = 11143;
static uint32_t next_u32() {  // xorshift64*
  state ^= state >> 12;
  state ^= state << 25;
  state ^= state >> 27;
  return (uint32_t)((state * 2685821657736338717ull) >> 32);
}
static int32_t pick(const std::vector<int32_t>& v) { return v[next_u32() % v.size()]; }

static int fails = 0;
#define EXPECT(c)                                              \
  do {                                                         \
    if (!(c)) {                                                \
      fprintf(stderr, "line %d: %s failed\n", __LINE__, #c);   \
      ++fails;                                                 \
    }                                                          \
  } while (0)

int main() {
  const std::vector<int32_t> sizes = {-1, 0, 1, 2, 3, 7, 8, 16, 17, 64, 255, 256, 4096, 65536, 1 << 20, 1 << 30,
                                      0x7fffffff, (int32_t)0x80000000};
  const std::vector<int32_t> dims = {-64, 0, 32, 64, 96, 128, 256};
  alignas(16) static char dummy[256];
  for (int it = 0; it < 20000; ++it) {
    pda_problem p;
    p.num_seqs = pick(sizes);
    p.num_q_heads = pick(sizes);
    p.num_kv_heads = pick(sizes);
    if (next_u32() % 2) {  // mostly valid head counts
      p.num_kv_heads = 1 + next_u32() % 8;
      p.num_q_heads = p.num_kv_heads * (1 + next_u32() % 17);
    }
    p.head_dim = next_u32() % 4 ? (next_u32() % 2 ? 64 : 128) : pick(dims);
    p.block_size = next_u32() % 8 ? 16 : pick(sizes);
    p.num_blocks = pick(sizes);
    p.max_blocks_per_seq = pick(sizes);
    p.max_context_len = next_u32() % 2 ? (int32_t)(next_u32() % 70000) : pick(sizes);
    p.partition_tokens = next_u32() % 2 ? 0 : (next_u32() % 3 ? 16 * (int32_t)(next_u32() % 300) : pick(sizes));
    p.num_query_tokens = next_u32() % 2 ? 1 : pick(sizes);
    pda_plan_info info;
    const int rc = pda_plan(&p, &info);
    size_t ws = 0;
    EXPECT(pda_workspace_bytes(&p, &ws) == rc);
    if (rc == PDA_OK) {
      EXPECT(ws == info.workspace_bytes);
      const int before = fails;
      EXPECT(info.partition_tokens > 0 && info.partition_tokens % 16 == 0);
      EXPECT(info.num_partitions >= 1);
      EXPECT((int64_t)info.num_partitions * info.partition_tokens >= p.max_context_len);
      EXPECT(p.num_seqs == 0 || ws > 0);
      if (fails != before)
        fprintf(stderr, "  descriptor B=%d Hq=%d Hkv=%d D=%d mbps=%d mcl=%d tp=%d n=%d -> tp %d P %d\n", p.num_seqs,
                p.num_q_heads, p.num_kv_heads, p.head_dim, p.max_blocks_per_seq, p.max_context_len,
                p.partition_tokens, p.num_query_tokens, info.partition_tokens, info.num_partitions);
      // a valid step reaches its first launch, which fails here
      const int drc = pda_decode(&p, dummy, dummy, dummy, (const int32_t*)dummy, (const int32_t*)dummy, 0.125f,
                                 (float*)dummy, dummy, ws, nullptr);
      EXPECT(drc == (p.num_seqs == 0 ? PDA_OK : PDA_ERR_HIP));
    }
    pda_prefix_groups g;
    g.num_groups = next_u32() % 2 ? (int32_t)(next_u32() % 40) : pick(sizes);
    g.max_group_size = next_u32() % 2 ? (int32_t)(1 + next_u32() % 20) : pick(sizes);
    g.max_prefix_len = next_u32() % 2 ? 16 * (int32_t)(next_u32() % 100) : pick(sizes);
    g.group_start = (const int32_t*)dummy;
    g.group_prefix_len = (const int32_t*)dummy;
    const int grc = pda_plan_shared_prefix(&p, &g, &info);
    if (grc == PDA_OK) {
      // one member's rows fit a prefix item; larger groups take several row groups
      EXPECT((int64_t)(p.num_query_tokens > 0 ? p.num_query_tokens : 1) * (p.num_q_heads / p.num_kv_heads) <= 64);
      EXPECT(p.num_seqs == 0 || info.workspace_bytes > 0);
    }
  }
  // host validation of device contents on random tables
  for (int it = 0; it < 200; ++it) {
    pda_problem p{};
    p.num_seqs = 1 + next_u32() % 20;
    p.num_q_heads = 8;
    p.num_kv_heads = 2;
    p.head_dim = 64;
    p.block_size = 16;
    p.num_blocks = 1 + next_u32() % 50;
    p.max_blocks_per_seq = 1 + next_u32() % 10;
    p.max_context_len = (int32_t)(next_u32() % (16 * p.max_blocks_per_seq + 1));
    std::vector<int32_t> table((size_t)p.num_seqs * p.max_blocks_per_seq), lens(p.num_seqs);
    for (auto& x : table) x = (int32_t)(next_u32() % (p.num_blocks + 2)) - 1;
    for (auto& x : lens) x = (int32_t)(next_u32() % (p.max_context_len + 3)) - 1;
    int64_t bad = -1;
    const int rc = pda_validate_host(&p, table.data(), lens.data(), &bad);
    EXPECT(rc == PDA_OK || (rc == PDA_ERR_VALUE && bad >= 0));
  }
  // log-prob argument checks
  EXPECT(pda_token_logprobs(4, 0, 0, PDA_DTYPE_BF16, dummy, (const int32_t*)dummy, 1.f, (float*)dummy, nullptr,
                            nullptr, 0, nullptr) == PDA_ERR_SHAPE);
  EXPECT(pda_token_logprobs(4, 0x7fffffff, 0x7fffffff, PDA_DTYPE_F32, dummy, (const int32_t*)dummy, 1.f,
                            (float*)dummy, nullptr, nullptr, 0, nullptr) == PDA_ERR_SHAPE);
  EXPECT(pda_token_logprobs(4, 1000, 1000, PDA_DTYPE_BF16, dummy, (const int32_t*)dummy, 1.f, (float*)dummy,
                            nullptr, nullptr, 0, nullptr) == PDA_ERR_HIP);
  // log-prob workspace sizes over random shapes
  for (int it = 0; it < 2000; ++it) {
    const int32_t rows = pick(sizes), vocab = pick(sizes);
    size_t bytes = 1;
    const int rc = pda_logprob_workspace_bytes(rows, vocab, (int32_t)(next_u32() % 3), &bytes);
    EXPECT(rc != PDA_OK || rows < 0 || vocab < 1 || bytes == 0 || bytes % 16 == 0);
  }
  for (int s = -2; s < 12; ++s) EXPECT(strlen(pda_status_string(s)) > 0);
  if (fails) {
    fprintf(stderr, "%d check(s) failed\n", fails);
    return 1;
  }
  printf("host ABI sanitizer driver: all checks passed\n");
  return 0;
}
