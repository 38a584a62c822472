// KV-cache append: store the keys and values of each sequence's new tokens
// in the paged cache, the step that precedes attention in every decode step
// (KV-cache management of the rollout stage, Appendix C).
//
// New token i of sequence b (n new tokens, context length L counting them)
// goes to position t = L - n + i: block table[b][t / 16], slot t % 16.  One
// thread moves one 16-byte piece (8 consecutive elements of one head's row):
// in V that is part of the slot's row, in K it is the slot's entry of one
// d-chunk, [p][g][d/8][slot][0..8).  Positions t < 0 are skipped, and so is
// a block id outside the pool (the caller's contract; never written).
#include "pda_internal.h"

namespace pda {
namespace {

constexpr int kAppendThreads = 256;

template <int D>
__global__ void __launch_bounds__(kAppendThreads)
append_kernel(const StepArgs a, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache) {
  constexpr int CPR = D / 8;  // 16-byte pieces per head row
  const int n = a.num_query_tokens;
  const int Hkv = a.num_kv_heads;
  const size_t idx = (size_t)blockIdx.x * kAppendThreads + threadIdx.x;  // [b][i][g][c]
  if (idx >= (size_t)a.num_seqs * n * Hkv * CPR) return;
  const int c = (int)(idx % CPR);
  const int g = (int)((idx / CPR) % Hkv);
  const int i = (int)((idx / ((size_t)CPR * Hkv)) % n);
  const int b = (int)(idx / ((size_t)CPR * Hkv * n));
  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  const int t = L - n + i;
  if (t < 0) return;
  const int p = a.table[(size_t)b * a.max_blocks_per_seq + t / kBlockTokens];
  if ((unsigned)p >= (unsigned)a.num_blocks) return;
  const int o = t % kBlockTokens;
  const uint4 kv = reinterpret_cast<const uint4*>(k_new)[idx];
  const uint4 vv = reinterpret_cast<const uint4*>(v_new)[idx];
  const size_t tile = (size_t)p * Hkv + g;
  reinterpret_cast<uint4*>(k_cache)[(tile * CPR + c) * kBlockTokens + o] = kv;
  reinterpret_cast<uint4*>(v_cache)[(tile * kBlockTokens + o) * CPR + c] = vv;
}

template <int D>
hipError_t launch_d(const StepArgs& a, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                    uint16_t* v_cache, hipStream_t stream) {
  const size_t total = (size_t)a.num_seqs * a.num_query_tokens * a.num_kv_heads * (D / 8);
  const unsigned grid = (unsigned)((total + kAppendThreads - 1) / kAppendThreads);
  hipLaunchKernelGGL((append_kernel<D>), dim3(grid), dim3(kAppendThreads), 0, stream, a, k_new, v_new, k_cache,
                     v_cache);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_append(const StepArgs& a, const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                         uint16_t* v_cache, int head_dim, hipStream_t stream) {
  if (head_dim == 64) return launch_d<64>(a, k_new, v_new, k_cache, v_cache, stream);
  if (head_dim == 128) return launch_d<128>(a, k_new, v_new, k_cache, v_cache, stream);
  return hipErrorInvalidValue;
}

}  // namespace pda
