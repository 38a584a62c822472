// Internal interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

namespace pda {

constexpr int kBlockTokens = 16;  // tokens per KV-cache block
constexpr int kWaveSize = 64;     // CDNA wavefront
constexpr int kWaves = 4;         // wavefronts per partition workgroup
constexpr int kMaxGroup = 16;     // query heads per KV head handled by one MFMA row tile
constexpr int kOrderThreads = 1024;  // the work-order kernel is one workgroup of this size
constexpr int kOrderBuckets = 256;   // size classes of its counting sort (partition blocks, capped)

// Kernel arguments for one decode step (passed by value).
struct StepArgs {
  const uint16_t* q;       // bf16 [B][Hq][D]
  const uint16_t* k;       // bf16 [num_blocks][Hkv][D/8][16][8]
  const uint16_t* v;       // bf16 [num_blocks][Hkv][16][D]
  const int32_t* table;    // int32 [B][max_blocks_per_seq]
  const int32_t* lens;     // int32 [B]
  float* out;              // fp32 [B][Hq][D]
  int32_t* order;          // int32 [P*B*Hkv]: work items, largest partition first
  float* part_o;           // fp32 [B*Hq*P][D]  unnormalised partition outputs (P > 1)
  float* part_m;           // fp32 [B*Hq*P]     partition reference max, log2 domain
  float* part_l;           // fp32 [B*Hq*P]     partition softmax denominators
  float scale_log2;        // softmax scale * log2(e)
  int32_t num_seqs;        // B
  int32_t num_q_heads;     // Hq
  int32_t num_kv_heads;    // Hkv
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t max_context_len;
  int32_t partition_tokens;  // T_p, multiple of 16
  int32_t num_partitions;    // P = max(1, ceil(max_context_len / T_p))
};

// Calls f(integral_constant<G>, integral_constant<D>) for the runtime (group, head_dim).
template <typename F>
hipError_t dispatch_gd(int group, int head_dim, F&& f) {
  auto with_d = [&](auto dt) -> hipError_t {
    switch (group) {
#define PDA_CASE(G) case G: return f(std::integral_constant<int, G>{}, dt);
      PDA_CASE(1) PDA_CASE(2) PDA_CASE(3) PDA_CASE(4) PDA_CASE(5) PDA_CASE(6) PDA_CASE(7) PDA_CASE(8)
      PDA_CASE(9) PDA_CASE(10) PDA_CASE(11) PDA_CASE(12) PDA_CASE(13) PDA_CASE(14) PDA_CASE(15) PDA_CASE(16)
#undef PDA_CASE
      default: return hipErrorInvalidValue;
    }
  };
  if (head_dim == 64) return with_d(std::integral_constant<int, 64>{});
  if (head_dim == 128) return with_d(std::integral_constant<int, 128>{});
  return hipErrorInvalidValue;
}

// Launchers (asynchronous; return the hipGetLastError() of the launch).
hipError_t launch_order(const StepArgs& a, hipStream_t stream);
hipError_t launch_partition(const StepArgs& a, int group, int head_dim, hipStream_t stream);
hipError_t launch_merge(const StepArgs& a, int head_dim, hipStream_t stream);

}  // namespace pda
