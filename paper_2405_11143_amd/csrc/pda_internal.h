// Internal interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

namespace pda {

constexpr int kBlockTokens = 16;     // tokens per KV-cache block
constexpr int kWaveSize = 64;        // CDNA wavefront
constexpr int kWaves = 4;            // wavefronts per workgroup
constexpr int kMaxGroup = 16;        // query heads per KV head handled by one MFMA row tile
constexpr int kMaxStreamSeqs = 8192; // stream schedule keeps per-sequence block prefix sums in LDS

// Kernel arguments for one decode step (passed by value).
struct StepArgs {
  const uint16_t* q;       // bf16 [B][Hq][D]
  const uint16_t* k;       // bf16 [num_blocks][Hkv][D/8][16][8]
  const uint16_t* v;       // bf16 [num_blocks][Hkv][16][D]
  const int32_t* table;    // int32 [B][max_blocks_per_seq]
  const int32_t* lens;     // int32 [B]
  float* out;              // fp32 [B][Hq][D]
  // Partial softmax states.  Partition schedule: slot = (b*Hq + h)*P + p, one
  // head per slot.  Stream schedule: slot = unit + wave (unit = b*Hkv + g),
  // G heads per slot.
  float* part_o;           // fp32 [slots][D]  unnormalised outputs
  float* part_m;           // fp32 [slots]     reference max, log2 domain
  float* part_l;           // fp32 [slots]     softmax denominators
  int32_t* unit_info;      // stream schedule: int32 [B*Hkv][2] = (first wave, segments)
  float scale_log2;        // softmax scale * log2(e)
  int32_t num_seqs;        // B
  int32_t num_q_heads;     // Hq
  int32_t num_kv_heads;    // Hkv
  int32_t num_blocks;
  int32_t max_blocks_per_seq;
  int32_t max_context_len;
  int32_t partition_tokens;  // partition schedule: T_p, multiple of 16
  int32_t num_partitions;    // partition schedule: P = max(1, ceil(max_context_len / T_p))
  int32_t num_workers;       // stream schedule: wavefronts sharing the work (multiple of kWaves)
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
hipError_t launch_partition(const StepArgs& a, int group, int head_dim, hipStream_t stream);
hipError_t launch_stream(const StepArgs& a, int group, int head_dim, hipStream_t stream);
hipError_t launch_merge_partition(const StepArgs& a, int head_dim, hipStream_t stream);
hipError_t launch_merge_stream(const StepArgs& a, int group, int head_dim, hipStream_t stream);

// Stream schedule: dynamic LDS bytes of pass 1 and the number of its
// workgroups one compute unit holds at once (HIP occupancy query).
size_t stream_lds_bytes(int num_seqs);
hipError_t stream_blocks_per_cu(int group, int head_dim, int num_seqs, int* blocks);

}  // namespace pda
