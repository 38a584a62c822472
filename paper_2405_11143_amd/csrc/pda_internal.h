// Internal interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pda {

constexpr int kBlockTokens = 16;  // tokens per KV-cache block
constexpr int kWaveSize = 64;     // CDNA wavefront
constexpr int kWaves = 4;         // wavefronts per partition workgroup
constexpr int kMaxGroup = 16;     // query heads per KV head handled by one MFMA row tile

// Kernel arguments for one decode step (passed by value).
struct StepArgs {
  const uint16_t* q;       // bf16 [B][Hq][D]
  const uint16_t* k;       // bf16 [num_blocks][Hkv][16][D]
  const uint16_t* v;       // bf16 [num_blocks][Hkv][16][D]
  const int32_t* table;    // int32 [B][max_blocks_per_seq]
  const int32_t* lens;     // int32 [B]
  float* out;              // fp32 [B][Hq][D]
  float* part_o;           // fp32 [B][Hq][P][D]   unnormalised partition outputs
  float* part_m;           // fp32 [B][Hq][P]      partition max, log2 domain
  float* part_l;           // fp32 [B][Hq][P]      partition softmax denominators
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

// Launchers (asynchronous; return the hipGetLastError() of the launch).
hipError_t launch_partition(const StepArgs& a, int group, int head_dim, hipStream_t stream);
hipError_t launch_merge(const StepArgs& a, int head_dim, hipStream_t stream);

}  // namespace pda
