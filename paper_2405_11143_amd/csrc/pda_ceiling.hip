// HBM read ceilings of the decode step's traffic (include/pda_ceiling.h):
// the K/V tiles a step reads, gathered with the attention kernel's loads but
// without its arithmetic, and a plain contiguous stream.  A measurement aid:
// the attention kernel's bytes per second over the gather's says how much of
// what the chip delivers for this access pattern the step uses.
#include "pda.h"
#include "pda_ceiling.h"
#include "pda_wave.h"

namespace pda {
namespace {

constexpr int kCeilThreads = kWaves * kWaveSize;

__device__ __forceinline__ unsigned fold(uint4 x) { return x.x ^ x.y ^ x.z ^ x.w; }

// One wavefront's XOR of everything it read, written by its lane 0.
__device__ __forceinline__ void publish_xor(unsigned acc, uint32_t* sink) {
  for (int o = 1; o < kWaveSize; o <<= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & (kWaveSize - 1)) == 0) sink[blockIdx.x * kWaves + (threadIdx.x >> 6)] = acc;
}

template <int D>
__global__ void __launch_bounds__(kCeilThreads) gather_kernel(const char* k, const char* v, const int32_t* ids,
                                                              int n_ids, int Hkv, int num_blocks, int64_t per_wg,
                                                              uint32_t* sink) {
  constexpr int TB = kBlockTokens * D * 2;  // bytes of one K or V tile
  constexpr int NC = D / 32;                // K loads per lane and tile (1 KiB per instruction)
  constexpr int RB = D * 2;                 // bytes of one V row
  const int lane = threadIdx.x & (kWaveSize - 1);
  const int w = threadIdx.x >> 6;
  const int64_t total = (int64_t)n_ids * Hkv;
  const int64_t u0 = min(total, (int64_t)blockIdx.x * per_wg);
  const int64_t u1 = min(total, u0 + per_wg);
  const int64_t per_wave = (u1 - u0 + kWaves - 1) / kWaves;
  const int64_t a0 = min(u1, u0 + w * per_wave);
  const int64_t a1 = min(u1, a0 + per_wave);
  const size_t block_bytes = (size_t)Hkv * TB;
  const int k_off = 16 * lane;
  const int v_off = 4 * (lane >> 4) * RB + 16 * ((lane & 15) % (D / 8));
  unsigned acc = 0;
  uint4 kr[2][NC], vr[2][4];
  // issue the loads of unit u into buffer s (a unit past the range, or with a
  // block id outside the pool, gets zero-length descriptors: nothing is read)
  auto issue = [&](int64_t u, int s) {
    const bool in = u < a1;
    const int g = in ? (int)(u / n_ids) : 0;
    int id = in ? ids[u % n_ids] : 0;
    const bool ok = in && (unsigned)id < (unsigned)num_blocks;
    id = ok ? id : 0;
    const size_t off = (size_t)id * block_bytes + (size_t)g * TB;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(k + off, ok ? TB : 0);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(v + off, ok ? TB : 0);
#pragma unroll
    for (int c = 0; c < NC; ++c) kr[s][c] = load_stream(rk, k_off + c * 1024);
#pragma unroll
    for (int e = 0; e < 4; ++e) vr[s][e] = load_stream(rv, v_off + e * RB);
  };
  auto consume = [&](int s) {
#pragma unroll
    for (int c = 0; c < NC; ++c) acc ^= fold(kr[s][c]);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc ^= fold(vr[s][e]);
  };
  if (a0 < a1) issue(a0, 0);
  for (int64_t u = a0; u < a1; u += 2) {
    issue(u + 1, 1);
    __builtin_amdgcn_sched_barrier(0);
    consume(0);
    if (u + 1 >= a1) break;
    issue(u + 2, 0);
    __builtin_amdgcn_sched_barrier(0);
    consume(1);
  }
  publish_xor(acc, sink);
}

__global__ void __launch_bounds__(kCeilThreads) stream_kernel(const uint4* buf, int64_t n16, uint32_t* sink) {
  typedef unsigned u4 __attribute__((ext_vector_type(4)));
  const int64_t stride = (int64_t)gridDim.x * kCeilThreads;
  unsigned acc = 0;
  int64_t i = (int64_t)blockIdx.x * kCeilThreads + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    u4 x[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) x[r] = __builtin_nontemporal_load(reinterpret_cast<const u4*>(buf + i + r * stride));
#pragma unroll
    for (int r = 0; r < 4; ++r) acc ^= x[r][0] ^ x[r][1] ^ x[r][2] ^ x[r][3];
  }
  for (; i < n16; i += stride) {
    const u4 x = __builtin_nontemporal_load(reinterpret_cast<const u4*>(buf + i));
    acc ^= x[0] ^ x[1] ^ x[2] ^ x[3];
  }
  publish_xor(acc, sink);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace
}  // namespace pda

extern "C" {

int pda_gather_ceiling(int32_t num_kv_heads, int32_t head_dim, int32_t num_blocks, const void* k_cache,
                       const void* v_cache, const int32_t* block_ids, int32_t num_ids, int32_t workgroups,
                       uint32_t* sink, hipStream_t stream) {
  if (num_kv_heads < 1 || num_blocks < 1 || num_ids < 0 || workgroups < 1) return PDA_ERR_SHAPE;
  if (head_dim != 64 && head_dim != 128) return PDA_ERR_SHAPE;
  if (!k_cache || !v_cache || !sink || (num_ids > 0 && !block_ids)) return PDA_ERR_NULL;
  if (!pda::aligned16(k_cache) || !pda::aligned16(v_cache)) return PDA_ERR_ALIGNMENT;
  const int64_t total = (int64_t)num_ids * num_kv_heads;
  const int64_t per_wg = (total + workgroups - 1) / workgroups;
  const char* k = static_cast<const char*>(k_cache);
  const char* v = static_cast<const char*>(v_cache);
  if (head_dim == 64)
    hipLaunchKernelGGL(pda::gather_kernel<64>, dim3(workgroups), dim3(pda::kCeilThreads), 0, stream, k, v,
                       block_ids, num_ids, num_kv_heads, num_blocks, per_wg, sink);
  else
    hipLaunchKernelGGL(pda::gather_kernel<128>, dim3(workgroups), dim3(pda::kCeilThreads), 0, stream, k, v,
                       block_ids, num_ids, num_kv_heads, num_blocks, per_wg, sink);
  return hipGetLastError() == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

int pda_stream_ceiling(const void* buf, size_t bytes, int32_t workgroups, uint32_t* sink, hipStream_t stream) {
  if (bytes == 0 || bytes % 16 != 0 || workgroups < 1) return PDA_ERR_SHAPE;
  if (!buf || !sink) return PDA_ERR_NULL;
  if (!pda::aligned16(buf)) return PDA_ERR_ALIGNMENT;
  hipLaunchKernelGGL(pda::stream_kernel, dim3(workgroups), dim3(pda::kCeilThreads), 0, stream,
                     static_cast<const uint4*>(buf), (int64_t)(bytes / 16), sink);
  return hipGetLastError() == hipSuccess ? PDA_OK : PDA_ERR_HIP;
}

}  // extern "C"
