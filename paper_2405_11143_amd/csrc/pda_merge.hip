// Pass 2 of paged decode attention: merge per-partition softmax states.
//
// A context split into partitions p = 0..n-1 leaves, per query head, the
// partition reference maximum m_p (log2 domain), denominator l_p and
// unnormalised output O_p.  Softmax over the whole context is recovered
// exactly by rescaling every partition to the common maximum M = max_p m_p:
//   out = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p.
// The output sum runs in ascending p and the denominator in a fixed
// butterfly, so the result is reproducible.  One wavefront per (sequence,
// query head); each lane owns D/64 output columns.
#include "pda_internal.h"

namespace pda {
namespace {

// Maximum over the wavefront; every lane gets the same value.
__device__ __forceinline__ float wave_max(float x) {
  for (int o = 1; o < kWaveSize; o <<= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

// Sum over the wavefront in a fixed butterfly order; every lane gets the same bits.
__device__ __forceinline__ float wave_sum(float x) {
  for (int o = 1; o < kWaveSize; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

template <int D>
__global__ void __launch_bounds__(kWaveSize) merge_kernel(const StepArgs a) {
  constexpr int PER = D / kWaveSize;
  constexpr float kNegInf = -__builtin_huge_valf();
  const int row = blockIdx.x;  // b * Hq + h
  const int b = row / a.num_q_heads;
  const int lane = threadIdx.x;
  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  const int nparts = (L + a.partition_tokens - 1) / a.partition_tokens;
  if (nparts <= 1) return;  // pass 1 wrote the final row
  const size_t base = (size_t)row * a.num_partitions;
  const float* pm = a.part_m + base;
  const float* pl = a.part_l + base;
  const float* po = a.part_o + base * D + lane * PER;

  // Partition states are read lane-parallel (lane x holds partition p0 + x),
  // so the dependent chain is lens -> states -> outputs, whatever nparts is.
  float M = kNegInf;
  for (int p0 = 0; p0 < nparts; p0 += kWaveSize)
    if (p0 + lane < nparts) M = fmaxf(M, pm[p0 + lane]);
  M = wave_max(M);

  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  float lpart = 0.f;
  for (int p0 = 0; p0 < nparts; p0 += kWaveSize) {
    const int p = p0 + lane;
    const float wgt = p < nparts ? __builtin_amdgcn_exp2f(pm[p] - M) : 0.f;  // 2^(m_p - M)
    if (p < nparts) lpart = fmaf(wgt, pl[p], lpart);
    const int n = min(kWaveSize, nparts - p0);
    for (int x = 0; x < n; ++x) {
      const float sc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wgt), x));
      const float* src = po + (size_t)(p0 + x) * D;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = fmaf(sc, src[e], acc[e]);
    }
  }
  const float lsum = wave_sum(lpart);
  float* o = a.out + (size_t)row * D + lane * PER;
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = acc[e] / lsum;
}

}  // namespace

hipError_t launch_merge(const StepArgs& a, int head_dim, hipStream_t stream) {
  const unsigned grid = (unsigned)a.num_seqs * (unsigned)a.num_q_heads;
  if (head_dim == 64)
    hipLaunchKernelGGL(merge_kernel<64>, dim3(grid), dim3(kWaveSize), 0, stream, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL(merge_kernel<128>, dim3(grid), dim3(kWaveSize), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pda
