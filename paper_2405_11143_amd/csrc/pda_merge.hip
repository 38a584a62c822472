// Pass 2 of paged decode attention: merge per-partition softmax states.
//
// A context split into partitions p = 0..n-1 leaves, per query head, the
// partition maximum m_p (log2 domain), denominator l_p and unnormalised
// output O_p.  Softmax over the whole context is recovered exactly by
// rescaling every partition to the common maximum M = max_p m_p:
//   out = sum_p 2^(m_p - M) O_p / sum_p 2^(m_p - M) l_p.
// The sum runs in ascending p, so the result is reproducible.  One
// wavefront per (sequence, query head); each lane owns D/64 output columns.
#include "pda_internal.h"

namespace pda {
namespace {

template <int D>
__global__ void __launch_bounds__(kWaveSize) merge_kernel(const StepArgs a) {
  constexpr int PER = D / kWaveSize;
  constexpr float kNegInf = -__builtin_huge_valf();
  const int row = blockIdx.x;  // b * Hq + h
  const int b = row / a.num_q_heads;
  int L = a.lens[b];
  L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
  const int nparts = (L + a.partition_tokens - 1) / a.partition_tokens;
  if (nparts <= 1) return;  // pass 1 wrote the final row
  const size_t base = (size_t)row * a.num_partitions;
  const float* pm = a.part_m + base;
  const float* pl = a.part_l + base;
  const float* po = a.part_o + base * D + threadIdx.x * PER;

  float M = kNegInf;
  for (int p = 0; p < nparts; ++p) M = fmaxf(M, pm[p]);
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  float lsum = 0.f;
  for (int p = 0; p < nparts; ++p) {
    const float sc = __builtin_amdgcn_exp2f(pm[p] - M);
    lsum = fmaf(sc, pl[p], lsum);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = fmaf(sc, po[(size_t)p * D + e], acc[e]);
  }
  float* o = a.out + (size_t)row * D + threadIdx.x * PER;
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
