// Pass 2 of paged decode attention: merge partial softmax states.
//
// A context split into partitions k = 0..n-1 leaves, per query head, the
// partition's reference maximum m_k (log2 domain), denominator l_k and
// unnormalised output O_k (a partition that the row does not reach has
// m_k = -1e30, l_k = 0, O_k = 0).  Softmax over the whole context is recovered
// exactly by rescaling every partition to the common maximum M = max_k m_k:
//   out = sum_k 2^(m_k - M) O_k / sum_k 2^(m_k - M) l_k.
// The output sum runs in ascending k and the denominator in a fixed
// butterfly, so the result is reproducible.  One wavefront per output row
// (sequence, new token, query head), 4 rows per workgroup; each lane owns
// D/64 output columns.
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

// Merge n partitions of one row: partition k (k < n) sits at state index
// first + k for k < n_pre (the group's prefix partitions) and at
// first + gap + k after them (the row's own partitions); the outputs sit at
// D times those indices in part_o.
template <int D>
__device__ __forceinline__ void merge_partitions(const StepArgs& a, size_t first, int n_pre, int gap, int n,
                                                 float* orow) {
  constexpr int PER = D / kWaveSize;
  const int lane = threadIdx.x & (kWaveSize - 1);
  auto slot = [&](int k) { return first + (size_t)k + (k >= n_pre ? gap : 0); };
  // States are read lane-parallel (lane x holds partition p0 + x), so the
  // dependent chain is states -> outputs, whatever n is.
  float M = -__builtin_huge_valf();
  for (int p0 = 0; p0 < n; p0 += kWaveSize)
    if (p0 + lane < n) M = fmaxf(M, a.part_m[slot(p0 + lane)]);
  M = wave_max(M);
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  float lpart = 0.f;
  for (int p0 = 0; p0 < n; p0 += kWaveSize) {
    const int p = p0 + lane;
    const float wgt = p < n ? __builtin_amdgcn_exp2f(a.part_m[slot(p)] - M) : 0.f;  // 2^(m_p - M)
    if (p < n) lpart = fmaf(wgt, a.part_l[slot(p)], lpart);
    const int cnt = min(kWaveSize, n - p0);
    for (int x = 0; x < cnt; ++x) {
      const float sc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wgt), x));
      const float* src = a.part_o + slot(p0 + x) * D + lane * PER;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = fmaf(sc, src[e], acc[e]);
    }
  }
  const float lsum = wave_sum(lpart);
  const bool pos = lsum > 0.f;  // 0: the row sees nothing
  if constexpr (PER == 2)
    store_nt2(orow + lane * PER, pos ? acc[0] / lsum : acc[0], pos ? acc[1] / lsum : acc[1]);
  else
    __builtin_nontemporal_store(pos ? acc[0] / lsum : acc[0], orow + lane);
}

__device__ __forceinline__ int clamped_len(const StepArgs& a, int b) {
  const int L = a.lens[b];
  return L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
}

// Output row (b, i, h), row = (b * n + i) * Hq + h, has its partial states
// at slots row * S .. row * S + S - 1 (S = slots_per_row): first the prefix
// partitions of its group, then, from slot row * S + Pp, its own partitions
// (as many as the query chunk of new token i sees after the prefix).
//
// Without groups and with at most kSpec slots per row (every split decode
// step up to 8 partitions), the row's states are loaded before its length
// is known -- they lie in the row's own slots, whatever it sees -- so that
// the length, the states and the outputs take one memory round trip instead
// of a chain of them; the arithmetic is that of merge_partitions, in the
// same order.
constexpr int kSpec = 8;

constexpr int kMergeRows = 4;  // rows (wavefronts) per workgroup

template <int D>
__global__ void __launch_bounds__(kMergeRows * kWaveSize) merge_kernel(const StepArgs a) {
  constexpr int PER = D / kWaveSize;
  const int row = blockIdx.x * kMergeRows + (threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWaveSize - 1);
  if ((size_t)row >= (size_t)a.num_seqs * a.num_query_tokens * a.num_q_heads) return;  // spare wavefronts
  const int i = (row / a.num_q_heads) % a.num_query_tokens;
  const int b = row / (a.num_q_heads * a.num_query_tokens);
  const int S = a.slots_per_row;
  const size_t first = (size_t)row * S;
  const bool spec = a.num_groups == 0 && S <= kSpec;  // uniform
  float m_s = -__builtin_huge_valf(), l_s = 0.f;
  float o_s[kSpec][PER];
  if (spec) {
    if (lane < S) {
      m_s = a.part_m[first + lane];
      l_s = a.part_l[first + lane];
    }
#pragma unroll
    for (int x = 0; x < kSpec; ++x)
#pragma unroll
      for (int e = 0; e < PER; ++e) o_s[x][e] = x < S ? a.part_o[(first + x) * D + lane * PER + e] : 0.f;
  }
  const int L = clamped_len(a, b);
  const int vis = chunk_visible(a, L, i / a.query_chunk);
  if (vis <= 0) return;  // pass 1 wrote zeros
  const int Tp = a.partition_tokens;
  const int t0 = min(seq_prefix_len(a, b), vis);
  const int n_pre = (t0 + Tp - 1) / Tp;
  const int n_own = (vis - t0 + Tp - 1) / Tp;
  if (n_pre == 0 && n_own <= 1) return;  // pass 1 wrote the final row
  float* orow = a.out + (size_t)row * D;
  if (!spec) {
    merge_partitions<D>(a, first, n_pre, a.prefix_partitions - n_pre, n_pre + n_own, orow);
    return;
  }
  const int n = n_own;  // no groups: the row's partitions are slots 0 .. n - 1 (n <= S)
  const float M = wave_max(lane < n ? fmaxf(-__builtin_huge_valf(), m_s) : -__builtin_huge_valf());
  const float wgt = lane < n ? __builtin_amdgcn_exp2f(m_s - M) : 0.f;  // 2^(m_p - M)
  const float lpart = lane < n ? fmaf(wgt, l_s, 0.f) : 0.f;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
#pragma unroll
  for (int x = 0; x < kSpec; ++x) {
    if (x < n) {
      const float sc = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, wgt), x));
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = fmaf(sc, o_s[x][e], acc[e]);
    }
  }
  const float lsum = wave_sum(lpart);
  const bool pos = lsum > 0.f;  // 0: the row sees nothing
  if constexpr (PER == 2)
    store_nt2(orow + lane * PER, pos ? acc[0] / lsum : acc[0], pos ? acc[1] / lsum : acc[1]);
  else
    __builtin_nontemporal_store(pos ? acc[0] / lsum : acc[0], orow + lane);
}

}  // namespace

hipError_t launch_merge(const StepArgs& a, int head_dim, hipStream_t stream) {
  const unsigned rows = (unsigned)a.num_seqs * (unsigned)a.num_query_tokens * (unsigned)a.num_q_heads;
  const unsigned grid = (rows + kMergeRows - 1) / kMergeRows;
  if (head_dim == 64)
    hipLaunchKernelGGL(merge_kernel<64>, dim3(grid), dim3(kMergeRows * kWaveSize), 0, stream, a);
  else if (head_dim == 128)
    hipLaunchKernelGGL(merge_kernel<128>, dim3(grid), dim3(kMergeRows * kWaveSize), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pda
