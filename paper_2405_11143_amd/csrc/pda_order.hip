// Work order of pass 1: the (partition, sequence, KV head, query chunk)
// items, largest partition first.
//
// Pass 1 launches one workgroup per item and the GPU starts workgroups in
// index order, so the order of the items is the schedule.  Contexts are
// ragged, and the last partition of each context is shorter than the others;
// with the items in their natural order the short and the long ones are
// mixed and the step ends with a tail of long items on a half-empty GPU.
// Sorting the items by size, largest first (a greedy longest-processing-
// time schedule), leaves only short items for the end: on MI355X it raised
// pass 1 by 3-10% on the Llama-3-shaped decode steps.  Items of size zero
// (partitions past a context's end) come last and exit at once.
//
// One workgroup does a counting sort of the B*P (sequence, partition) pairs
// by size in blocks (classes capped at kOrderBuckets - 1 blocks) with LDS
// atomics, then writes the items of each pair (one per KV head and query
// chunk).  The order within a size
// class depends on atomic timing; no result does -- every item computes the
// same values whichever workgroup runs it.
#include "pda_internal.h"

namespace pda {
namespace {

__global__ void __launch_bounds__(kOrderThreads) order_kernel(const StepArgs a) {
  __shared__ int s_count[kOrderBuckets];  // pairs per size class, then the next free position
  const int tid = threadIdx.x;
  const int B = a.num_seqs;
  const int P = a.num_partitions;
  const int Tp = a.partition_tokens;
  const int pairs = B * P;
  // size class of pair (b, p): kOrderBuckets - 1 - blocks, so larger first
  auto bucket = [&](int idx) {
    const int b = idx % B;
    const int p = idx / B;
    int L = a.lens[b];
    L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
    const int tok = max(0, min(L, (p + 1) * Tp) - p * Tp);
    const int blocks = min((tok + kBlockTokens - 1) / kBlockTokens, kOrderBuckets - 1);
    return kOrderBuckets - 1 - blocks;
  };
  for (int i = tid; i < kOrderBuckets; i += kOrderThreads) s_count[i] = 0;
  __syncthreads();
  for (int idx = tid; idx < pairs; idx += kOrderThreads) atomicAdd(&s_count[bucket(idx)], 1);
  __syncthreads();
  if (tid < kWaveSize) {  // exclusive scan of the class counts by one wavefront
    constexpr int PER = kOrderBuckets / kWaveSize;
    int v[PER], sum = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      v[e] = s_count[tid * PER + e];
      sum += v[e];
    }
    int inc = sum;
    for (int o = 1; o < kWaveSize; o <<= 1) {
      const int t = __shfl_up(inc, o);
      if (tid >= o) inc += t;
    }
    int run = inc - sum;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      s_count[tid * PER + e] = run;
      run += v[e];
    }
  }
  __syncthreads();
  const int HC = a.num_kv_heads * a.num_query_chunks;  // items per pair
  for (int idx = tid; idx < pairs; idx += kOrderThreads) {
    const int pos = atomicAdd(&s_count[bucket(idx)], 1);
    const int b = idx % B;
    const int p = idx / B;
    for (int g = 0; g < HC; ++g) a.order[(size_t)pos * HC + g] = (p * B + b) * HC + g;
  }
}

}  // namespace

hipError_t launch_order(const StepArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pda
