// Work order of pass 1: every item, largest first.
//
// Pass 1 launches one workgroup per item and the GPU starts workgroups in
// index order, so the order of the items is the schedule.  Contexts are
// ragged, and the last partition of each context is shorter than the others;
// with the items in their natural order the short and the long ones are
// mixed and the step ends with a tail of long items on a half-empty GPU.
// Sorting the items by size, largest first (a greedy longest-processing-
// time schedule), leaves only short items for the end: on MI355X it raised
// pass 1 by 3-10% on the Llama-3-shaped decode steps.  Items of size zero
// (partitions past what a context needs) come last and exit at once.
//
// The items come in pairs of equal size: a regular pair (sequence, partition)
// stands for its items of every KV head and group of query chunks, a prefix pair
// (shared-prefix group, prefix partition, row group of members) for its items
// of every KV head (with groups a work item holds all query chunks of a
// sequence, so both kinds of pairs hold Hkv items).
// One workgroup counting-sorts the pairs by size in blocks (classes capped
// at kOrderBuckets - 1 blocks) with LDS atomics, then writes the items of
// each pair.  The order within a size class depends on atomic timing; no
// result does -- every item computes the same values whichever workgroup
// runs it.
//
// With shared-prefix groups the same workgroup first writes, for every
// sequence, the prefix length of its group (0 outside any group) into the
// workspace; the sizes of the regular pairs, pass 1 and the merge read it.
#include "pda_internal.h"

namespace pda {
namespace {

__global__ void __launch_bounds__(kOrderThreads) order_kernel(const StepArgs a) {
  __shared__ int s_count[kOrderBuckets];  // pairs per size class, then the next free position
  const int tid = threadIdx.x;
  const int B = a.num_seqs;
  const int P = a.num_partitions;
  const int Pp = a.prefix_partitions;
  const int RG = a.prefix_row_groups;
  const int Tp = a.partition_tokens;
  const int regular_pairs = B * P;
  const int pairs = regular_pairs + a.num_groups * Pp * RG;

  if (a.seq_prefix) {  // per-sequence prefix length (group contents clamped: device data)
    for (int b = tid; b < B; b += kOrderThreads) a.seq_prefix[b] = 0;
    __threadfence_block();
    __syncthreads();
    for (int grp = tid; grp < a.num_groups; grp += kOrderThreads) {
      const int first = min(max(a.group_start[grp], 0), B);
      const int last = min(min(a.group_start[grp + 1], B), first + a.max_group_size);
      int plen = a.group_prefix_len[grp];
      plen = plen < 0 ? 0 : (plen > a.max_prefix_len ? a.max_prefix_len : plen) / kBlockTokens * kBlockTokens;
      for (int b = first; b < last; ++b) a.seq_prefix[b] = plen;
    }
    __threadfence_block();
    __syncthreads();
  }

  // size class of pair idx: kOrderBuckets - 1 - blocks, so larger first
  auto bucket = [&](int idx) {
    int tok;
    if (idx < regular_pairs) {
      const int b = idx % B;
      const int p = idx / B;
      int L = a.lens[b];
      L = L < 0 ? 0 : (L > a.max_context_len ? a.max_context_len : L);
      const int t0 = min(seq_prefix_len(a, b), L);
      tok = max(0, min(L, t0 + (p + 1) * Tp) - (t0 + p * Tp));
    } else {  // prefix pair idx - regular_pairs = (grp * Pp + pp) * RG + rg
      const int x = idx - regular_pairs;
      const int rg = x % RG;
      const int pp = (x / RG) % Pp;
      const int grp = x / (RG * Pp);
      const int first = min(max(a.group_start[grp], 0), B);
      const int members = min(min(a.group_start[grp + 1], B) - first, a.max_group_size);
      int plen = a.group_prefix_len[grp];
      plen = plen < 0 ? 0 : (plen > a.max_prefix_len ? a.max_prefix_len : plen);
      tok = (int64_t)rg * a.members_per_row_group < members ? max(0, min(plen, (pp + 1) * Tp) - pp * Tp) : 0;
    }
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
  // Workgroups go to the 8 XCDs round-robin by slot, and each XCD has its own
  // L2.  Two placements of the HC items of sorted pair pos:
  //  * Hkv a multiple of 8: item (KV head g, chunk group cg) goes to slot
  //    pos HC + cg Hkv + g, i.e. to XCD g % 8.  Every KV head stays on one
  //    XCD, so sequences whose block tables share blocks (parallel samples of
  //    a prompt) meet in its L2, and so do the chunk groups of one (sequence,
  //    partition, KV head), which start within HC slots of each other.
  //  * otherwise the pairs are taken in octets: the octet holding pair pos
  //    starts at pair pos - r (r = pos % 8) and has c <= 8 pairs, and item x
  //    < HC of pair pos goes to slot (pos - r) HC + x c + r, so (with c = 8)
  //    every item of a pair, among them its chunk groups, runs on one XCD.
  // Prefix pairs (which come with groups only, where NCG = 1 and HC = Hkv) are placed
  // alike.  Pair idx holds items idx HC .. idx HC + HC - 1 (a regular pair
  // (p, b) has idx = p B + b, and the prefix items follow the regular ones),
  // item idx HC + g NCG + cg being KV head g, chunk group cg.
  const int Hkv = a.num_kv_heads;
  const int NCG = a.num_chunk_groups;
  const int HC = Hkv * NCG;
  for (int idx = tid; idx < pairs; idx += kOrderThreads) {
    const int pos = atomicAdd(&s_count[bucket(idx)], 1);
    if (Hkv % 8 == 0) {
      for (int x = 0; x < HC; ++x) a.order[(size_t)pos * HC + x] = idx * HC + (x % Hkv) * NCG + x / Hkv;
    } else {
      const int r = pos % 8;
      const int c = min(8, pairs - (pos - r));
      const size_t base = (size_t)(pos - r) * HC + r;
      for (int x = 0; x < HC; ++x) a.order[base + (size_t)x * c] = idx * HC + x;
    }
  }
}

}  // namespace

hipError_t launch_order(const StepArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pda
