/*
 * pda_ceiling.h -- HBM read ceilings for the decode step's memory traffic
 * (a measurement aid of libpda.so, not part of the attention operation).
 *
 * The decode step is bound by HBM reads: it streams every key and value row
 * of every context once (the paged KV cache of the rollout step, Section 3.2,
 * "Accelerated CoT Inference with vLLM").  These two kernels read the same
 * bytes with no arithmetic on them, so that the attention kernel's rate can
 * be set against what the chip delivers for the same access pattern:
 *
 *  - pda_gather_ceiling reads the K and V tiles (16 tokens x head_dim bf16
 *    each, in the k_cache / v_cache layouts of pda.h) of a list of physical
 *    block ids for every KV head, with the 16-byte non-temporal buffer loads
 *    the attention kernel uses (1 KiB of contiguous memory per K load
 *    instruction, four 256-byte V rows per V load at head_dim 128).  Unit u
 *    of the num_ids * num_kv_heads units is KV head u / num_ids of block
 *    block_ids[u % num_ids]; the units are split into `workgroups` equal
 *    contiguous ranges, one per workgroup of 4 wavefronts, and each wavefront
 *    takes a contiguous quarter of its range, two tiles in flight.  A block id
 *    outside [0, num_blocks) is skipped (nothing is read for it).
 *  - pda_stream_ceiling reads a contiguous buffer of `bytes` bytes (a
 *    multiple of 16, 16-byte aligned) with 16-byte non-temporal loads,
 *    grid-strided over `workgroups` workgroups of 256 threads.
 *
 * Each wavefront XORs what it read and writes one uint32 to
 * sink[4 * workgroup + wavefront] (sink: device uint32 [4 * workgroups]), so
 * no load can be dropped.  All pointers are device pointers owned by the
 * caller; nothing is allocated.  Returns PDA_OK, PDA_ERR_NULL,
 * PDA_ERR_SHAPE (negative or zero sizes, head_dim not 64/128, bytes not a
 * multiple of 16), PDA_ERR_ALIGNMENT (pools or buffer not 16-byte aligned) or
 * PDA_ERR_HIP (the launch failed); work is enqueued on `stream`.
 */
#ifndef PDA_CEILING_H
#define PDA_CEILING_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

int pda_gather_ceiling(int32_t num_kv_heads, int32_t head_dim, int32_t num_blocks, const void *k_cache,
                       const void *v_cache, const int32_t *block_ids, int32_t num_ids, int32_t workgroups,
                       uint32_t *sink, hipStream_t stream);

int pda_stream_ceiling(const void *buf, size_t bytes, int32_t workgroups, uint32_t *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PDA_CEILING_H */
