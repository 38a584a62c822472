"""Paged decode attention for AMD MI355X (gfx950).

The rollout hot path of RLHF/RLVR training (arXiv 2405.11143): one decode
step's attention of every sequence's new query token(s) over its paged KV
cache, with grouped-query heads (also with a shared prompt prefix attended once
for all the prompt's samples), the KV-cache append before it, and the step
captured as a HIP graph, and the sampled tokens' log-probabilities and
entropies -- hand-written HIP kernels behind a C ABI
(include/pda.h).  This package is the thin Python binding of that ABI.
"""
from .pda import (EXPORTED, LIB_PATH, BoundCall, ModelStepGraph, PdaError, StepGraph, bind_append_kv, bind_decode, bind_token_logprobs,  # noqa: F401
                  load_library, make_prefix_groups,
                  make_problem, pda_append_kv, pda_decode, pda_decode_shared_prefix, pda_merge_partitions,
                  pda_partition_attention, pda_plan, pda_plan_info, pda_plan_shared_prefix, pda_prefix_groups,
                  pda_problem, pda_status_string, pda_token_logprobs, pda_validate_host, pda_workspace_bytes,
                  pda_work_order, pda_decode_reusing_order, pda_decode_noalloc, bind_decode_noalloc,
                  bind_gather_ceiling, bind_stream_ceiling,
                  pda_decode_append, bind_decode_append)
