"""pda_decode_noalloc (the decode step with its workspace in the library's
static scratch, for callers that cannot allocate) against pda_decode, through
the C ABI: two calls in a row, the second on a smaller problem, each checked
bitwise and to the parity bar against pda_decode's output on the same inputs.
The first call leaves partial softmax states of a split step in the scratch;
the second must not depend on them."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_common import THREADS, check
from paper_2405_11143_amd import (PdaError, make_problem, pda_decode, pda_decode_noalloc, pda_plan,
                                  pda_workspace_bytes)
from paper_2405_11143_amd.pda import PDA_ERR_SCRATCH, PDA_NOALLOC_SCRATCH_BYTES

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def case(dev, lens, Hq, Hkv, D, n, tp, seed):
    st = W.custom_structure(len(lens), Hq, Hkv, D, lens, seed=seed)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev) if n > 1 else W.fill_values(st, dev, fill="nan")[0]
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    prob = make_problem(st.B, Hq, Hkv, D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len, tp,
                        num_query_tokens=n)
    return st, q, k, v, bt, ln, prob


def test_noalloc_matches_decode_two_calls(dev):
    cases = [  # (lens, Hq, Hkv, D, n, partition_tokens, seed): the first large and split, the second smaller
        ([4096, 3000, 1, 17, 2049, 4095, 700, 1500] * 8, 32, 8, 128, 1, 256, 501),
        ([1, 33, 700, 64, 65, 300], 8, 2, 64, 3, 64, 502),
    ]
    sizes = []
    for lens, Hq, Hkv, D, n, tp, seed in cases:
        st, q, k, v, bt, ln, prob = case(dev, lens, Hq, Hkv, D, n, tp, seed)
        plan = pda_plan(prob)
        sizes.append(plan["workspace_bytes"])
        assert plan["num_partitions"] > 1 and plan["workspace_bytes"] <= PDA_NOALLOC_SCRATCH_BYTES
        ref_out = pda_decode(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len, partition_tokens=tp)
        got = pda_decode_noalloc(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len,
                                 partition_tokens=tp)
        again = pda_decode_noalloc(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len,
                                   partition_tokens=tp)
        torch.cuda.synchronize()
        a, b, c = ref_out.cpu().numpy(), got.cpu().numpy(), again.cpu().numpy()
        print(f"noalloc B={st.B} Hq={Hq} Hkv={Hkv} D={D} n={n} Tp={tp}: plan {plan}", flush=True)
        assert np.array_equal(a, b), "pda_decode_noalloc differs from pda_decode"
        assert np.array_equal(b, c), "two pda_decode_noalloc calls differ"
        check(b, a.astype(np.float64), f"noalloc vs pda_decode n={n}")
        qb = W.bf16_bits(q)
        ref = (oracle.decode_multi if n > 1 else oracle.decode)(qb, W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                                                                 st.context_lens, st.scale, threads=THREADS)
        check(b, ref, f"noalloc vs oracle n={n}")
    assert sizes[1] < sizes[0]


def test_noalloc_rejects_a_step_beyond_the_scratch(dev):
    # 256 sequences x 64 new tokens x 32 heads in 16-token partitions of 4096-token contexts
    prob = make_problem(256, 32, 8, 128, 70000, 256, 4096, 16, num_query_tokens=64)
    assert pda_workspace_bytes(prob) > PDA_NOALLOC_SCRATCH_BYTES
    st = W.custom_structure(2, 32, 8, 128, [64, 64], seed=3)
    _, k, v = W.fill_values(st, dev, fill="zero")
    q = torch.zeros((256, 64, 32, 128), dtype=torch.bfloat16, device=dev)
    bt = torch.zeros((256, 256), dtype=torch.int32, device=dev)
    ln = torch.zeros((256,), dtype=torch.int32, device=dev)
    with pytest.raises(PdaError) as e:
        pda_decode_noalloc(q, k, v, bt, ln, 0.1, max_context_len=4096, partition_tokens=16)
    assert e.value.status == PDA_ERR_SCRATCH
