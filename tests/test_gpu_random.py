"""Seeded random descriptors through the C ABI against the fp64 oracle,
every output element: group sizes G = 1 ... 16 (odd ones included), head
dims 64 and 128, 1 to 70 new tokens per sequence (every kernel variant:
one tile in registers, up to 4 tiles staged, wide items of 5-8 chunks and
of 9-16 chunks on 8 wavefronts, several chunk groups), ragged contexts with
empty ones and ones shorter than the new tokens, automatic and forced
partition sizes (split contexts and the merge).  Same bar as the other
parity tests.  PDA_RANDOM_CASES sets the number of seeds (32 by default; a
wider sweep: PDA_RANDOM_CASES=2432)."""
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_common import THREADS, check
from paper_2405_11143_amd import make_problem, pda_decode, pda_plan

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def draw_case(case: int):
    r = np.random.default_rng(9000 + case)
    G = int(r.choice([1, 2, 3, 4, 5, 7, 8, 16]))
    Hkv = int(r.choice([1, 2]))
    D = int(r.choice([64, 128]))
    n = int(r.choice([1, 2, 3, 5, 8, 13, 24, 33, 48, 70]))
    B = int(r.integers(1, 7))
    pool = [0, 1, 2, n, n + 1, 17, 100, 333, 600, 1500, 2500]
    lens = [int(r.choice(pool)) for _ in range(B)]
    tp = int(r.choice([0, 0, 16, 48, 256, 1024]))
    return G, Hkv, D, n, lens, tp


@pytest.mark.parametrize("case", range(int(os.environ.get("PDA_RANDOM_CASES", "32"))))
def test_random_descriptor(dev, case):
    G, Hkv, D, n, lens, tp = draw_case(case)
    Hq = G * Hkv
    st = W.custom_structure(len(lens), Hq, Hkv, D, lens, seed=500 + case)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    plan = pda_plan(make_problem(st.B, Hq, Hkv, D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len,
                                 tp, num_query_tokens=n))
    what = f"case {case}: G={G} Hkv={Hkv} D={D} n={n} lens={lens} Tp={tp} plan={plan}"
    print(what, flush=True)
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    out = pda_decode(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len, partition_tokens=tp)
    torch.cuda.synchronize()
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table, st.context_lens,
                              st.scale, threads=THREADS)
    check(out.cpu().numpy(), ref, f"case {case}")
