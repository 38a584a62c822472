"""GPU parity of the shared-prefix decode step (parallel sampling: the
samples of one prompt share its KV blocks, Section 3.2) through the C ABI.

The operation is the same attention as the decode step, only scheduled so
that each group's prefix is attended once for all members; the fp64 oracle
is the plain decode definition.  Bar: max-abs <= 8e-3, mean-abs <= 1e-3 over
every compared element; bitwise run-to-run and under block shuffles.
PDA_RANDOM_GROUP_CASES sets the seeds of the two random-group tests (24 and
16 by default; a wider sweep: PDA_RANDOM_GROUP_CASES=624).
"""
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_common import THREADS, check
from paper_2405_11143_amd import make_prefix_groups, make_problem, pda_decode_shared_prefix, pda_plan_shared_prefix

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def run(st, q, k, v, dev, partition_tokens=0, max_group_size=None, max_prefix_len=None):
    gs = torch.from_numpy(st.group_start).to(dev)
    gp = torch.from_numpy(st.group_prefix_len).to(dev)
    sizes = np.diff(st.group_start)
    out = pda_decode_shared_prefix(
        q, k, v, torch.from_numpy(st.block_table).to(dev), torch.from_numpy(st.context_lens).to(dev), st.scale,
        gs, gp, max_context_len=st.max_context_len,
        max_group_size=int(sizes.max(initial=1)) if max_group_size is None else max_group_size,
        max_prefix_len=int(st.group_prefix_len.max(initial=0)) if max_prefix_len is None else max_prefix_len,
        partition_tokens=partition_tokens)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def reference(st, q, k, v):
    return oracle.decode(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table, st.context_lens,
                         st.scale, threads=THREADS)




GROUPS = [
    (1024, [1024, 1025, 1100, 3000, 1040, 2047, 1500, 4096]),  # 8 samples; one with an empty suffix
    (32, [33, 40, 100]),
    (0, [5, 300]),                                              # a group without a prefix
    (4096, [4100, 5000]),                                       # a prefix of several partitions
    (16, [16]),                                                 # one member, prefix = whole context
]


@pytest.mark.parametrize("Hq,Hkv,D", [(32, 8, 128), (8, 1, 128), (16, 8, 64), (4, 4, 128)], ids=str)
@pytest.mark.parametrize("partition_tokens", [0, 64, 1024])
def test_groups_and_loners(dev, Hq, Hkv, D, partition_tokens):
    st = W.custom_shared_structure(Hq, Hkv, D, GROUPS, loner_lens=[1, 700, 0, 2049], seed=Hq + D)
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev, partition_tokens)
    assert np.all(got[st.B - 2] == 0)  # the empty loner
    check(got, reference(st, q, k, v), f"groups Hq={Hq} Hkv={Hkv} D={D} Tp={partition_tokens}")


@pytest.mark.parametrize("G,members", [(4, 16), (8, 8), (1, 64), (16, 4), (3, 5)])
def test_largest_groups(dev, G, members):
    """Groups that fill one prefix item: members x G = 64 (or just below)
    query rows, i.e. 4 tiles of 16 rows in one work item."""
    r = np.random.default_rng(members)
    lens = [int(x) for x in 256 + r.integers(0, 600, members)]
    st = W.custom_shared_structure(2 * G, 2, 128, [(256, lens)], loner_lens=[300], seed=G)
    q, k, v = W.fill_values(st, dev, fill="nan")
    check(run(st, q, k, v, dev), reference(st, q, k, v), f"G={G} members={members}")


@pytest.mark.parametrize("G,Hkv,members,n", [
    (4, 2, 24, 1),   # 16 + 8 members
    (8, 1, 16, 1),   # the 70B TP=8 shard's G: 8 + 8
    (7, 4, 16, 1),   # the R1-Qwen-7B heads (28 / 4): 9 + 7
    (1, 1, 200, 1),  # 64 + 64 + 64 + 8
    (16, 1, 9, 1),   # 4 + 4 + 1
    (4, 2, 8, 4),    # 4 draft tokens over 8 samples: 4 + 4
    (3, 2, 3, 21),   # 63 rows per member, items of 6 query chunks (the wide variant): 1 + 1 + 1
    (9, 1, 2, 7),    # 63 rows per member, 7 query chunks: 1 + 1
    (6, 2, 4, 10),   # 60 rows per member: 1 + 1 + 1 + 1
], ids=str)
def test_groups_beyond_one_item(dev, G, Hkv, members, n):
    """Groups whose rows exceed the 64 of one prefix item: the members are
    taken 64 / (n G) at a time, each row group reading the prefix once.  One
    member's new tokens start inside the prefix; sequences in no group; every
    element against the oracle, and bitwise run to run."""
    r = np.random.default_rng(members * 31 + G)
    lens = [256 + n + int(x) for x in r.integers(0, 700, members)]
    lens[members // 2] = 256 + max(n - 2, 0)  # new tokens reaching back into the prefix (n > 2)
    groups = [(256, lens), (32, [40, 32 + n][:max(1, members // 4)])]
    st = W.custom_shared_structure(G * Hkv, Hkv, 128, groups, loner_lens=[n + 5, 0], seed=G + members)
    q, k, v = W.fill_values(st, dev, fill="nan")
    if n > 1:
        q = W.fill_multi_q(st, n, dev)
    got = run(st, q, k, v, dev)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table, st.context_lens,
                              st.scale, threads=THREADS) if n > 1 else reference(st, q, k, v)
    check(got, ref, f"G={G} Hkv={Hkv} members={members} n={n}")
    assert np.array_equal(got, run(st, q, k, v, dev)), "run-to-run"
    # a host bound above the contents: more (empty) row groups, same result
    np.testing.assert_allclose(run(st, q, k, v, dev, max_group_size=4 * members), got, rtol=0, atol=1e-5)


def test_bitwise_run_to_run_and_shuffle(dev):
    st = W.custom_shared_structure(32, 8, 128, GROUPS, loner_lens=[900], seed=5)
    q, k, v = W.fill_values(st, dev, fill="nan")
    base = run(st, q, k, v, dev)
    assert np.array_equal(base, run(st, q, k, v, dev)), "run-to-run"
    st2, k2, v2 = W.permute_pool(st, k, v, seed=2)
    assert np.array_equal(base, run(st2, q, k2, v2, dev)), "block shuffle"
    _, kz, vz = W.fill_values(st, dev, fill="zero")
    assert np.array_equal(base, run(st, q, kz, vz, dev)), "NaN poison vs zero fill"


def test_host_bounds_above_contents(dev):
    """Bounds larger than the contents (more room per group, a longer prefix
    bound) give the same result."""
    st = W.custom_shared_structure(32, 8, 128, GROUPS[:3], loner_lens=[50], seed=6)
    q, k, v = W.fill_values(st, dev, fill="nan")
    a = run(st, q, k, v, dev)
    b = run(st, q, k, v, dev, max_group_size=16, max_prefix_len=2048)
    check(b, reference(st, q, k, v), "larger host bounds")
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-5)


def test_members_past_the_host_bound(dev):
    """A group with more members than max_group_size: the members past the
    bound attend as sequences in no group (their own items cover the whole
    context), so the step still equals the plain decode step."""
    st = W.custom_shared_structure(32, 8, 128, [(512, [600, 700, 512, 900, 1300, 520, 800, 640, 2000, 515])],
                                   loner_lens=[77], seed=9)
    q, k, v = W.fill_values(st, dev, fill="nan")
    check(run(st, q, k, v, dev, max_group_size=4), reference(st, q, k, v), "10 members, max_group_size 4")


def test_shared_prefix_config_full_size(dev):
    """The 32 prompts x 8 samples workload at full size, in the launch
    configuration the benchmark times: sampled rows first, then every one of
    the B*Hq*D output elements against the oracle."""
    st = W.make_structure("shared_prefix")
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len)
    plan = pda_plan_shared_prefix(prob, make_prefix_groups(len(st.group_prefix_len), 8, 1024))
    print(f"shared_prefix plan: {plan}", flush=True)
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev)
    assert np.isfinite(got).all()
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    del k, v
    rows = W.sample_rows(st, 64)
    ref = oracle.decode_rows(qb, kb, vb, st.block_table, st.context_lens, st.scale, rows, threads=THREADS)
    check(got[rows[:, 0], rows[:, 1]], ref, "shared_prefix sampled rows")
    ref = oracle.decode(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=THREADS)
    check(got, ref, "shared_prefix every element", f"B*Hq*D = {st.B}*{st.Hq}*{st.D}")


def test_shared_prefix_config_full_size_four_tokens(dev):
    """The 32 prompts x 8 samples workload with 4 new tokens per sequence,
    as `bench.py --op prefix --tokens 4` times it (two row groups of 4
    samples per prompt): every one of the B*n*Hq*D output elements against
    the oracle's multi-token attention."""
    n = 4
    st = W.make_structure("shared_prefix")
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len,
                        num_query_tokens=n)
    plan = pda_plan_shared_prefix(prob, make_prefix_groups(len(st.group_prefix_len), 8, 1024))
    print(f"shared_prefix x {n} tokens plan: {plan}", flush=True)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    got = run(st, q, k, v, dev, max_group_size=8, max_prefix_len=1024)
    assert np.isfinite(got).all()
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    del k, v
    ref = oracle.decode_multi(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=THREADS)
    check(got, ref, f"shared_prefix {n} new tokens, every element", f"B*n*Hq*D = {st.B}*{n}*{st.Hq}*{st.D}")


def draw_groups(case: int):
    """Seeded random shared-prefix descriptors: 1-4 groups of 1 to 3 x 64/G
    members (up to three row groups) with prefixes of 0 to 2048 tokens (whole
    blocks), members' own tokens 0 to 1500 after it, and 0-3 sequences in no
    group."""
    r = np.random.default_rng(7000 + case)
    G = int(r.choice([1, 2, 4, 5, 7, 8, 16]))
    Hkv = int(r.choice([1, 2]))
    D = int(r.choice([64, 128]))
    groups = []
    for _ in range(int(r.integers(1, 5))):
        prefix = 16 * int(r.integers(0, 129))
        members = int(r.integers(1, 3 * (64 // G) + 1))
        groups.append((prefix, [prefix + int(r.choice([0, 1, 15, 16, 17, 300, 1500])) for _ in range(members)]))
    loners = [int(r.choice([0, 1, 100, 2000])) for _ in range(int(r.integers(0, 4)))]
    tp = int(r.choice([0, 0, 16, 64, 512]))
    return G, Hkv, D, groups, loners, tp


@pytest.mark.parametrize("case", range(int(os.environ.get("PDA_RANDOM_GROUP_CASES", "24"))))
def test_random_groups(dev, case):
    """Random group layouts (sizes up to three prefix items of 64 rows,
    prefixes from none to several partitions, empty suffixes, sequences in no
    group, forced partition sizes): every element against the plain decode
    definition."""
    G, Hkv, D, groups, loners, tp = draw_groups(case)
    st = W.custom_shared_structure(G * Hkv, Hkv, D, groups, loners, seed=300 + case)
    q, k, v = W.fill_values(st, dev, fill="nan")
    print(f"case {case}: G={G} Hkv={Hkv} D={D} groups={[(p, len(m)) for p, m in groups]} loners={loners} Tp={tp}",
          flush=True)
    got = run(st, q, k, v, dev, tp)
    check(got, reference(st, q, k, v), f"random groups case {case}")


@pytest.mark.parametrize("n", [2, 4, 8])
@pytest.mark.parametrize("partition_tokens", [0, 64])
def test_groups_with_several_new_tokens(dev, n, partition_tokens):
    """Shared-prefix groups with n new tokens per sequence (speculative
    decoding over parallel samples): members x n x G rows per prefix item, up
    to 64; a member whose new tokens reach back into the prefix (its rows see
    only the prefix tokens before their positions), a group without a
    prefix, sequences in no group with fewer tokens than n.  Every element
    against the oracle's multi-token attention."""
    G, Hkv = 4, 2
    size = 64 // (n * G)
    groups = [
        (256, [256 + n + 5, 300, 1000, 257, 2000, 400, 256 + n, 777][:size]),
        (64, [64 + n - 1, 500, 65, 90, 1200, 64, 70, 80][:size]),  # the first member's new tokens start inside
        (0, [n + 3, 40][:size]),
    ]
    st = W.custom_shared_structure(G * Hkv, Hkv, 128, groups, [n + 10, 1, 0], seed=40 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    got = run(st, q, k, v, dev, partition_tokens)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table, st.context_lens,
                              st.scale, threads=THREADS)
    check(got, ref, f"groups with {n} new tokens, Tp={partition_tokens}")
    assert np.array_equal(got, run(st, q, k, v, dev, partition_tokens)), "run-to-run"


@pytest.mark.parametrize("case", range(int(os.environ.get("PDA_RANDOM_GROUP_CASES", "16"))))
def test_random_groups_several_new_tokens(dev, case):
    """Random group layouts with 2 to 21 new tokens per sequence (members up
    to 2 x 64 / (n G) + 1: one to three row groups), new tokens sometimes
    reaching back into the prefix."""
    r = np.random.default_rng(8000 + case)
    G = int(r.choice([1, 2, 3, 4, 6, 7, 8, 9]))
    n = int(r.choice([2, 3, 4, 7, 8, 10, 21]))
    if n * G > 64:
        n = 64 // G
    Hkv = int(r.choice([1, 2]))
    D = int(r.choice([64, 128]))
    groups = []
    for _ in range(int(r.integers(1, 4))):
        prefix = 16 * int(r.integers(0, 65))
        members = int(r.integers(1, 2 * (64 // (n * G)) + 2))
        groups.append((prefix, [prefix + int(r.choice([0, 1, n - 1, n, n + 1, 17, 300, 900])) for _ in range(members)]))
    loners = [int(r.choice([0, 1, n, 100, 1500])) for _ in range(int(r.integers(0, 3)))]
    tp = int(r.choice([0, 0, 16, 64, 512]))
    st = W.custom_shared_structure(G * Hkv, Hkv, D, groups, loners, seed=500 + case)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    print(f"case {case}: G={G} n={n} Hkv={Hkv} D={D} groups={[(p, len(m)) for p, m in groups]} Tp={tp}", flush=True)
    got = run(st, q, k, v, dev, tp)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table, st.context_lens,
                              st.scale, threads=THREADS)
    check(got, ref, f"random groups, {n} new tokens, case {case}")
