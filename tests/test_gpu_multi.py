"""GPU parity of several new query tokens per sequence (speculative decoding,
chunked prefill: Section 3.2) through the C ABI, against the fp64 oracle.

New token i of a sequence with n new tokens and context length L sits at
position L - n + i and attends to tokens t < L - n + 1 + i.  Bar as for the
decode step: max-abs <= 8e-3 and mean-abs <= 1e-3 over every compared
element.  Small problems and the full-size steps (Llama-3-8B, long
chain-of-thought and 70B-shard shapes with 4 to 64 new tokens) are compared
on every element.
"""
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


def run_multi(st, q, k, v, dev, partition_tokens=0):
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(st.context_lens).to(dev)
    out = pda_decode(q, k, v, bt, lens, st.scale, max_context_len=st.max_context_len,
                     partition_tokens=partition_tokens)
    torch.cuda.synchronize()
    return out.cpu().numpy()




LENS = [1, 2, 3, 4, 5, 15, 16, 17, 21, 33, 64, 65, 300, 1000, 2049]
CASES = [  # (Hq, Hkv, D, n): rows per work item = min(n, 16 // G) * G
    (32, 8, 128, 4),   # G=4: one 16-row chunk
    (32, 8, 128, 7),   # two chunks (4 + 3 tokens): both folded by every wavefront, in registers
    (8, 1, 128, 4),    # G=8: two chunks of 2 tokens
    (32, 8, 64, 8),    # G=4, D=64: two full chunks
    (8, 1, 128, 2),    # G=8
    (8, 8, 128, 16),   # G=1: 16 tokens in one chunk
    (16, 1, 64, 3),    # G=16: one token per chunk
    (12, 4, 64, 5),    # G=3: chunks of 5 tokens, 15 rows
    (8, 2, 64, 1),     # a decode step given as [B][1][Hq][D]
    (8, 1, 128, 8),    # G=8: 4 chunks in one work item, one 16-row tile per wavefront
    (32, 8, 128, 13),  # G=4: 4 chunks (3 full, 1 partial) in one item
    (32, 8, 64, 21),   # G=4: 6 chunks in one item, two tiles on wavefronts 0-1
    (4, 4, 128, 40),   # G=1: 3 chunks (16 + 16 + 8 tokens)
    (32, 8, 128, 32),  # G=4: 8 chunks in one item, two tiles per wavefront
    (8, 1, 128, 12),   # G=8: 6 chunks, two tiles on wavefronts 0-1
    (12, 4, 128, 26),  # G=3: 6 chunks of 5 tokens (the last one 1), 15 rows each
    (32, 8, 128, 37),  # G=4: 10 chunks in one item on 8 wavefronts (two tiles on wavefronts 0-1)
    (32, 8, 128, 64),  # G=4: 16 chunks in one item, two tiles on each of 8 wavefronts
    (32, 8, 128, 72),  # G=4: 18 chunks, two items (16 + 2 chunks)
    (8, 1, 128, 40),   # G=8: 20 chunks of 2 tokens, two items (16 + 4 chunks)
]


def test_many_chunk_groups(dev):
    """128 new tokens at G = 4: 32 query chunks in 2 work items of 16 chunks
    (8 wavefronts of two tiles) per (partition, sequence, KV head), every
    element against the oracle."""
    lens = [1, 200, 700, 3000, 128, 1500]
    n = 128
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=73)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    got = run_multi(st, q, k, v, dev)
    check(got, ref, "128 new tokens, 2 chunk groups")


@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 1)], ids=["G4", "G8"])
@pytest.mark.parametrize("n", [256, 512])
@pytest.mark.parametrize("partition_tokens", [0, 256])
def test_chunked_prefill_sizes(dev, Hq, Hkv, n, partition_tokens):
    """Chunked-prefill-sized steps (256 and 512 new tokens per sequence: 32 to
    128 query chunks in 4 to 16 wide items per (partition, sequence, KV
    head)), with contexts shorter than the chunk (its first tokens see
    nothing or a few tokens), equal to it and longer, whole and split in
    256-token partitions; every element against the oracle."""
    lens = [n - 100, n, n + 37, 1500, 2049]
    st = W.custom_structure(len(lens), Hq, Hkv, 128, lens, seed=400 + n + Hq)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, partition_tokens, num_query_tokens=n))
    print(f"chunked prefill n={n} G={Hq // Hkv} Tp={partition_tokens}: plan {plan}", flush=True)
    got = run_multi(st, q, k, v, dev, partition_tokens)
    for b, L in enumerate(lens):  # rows of tokens before the context's start see nothing
        assert np.all(got[b, :max(0, n - L)] == 0), b
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    check(got, ref, f"chunked prefill n={n} Hq={Hq} Hkv={Hkv} Tp={partition_tokens}",
          f"B*n*Hq*D = {st.B}*{n}*{Hq}*128")


def test_chunked_prefill_full_size_sampled(dev):
    """The chunked-prefill workload at full size (32 sequences, contexts of
    1024-8192 tokens whose last 512 are the chunk), in the launch
    configuration the benchmark times; rows sampled over sequences, chunk
    positions and heads (the oracle would need minutes for all of them), plus
    properties of every row: finite, and each a convex combination of V rows."""
    st = W.make_structure("chunked_prefill")
    n = 512
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, num_query_tokens=n))
    print(f"chunked_prefill x {n}: plan={plan}", flush=True)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    got = run_multi(st, q, k, v, dev)
    assert np.isfinite(got).all()
    vmax = float(torch.nan_to_num(v.float().abs(), nan=0.0).max())
    assert np.abs(got).max() <= vmax
    r = np.random.default_rng(17)
    rows = np.stack([r.integers(0, st.B, 256), r.integers(0, n, 256), r.integers(0, st.Hq, 256)], axis=1)
    rows[:8, 1] = [0, 1, 2, 255, 256, 509, 510, 511]
    ref = oracle.decode_multi_rows(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                                   st.context_lens, st.scale, rows.astype(np.int32), threads=THREADS)
    check(got[rows[:, 0], rows[:, 1], rows[:, 2]], ref, "chunked_prefill 512 new tokens, sampled rows")


@pytest.mark.parametrize("Hq,Hkv,D,n", CASES, ids=lambda x: str(x))
@pytest.mark.parametrize("partition_tokens", [0, 16, 64])
def test_multi_token_parity(dev, Hq, Hkv, D, n, partition_tokens):
    st = W.custom_structure(len(LENS), Hq, Hkv, D, LENS, seed=100 + Hq + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    got = run_multi(st, q, k, v, dev, partition_tokens)
    # rows of tokens that see nothing (L < n) are zero
    for b, L in enumerate(LENS):
        for i in range(n):
            if L - n + 1 + i <= 0:
                assert np.all(got[b, i] == 0), (b, i)
    check(got, ref, f"multi Hq={Hq} Hkv={Hkv} D={D} n={n} Tp={partition_tokens}")


def test_one_token_equals_decode_step(dev):
    """q as [B][1][Hq][D] runs the same arithmetic as the decode step: bitwise."""
    lens = [1, 17, 300, 2049, 4096, 0]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=7)
    q, k, v = W.fill_values(st, dev, fill="nan")
    a = run_multi(st, q, k, v, dev)
    b = run_multi(st, q[:, None].contiguous(), k, v, dev)
    assert np.array_equal(a, b[:, 0])


@pytest.mark.parametrize("n", [4, 32])
def test_multi_token_poison_and_shuffle_bit_identical(dev, n):
    lens = [40, 7, 900, 2047]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=9)
    q = W.fill_multi_q(st, n, dev)
    _, k, v = W.fill_values(st, dev, fill="nan")
    base = run_multi(st, q, k, v, dev)
    assert np.array_equal(base, run_multi(st, q, k, v, dev)), "run-to-run"
    st2, k2, v2 = W.permute_pool(st, k, v, seed=3)
    assert np.array_equal(base, run_multi(st2, q, k2, v2, dev)), "block shuffle"
    _, kz, vz = W.fill_values(st, dev, fill="zero")
    assert np.array_equal(base, run_multi(st, q, kz, vz, dev)), "NaN poison vs zero fill"


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("n", [1, 8, 32, 60], ids=["register", "mixed", "wide", "wide16"])
@pytest.mark.parametrize("partition_tokens", [0, 64])
def test_run_to_run_bitwise_every_variant(dev, D, n, partition_tokens):
    """Three runs give identical bits in each compiled variant of the
    partition kernel at both head dims: one 16-row tile per item in registers
    (n = 1), up to 4 tiles staged through LDS (n = 8 at G = 4: 2 tiles), the
    wide variant with two tiles per wavefront (n = 32: 8 tiles) and its
    8-wavefront form (n = 60: 15 tiles); with whole and split contexts.  These runs guard the ordering of the score
    MFMAs and their first VALU reads, which the compiler once left without
    the wait states a read of an MFMA result needs."""
    lens = [1, 17, 300, 2049, 40, 64, 1000, 513]
    st = W.custom_structure(len(lens), 32, 8, D, lens, seed=300 + n + D)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    base = run_multi(st, q, k, v, dev, partition_tokens)
    for _ in range(2):
        assert np.array_equal(base, run_multi(st, q, k, v, dev, partition_tokens)), "run-to-run"
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    check(base, ref, f"variant n={n} D={D} Tp={partition_tokens}")


@pytest.mark.parametrize("name,n", [("llama3_8b", 4), ("llama3_8b", 32), ("llama3_70b_tp8", 16),
                                    ("long_cot", 64)], ids=lambda x: str(x))
def test_multi_token_full_size(dev, name, n):
    """Full-size steps with n new tokens per sequence (4 draft tokens to
    verify in speculative decoding; 16-64 for wide items, split contexts and
    two chunk groups), in the launch configuration the benchmark times:
    sampled rows first, then every one of the B*n*Hq*D output elements."""
    st = W.make_structure(name)
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, num_query_tokens=n))
    print(f"{name} x {n} tokens: plan={plan}", flush=True)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    got = run_multi(st, q, k, v, dev)
    assert np.isfinite(got).all()
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    del k, v
    r = np.random.default_rng(5)
    rows = np.stack([r.integers(0, st.B, 64), r.integers(0, n, 64), r.integers(0, st.Hq, 64)], axis=1)
    rows[0] = [int(np.argmax(st.context_lens)), n - 1, st.Hq - 1]
    rows[1] = [int(np.argmin(st.context_lens)), 0, 0]
    ref = oracle.decode_multi_rows(qb, kb, vb, st.block_table, st.context_lens, st.scale, rows.astype(np.int32),
                                   threads=THREADS)
    check(got[rows[:, 0], rows[:, 1], rows[:, 2]], ref, f"{name} {n} new tokens, sampled rows")
    ref = oracle.decode_multi(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=THREADS)
    check(got, ref, f"{name} {n} new tokens, every element", f"B*n*Hq*D = {st.B}*{n}*{st.Hq}*{st.D}")


@pytest.mark.parametrize("factor", [-1.0, 0.0, 3.0, 25.0])
def test_scale_sign_zero_and_peaked(dev, factor):
    """Negative, zero and large scales, on the register path (one tile per
    work item) and on the staged path (several tiles, folded in pairs of
    blocks).  The kernels fold the sign of the scale into q and a zero scale
    into zero scores; a large scale makes the softmax peaked, so the running
    max moves often."""
    lens = [1, 17, 300, 2049, 40, 64]
    for (Hq, Hkv, D, n) in [(32, 8, 128, 1), (8, 2, 64, 1), (32, 8, 128, 16), (8, 1, 128, 8), (16, 4, 64, 13)]:
        st = W.custom_structure(len(lens), Hq, Hkv, D, lens, seed=40 + n)
        _, k, v = W.fill_values(st, dev, fill="nan")
        q = W.fill_multi_q(st, n, dev)
        scale = float(np.float32(st.scale * factor))
        bt = torch.from_numpy(st.block_table).to(dev)
        ln = torch.from_numpy(st.context_lens).to(dev)
        got = pda_decode(q, k, v, bt, ln, scale, max_context_len=st.max_context_len).cpu().numpy()
        ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                                  st.context_lens, scale, threads=THREADS)
        check(got, ref, f"scale x{factor} Hq={Hq} Hkv={Hkv} D={D} n={n}")
