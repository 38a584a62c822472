"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bar (floating point): over every compared element, max-abs error <= 8e-3 and
mean-abs error <= 1e-3 against the oracle's fp64 result.  Bitwise where the
method fixes the bits: a one-token context returns its V row exactly, moving
physical blocks around the pool or filling unread slots with NaN leaves the
output bit-identical, and two runs give identical bits.

Small problems are compared on every element.  The named decode
configurations run at full size in the launch configuration the benchmark
times and are compared on every element too (after a quick check of
sampled rows); the 64K-token case is compared on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from parity_common import THREADS, check
from paper_2405_11143_amd import pda_decode, pda_plan, make_problem

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def gpu_tensors(st, dev):
    return (torch.from_numpy(st.block_table).to(dev), torch.from_numpy(st.context_lens).to(dev))


def run(st, q, k, v, dev, partition_tokens=0, max_context_len=None):
    bt, lens = gpu_tensors(st, dev)
    mcl = st.max_context_len if max_context_len is None else max_context_len
    out = pda_decode(q, k, v, bt, lens, st.scale, max_context_len=mcl, partition_tokens=partition_tokens)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def reference(st, q, k, v):
    return oracle.decode(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                         st.context_lens, st.scale, threads=THREADS)




# ------------------------------------------------------------ small, full --

@pytest.mark.parametrize("partition_tokens", [0, 16, 64, 128])
def test_tiny_config(dev, partition_tokens):
    st = W.make_structure("tiny")
    q, k, v = W.fill_values(st, dev, fill="nan")
    check(run(st, q, k, v, dev, partition_tokens), reference(st, q, k, v), f"tiny Tp={partition_tokens}")


EDGE_LENS = [1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 511, 512, 513, 1000, 2049]
SHAPES = [(8, 2, 64), (32, 8, 128), (8, 1, 128), (4, 4, 128), (12, 2, 128), (28, 4, 128),
          (40, 8, 128), (16, 1, 64), (6, 2, 64), (3, 1, 128)]


@pytest.mark.parametrize("Hq,Hkv,D", SHAPES, ids=lambda x: str(x))
@pytest.mark.parametrize("partition_tokens", [0, 64])
def test_shapes_and_edge_lengths(dev, Hq, Hkv, D, partition_tokens):
    """Every group size kind (G = 1, 3, 4, 5, 6, 7, 8, 16), both head dims, and
    context lengths at block and partition boundaries."""
    st = W.custom_structure(len(EDGE_LENS), Hq, Hkv, D, EDGE_LENS, seed=Hq * 100 + D)
    q, k, v = W.fill_values(st, dev, fill="nan")
    check(run(st, q, k, v, dev, partition_tokens), reference(st, q, k, v),
          f"Hq={Hq} Hkv={Hkv} D={D} Tp={partition_tokens}")


@pytest.mark.parametrize("partition_tokens", [16, 48, 256, 512, 4096])
def test_split_sizes_agree(dev, partition_tokens):
    lens = [3000, 1, 700, 4096, 513, 2222, 17, 1024]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=5)
    q, k, v = W.fill_values(st, dev, fill="nan")
    check(run(st, q, k, v, dev, partition_tokens), reference(st, q, k, v), f"split Tp={partition_tokens}")


@pytest.mark.parametrize("partition_tokens", [0, 16, 256])
def test_ragged_batch_with_empty_contexts(dev, partition_tokens):
    """Many partitions of very different sizes in one step, so the largest-
    first work order differs from the natural one; empty contexts at the
    start, middle and end of the batch come out as zero rows."""
    lens = [0, 3000, 1, 700, 0, 4096, 513, 17, 1024, 2049, 16, 0]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=21 + partition_tokens)
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev, partition_tokens)
    assert np.all(got[[0, 4, 11]] == 0)
    check(got, reference(st, q, k, v), f"ragged Tp={partition_tokens}")


@pytest.mark.parametrize("partition_tokens", [0, 64, 4096])
def test_dirty_workspace(dev, partition_tokens):
    """Each pass may only read what the step itself wrote: a workspace full of
    0xFF bytes (NaN partial states, out-of-range work items) must not matter."""
    for lens in ([5, 40, 1, 300, 0, 77], [2000, 3000, 1500]):
        st = W.custom_structure(len(lens), 16, 4, 128, lens, seed=31)
        q, k, v = W.fill_values(st, dev, fill="nan")
        prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                            st.max_context_len, partition_tokens)
        ws = torch.full((pda_plan(prob)["workspace_bytes"],), 0xFF, dtype=torch.uint8, device=dev)
        bt, ln = gpu_tensors(st, dev)
        out = pda_decode(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len,
                         partition_tokens=partition_tokens, workspace=ws)
        torch.cuda.synchronize()
        check(out.cpu().numpy(), reference(st, q, k, v), f"dirty workspace Tp={partition_tokens} lens={lens}")


# ------------------------------------------------------------ invariants --

def test_length_one_returns_v_exactly(dev):
    for (Hq, Hkv, D, tp) in [(32, 8, 128, 0), (8, 2, 64, 16), (16, 1, 128, 0)]:
        st = W.custom_structure(40, Hq, Hkv, D, [1] * 40, seed=3)
        q, k, v = W.fill_values(st, dev, fill="nan")
        got = run(st, q, k, v, dev, tp)
        vf = v.float().cpu().numpy()
        G = Hq // Hkv
        for b in range(st.B):
            p = st.block_table[b, 0]
            for h in range(Hq):
                assert np.array_equal(got[b, h], vf[p, h // G, 0]), (Hq, Hkv, D, b, h)


def test_constant_v_gives_constant(dev):
    lens = [1, 16, 17, 300, 2000, 5000]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=4)
    q, k, v = W.fill_values(st, dev, fill="nan")
    mask = torch.from_numpy(W.unread_slot_mask(st)).to(dev)[:, None, :, None]
    v = torch.ones_like(v).masked_fill_(mask, float("nan"))
    # The P.V product takes each probability p as two bf16 halves, hi = p
    # truncated to bf16 and lo = bf16(p - hi), so every weight carries a
    # relative error below 2^-16 against the fp32 denominator; the output, a
    # convex combination of ones, is 1 within that bound (plus fp32 rounding).
    for tp in (0, 64):
        got = run(st, q, k, v, dev, tp)
        assert np.abs(got - 1.0).max() <= 2.0 ** -16 + 1e-6


def test_gqa_mapping(dev):
    for (Hq, Hkv) in [(32, 8), (8, 1), (12, 4), (10, 2)]:
        st = W.custom_structure(3, Hq, Hkv, 128, [50, 700, 1], seed=6)
        q, k, _ = W.fill_values(st, dev, fill=None)
        v = (torch.arange(Hkv, device=dev, dtype=torch.float32) + 1).view(1, Hkv, 1, 1)
        v = v.expand(st.num_blocks, Hkv, 16, 128).contiguous().to(torch.bfloat16)
        got = run(st, q, k, v, dev, 64)
        G = Hq // Hkv
        for h in range(Hq):
            # weights carry a relative error below 2^-16 (bf16 hi/lo probabilities)
            assert np.abs(got[:, h] - (h // G + 1)).max() <= (h // G + 1) * (2.0 ** -16 + 1e-6), (Hq, Hkv, h)


def test_block_shuffle_and_poison_bit_identical(dev):
    lens = [33, 1, 900, 2047, 64, 129]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=7)
    for tp in (0, 64):
        q, k, v = W.fill_values(st, dev, fill="nan")
        base = run(st, q, k, v, dev, tp)
        assert np.array_equal(base, run(st, q, k, v, dev, tp)), "run-to-run"
        st2, k2, v2 = W.permute_pool(st, k, v, seed=11)
        assert np.array_equal(base, run(st2, q, k2, v2, dev, tp)), "block shuffle"
        qz, kz, vz = W.fill_values(st, dev, fill="zero")
        assert np.array_equal(base, run(st, qz, kz, vz, dev, tp)), "NaN poison vs zero fill"


def test_empty_and_nonpositive_lengths(dev):
    st = W.custom_structure(4, 8, 2, 64, [0, 20, -5, 1], seed=8)
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev, 0)
    assert np.all(got[0] == 0) and np.all(got[2] == 0)
    check(got, reference(st, q, k, v), "lengths 0, 20, -5, 1")
    # an empty batch launches nothing
    e = torch.empty((0, 8, 64), dtype=torch.bfloat16, device=dev)  # k, v from the problem above
    out = pda_decode(e, k, v, torch.empty((0, 2), dtype=torch.int32, device=dev),
                     torch.empty((0,), dtype=torch.int32, device=dev), 0.125, max_context_len=0)
    assert out.shape == (0, 8, 64)


# ------------------------------------------------- full-size configurations --

@pytest.mark.parametrize("name", ["llama3_8b", "long_cot", "llama3_70b_tp8", "shared_prefix", "r1_qwen7b",
                                  "r1_qwen14b"])
def test_full_config(dev, name):
    """A named decode configuration at full size, in the launch configuration
    the benchmark times: sampled rows first (a quick check that names the
    rows), then every one of the B*Hq*D output elements against the oracle."""
    st = W.make_structure(name)
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len))
    print(f"{name}: B={st.B} pool={st.num_blocks} blocks, plan={plan}", flush=True)
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev)
    assert np.isfinite(got).all()
    vmax = float(torch.nan_to_num(v.float().abs(), nan=0.0).max())
    assert np.abs(got).max() <= vmax  # each output is a convex combination of V rows
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    del k, v
    rows = W.sample_rows(st, 64)
    ref = oracle.decode_rows(qb, kb, vb, st.block_table, st.context_lens, st.scale, rows, threads=THREADS)
    check(got[rows[:, 0], rows[:, 1]], ref, f"{name} sampled rows")
    ref = oracle.decode(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=THREADS)
    check(got, ref, f"{name} every element", f"B*Hq*D = {st.B}*{st.Hq}*{st.D}")


def test_long_contexts_sampled(dev):
    """Contexts up to 64K tokens with the automatic partition size (16
    partitions, so the merge takes its general path), sampled rows against
    the oracle, including every row of the longest context's first KV head."""
    lens = [65536, 40000, 1, 17, 8191, 65535, 30000, 4096, 100, 65520, 12345, 2]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=71)
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len))
    print(f"long contexts: plan={plan}", flush=True)
    assert plan["num_partitions"] > 8
    q, k, v = W.fill_values(st, dev, fill="nan")
    got = run(st, q, k, v, dev)
    assert np.isfinite(got).all()
    r = np.random.default_rng(72)
    rows = np.stack([r.integers(0, st.B, 48), r.integers(0, st.Hq, 48)], axis=1)
    rows = np.concatenate([rows, np.stack([np.zeros(4, int), np.arange(4)], axis=1)]).astype(np.int32)
    ref = oracle.decode_rows(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                             st.context_lens, st.scale, rows, threads=THREADS)
    check(got[rows[:, 0], rows[:, 1]], ref, "long contexts, sampled rows")


@pytest.mark.parametrize("Hq,Hkv,n", [(8, 1, 1), (16, 2, 1), (8, 1, 12), (32, 8, 24), (32, 8, 40)], ids=str)
def test_work_order_placements(dev, Hq, Hkv, n):
    """Steps with more work items than the GPU runs at once, so the work-order
    kernel runs: with fewer than 8 KV heads (pairs placed in octets, the last
    one partial: 301 sequences x 10 partitions) and with 8 (KV heads kept on
    their XCD), with one group of query chunks per (sequence, KV head) and
    with two (40 new tokens: 10 chunks in groups of 8 and 2)."""
    r = np.random.default_rng(Hq * 7 + n)
    lens = [int(x) for x in r.integers(n, 600, 301)]
    st = W.custom_structure(len(lens), Hq, Hkv, 128, lens, seed=60 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    tp = 64
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, tp, num_query_tokens=n))
    G = Hq // Hkv
    chunks = -(-n // max(1, 16 // G))
    pairs = plan["num_partitions"] * st.B
    per_item = 8 if chunks > 4 else 4  # chunks per work item
    items = pairs * Hkv * -(-chunks // per_item)
    assert items > 768 and (Hkv % 8 == 0 or pairs % 8 != 0), (items, pairs)
    bt, ln = gpu_tensors(st, dev)
    got = pda_decode(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len,
                     partition_tokens=tp).cpu().numpy()
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    check(got, ref, f"order placement Hq={Hq} Hkv={Hkv} n={n} plan={plan}")


@pytest.mark.parametrize("n,partition_tokens", [(1, 0), (1, 64), (8, 0), (16, 64)], ids=str)
def test_out_of_range_block_ids_give_nan_rows(dev, n, partition_tokens):
    """A block-table entry outside the pool (within a context) is never
    dereferenced: every output row of that sequence comes out NaN, and the
    other sequences are unaffected.  Covers the register path (one tile per
    work item) and the staged path (8 and 16 new tokens at G = 4), with and
    without split contexts."""
    lens = [100, 300, 50, 1000, 777]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=90 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    table = st.block_table.copy()
    table[1, 3] = st.num_blocks + 7
    table[3, 40] = -1
    bt = torch.from_numpy(table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    got = pda_decode(q, k, v, bt, ln, st.scale, max_context_len=st.max_context_len,
                     partition_tokens=partition_tokens).cpu().numpy()
    assert np.isnan(got[1]).all() and np.isnan(got[3]).all()
    ok = [0, 2, 4]
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    check(got[ok], ref[ok], f"sequences with valid tables n={n} Tp={partition_tokens}")


@pytest.mark.parametrize("n,partition_tokens", [(1, 0), (1, 64), (8, 0), (40, 64)], ids=str)
def test_nan_inside_a_context_propagates_like_the_oracle(dev, n, partition_tokens):
    """A NaN key element inside a context makes every row that sees that
    token NaN; a NaN value element makes that output column NaN in those
    rows; everything else is unaffected.  The positions of NaN outputs equal
    the oracle's and the other elements meet the bar.  The poisoned tokens
    come before the new tokens, so every row of the sequence sees them (the
    register path, the staged path and 8-wavefront items; whole and split
    contexts)."""
    lens = [200, 300, 150, 1000, 777]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=95 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=dev)
    # key of sequence 1, KV head 2, token 37, element 5; value of sequence 3, KV head 5, token 600, element 77
    p1 = int(st.block_table[1, 37 // 16])
    k[p1, 2, 5 // 8, 37 % 16, 5 % 8] = nan
    p3 = int(st.block_table[3, 600 // 16])
    v[p3, 5, 600 % 16, 77] = nan
    got = run(st, q, k, v, dev, partition_tokens)
    ref = oracle.decode_multi(W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v), st.block_table,
                              st.context_lens, st.scale, threads=THREADS)
    got = got.reshape(ref.shape)
    assert np.isnan(ref[1, :, 8:12]).all() and np.isnan(ref[3, :, 20:24, 77]).all()  # the oracle's reading
    assert np.array_equal(np.isnan(got), np.isnan(ref)), "NaN positions differ from the oracle's"
    fin = ~np.isnan(ref)
    check(got[fin], ref[fin], f"finite elements n={n} Tp={partition_tokens}")
