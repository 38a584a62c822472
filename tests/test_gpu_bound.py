"""Bound calls (bind_decode, bind_append_kv): the same entry points with their
arguments prepared once, as a serving loop calls them step after step.  They
must give exactly what the per-call functions give, and see the bound
buffers' current contents on every call."""
import numpy as np
import pytest
import torch

import workloads as W
from paper_2405_11143_amd import (bind_append_kv, bind_decode, make_problem, pda_append_kv, pda_decode,
                                  pda_decode_reusing_order, pda_merge_partitions, pda_partition_attention, pda_plan,
                                  pda_work_order, pda_workspace_bytes)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


@pytest.mark.parametrize("n", [1, 4, 21])
def test_bound_decode_matches_and_follows_contents(dev, n):
    lens = [1, 17, 300, 2049, 0, 700]
    st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=50 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev) if n > 1 else W.fill_values(st, dev, fill="nan")[0]
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=64)
    step = bind_decode(q, k, v, bt, ln, st.scale, **kw)
    for rep in range(3):
        got = step().clone()
        want = pda_decode(q, k, v, bt, ln, st.scale, **kw)
        torch.cuda.synchronize()
        assert torch.equal(got, want), rep
        q.mul_(-1.5)  # the next call must see the new queries
    # pass 1 alone: the outputs it finalises and the partial states it leaves
    # (both buffers zeroed first: pass 1 does not write every element of them)
    outs = [torch.zeros(q.shape, dtype=torch.float32, device=dev) for _ in range(2)]
    wss = [torch.zeros(step._keep[-1].numel(), dtype=torch.uint8, device=dev) for _ in range(2)]
    bind_decode(q, k, v, bt, ln, st.scale, outs[0], workspace=wss[0], pass1_only=True, **kw)()
    pda_partition_attention(q, k, v, bt, ln, st.scale, outs[1], workspace=wss[1], **kw)
    torch.cuda.synchronize()
    # the partial states lead the workspace; the work order after them may
    # list items of equal size in either order
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, 64, num_query_tokens=n))
    parts = plan["num_partitions"]
    state_bytes = st.B * n * st.Hq * parts * (st.D + 2) * 4 if parts > 1 else 0
    assert state_bytes > 0
    assert torch.equal(outs[0], outs[1]) and torch.equal(wss[0][:state_bytes], wss[1][:state_bytes])


@pytest.mark.parametrize("n", [1, 8])
def test_reused_work_order_matches_decode(dev, n):
    """One work order per step, reused by every layer: bitwise pda_decode's
    result, also when the order is stale (lengths changed since it was taken)
    and when an earlier pda_decode left it."""
    rng = np.random.default_rng(70 + n)
    B = 48
    lens = rng.integers(1, 3000, size=B).tolist()
    st = W.custom_structure(B, 32, 8, 128, lens, seed=71 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    qs = [W.fill_multi_q(st, n, dev) if n > 1 else W.fill_values(st, dev, fill="nan")[0] for _ in range(2)]
    qs[1].mul_(0.5)
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=64)
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len, 64,
                        num_query_tokens=n)
    plan = pda_plan(prob)
    assert plan["num_partitions"] * st.B * st.Hkv > 768  # large enough that pass 1 takes an ordered list
    ws = torch.zeros(pda_workspace_bytes(prob), dtype=torch.uint8, device=dev)
    pda_work_order(prob, ln, ws)
    for layer, q in enumerate(qs):
        got = pda_decode_reusing_order(q, k, v, bt, ln, st.scale, workspace=ws, **kw)
        want = pda_decode(q, k, v, bt, ln, st.scale, **kw)
        torch.cuda.synchronize()
        assert torch.equal(got, want), layer
    # stale order: after it was taken, the lengths change rank (each stays
    # within its own sequence's blocks, so no row reads an unwritten slot)
    ln2 = torch.from_numpy(np.minimum(rng.permutation(st.context_lens), st.context_lens)).to(dev)
    assert not torch.equal(ln2, ln)
    got = pda_decode_reusing_order(qs[0], k, v, bt, ln2, st.scale, workspace=ws, **kw)
    want = pda_decode(qs[0], k, v, bt, ln2, st.scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(got, want)
    # the order pda_decode leaves in its workspace serves the next layer
    ws2 = torch.zeros_like(ws)
    pda_decode(qs[0], k, v, bt, ln, st.scale, workspace=ws2, **kw)
    got = bind_decode(qs[1], k, v, bt, ln, st.scale, workspace=ws2, reuse_order=True, **kw)()
    want = pda_decode(qs[1], k, v, bt, ln, st.scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(got, want)
    # pass 1 alone with the reused order, then the merge: the same bits again
    got = bind_decode(qs[1], k, v, bt, ln, st.scale, workspace=ws2, pass1_only=True, reuse_order=True, **kw)()
    pda_merge_partitions(prob, ln, got, ws2)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


@pytest.mark.parametrize("n,tp,conc", [(24, 2048, 512), (40, 4096, 256)], ids=["wide", "wide16"])
def test_reused_work_order_between_variant_and_full_concurrency(dev, n, tp, conc):
    """A step of the wide variants with more items than that variant runs at
    once but at most 768 (what the one-tile variants run at once): the step
    takes an ordered list, so pda_work_order must write it too, and the
    reused order gives pda_decode's bits."""
    rng = np.random.default_rng(80 + n)
    B = 48
    lens = rng.integers(2100, 3000, size=B).tolist()
    st = W.custom_structure(B, 32, 8, 128, lens, seed=81 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    q = W.fill_multi_q(st, n, dev)
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=tp)
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len, tp,
                        num_query_tokens=n)
    items = pda_plan(prob)["num_partitions"] * st.B * st.Hkv  # one chunk group per (partition, sequence, head)
    assert conc < items <= 768, items
    ws = torch.full((pda_workspace_bytes(prob),), 0xFF, dtype=torch.uint8, device=dev)  # no order left over
    pda_work_order(prob, ln, ws)
    got = pda_decode_reusing_order(q, k, v, bt, ln, st.scale, workspace=ws, **kw)
    want = pda_decode(q, k, v, bt, ln, st.scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(got, want)


def test_bound_append_matches(dev):
    lens = [5, 33, 16, 1000]
    st = W.custom_structure(len(lens), 8, 2, 64, lens, seed=61)
    _, k, v = W.fill_values(st, dev, fill="zero")
    kn, vn = W.fill_new_kv(st, 2, dev)
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    k2, v2 = k.clone(), v.clone()
    bind_append_kv(kn, vn, bt, ln, k, v, max_context_len=st.max_context_len, num_q_heads=8)()
    pda_append_kv(kn, vn, bt, ln, k2, v2, max_context_len=st.max_context_len, num_q_heads=8)
    torch.cuda.synchronize()
    assert torch.equal(k, k2) and torch.equal(v, v2)
    assert not torch.equal(k, torch.zeros_like(k))


def test_bound_decode_rejects_bad_tensors(dev):
    st = W.custom_structure(2, 8, 2, 64, [3, 9], seed=62)
    q, k, v = W.fill_values(st, dev, fill="zero")
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    with pytest.raises(TypeError):
        bind_decode(q.float(), k, v, bt, ln, st.scale, max_context_len=st.max_context_len)
    with pytest.raises(ValueError):
        bind_decode(q, k, v, bt.cpu(), ln, st.scale, max_context_len=st.max_context_len)
