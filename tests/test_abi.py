"""The C ABI on the host (no GPU): the library loads, exports every symbol the
header declares, and rejects bad arguments before touching the GPU.

Every call here that passes pointers is built to fail host validation, so no
kernel is ever launched from these tests."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2405_11143_amd as pda
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def declared_functions():
    """Every pda_* function that a header under include/ declares."""
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if h.endswith(".h"):
            text = re.sub(r"/\*.*?\*/", "", open(os.path.join(INCLUDE, h)).read(), flags=re.S)
            names |= set(re.findall(r"\b(pda_\w+)\s*\(", text))
    return sorted(names)


def test_header_declarations_match_binding():
    assert declared_functions() == sorted(pda.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = pda.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    nm = subprocess.run(["nm", "-D", "--defined-only", pda.LIB_PATH], capture_output=True, text=True,
                        check=True).stdout
    exported = set(re.findall(r"\bT (pda_\w+)", nm))
    assert set(declared_functions()) <= exported


def prob(**kw):
    """A valid descriptor (planning needs no device)."""
    base = dict(num_seqs=4, num_q_heads=8, num_kv_heads=2, head_dim=64, num_blocks=128,
                max_blocks_per_seq=17, max_context_len=257, partition_tokens=0)
    base.update(kw)
    return pda.make_problem(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(num_seqs=-1), pda.pda.PDA_ERR_SHAPE),
    (dict(num_q_heads=0), pda.pda.PDA_ERR_SHAPE),
    (dict(num_q_heads=6, num_kv_heads=4), pda.pda.PDA_ERR_SHAPE),
    (dict(num_blocks=0), pda.pda.PDA_ERR_SHAPE),
    (dict(max_context_len=17 * 16 + 1), pda.pda.PDA_ERR_SHAPE),
    (dict(max_context_len=-1), pda.pda.PDA_ERR_SHAPE),
    (dict(partition_tokens=24), pda.pda.PDA_ERR_SHAPE),
    (dict(partition_tokens=-16), pda.pda.PDA_ERR_SHAPE),
    (dict(head_dim=96), pda.pda.PDA_ERR_UNSUPPORTED),
    (dict(block_size=32), pda.pda.PDA_ERR_UNSUPPORTED),
    (dict(num_q_heads=34, num_kv_heads=2), pda.pda.PDA_ERR_UNSUPPORTED),
])
def test_plan_rejects(kw, status):
    with pytest.raises(pda.PdaError) as e:
        pda.pda_plan(prob(**kw))
    assert e.value.status == status


def llama(**kw):
    base = dict(num_seqs=256, num_q_heads=32, num_kv_heads=8, head_dim=128, max_blocks_per_seq=1024,
                max_context_len=4096, num_blocks=50000)
    base.update(kw)
    return prob(**base)


def plan(**kw):
    d = pda.pda_plan(llama(**kw))
    return d["partition_tokens"], d["num_partitions"], d["workspace_bytes"]


def test_plan_workspace():
    # one fp32 partial state (D values + max + denominator) per query head and
    # partition when contexts are split, then one int32 per work item
    # (partition, sequence, KV head)
    assert plan(partition_tokens=2048) == (2048, 2, 256 * 32 * 2 * (128 + 2) * 4 + 2 * 256 * 8 * 4)
    assert plan(partition_tokens=4096) == (4096, 1, 256 * 8 * 4)
    assert plan(partition_tokens=8192) == (4096, 1, 256 * 8 * 4)  # beyond the longest context: clamped
    assert pda.pda_plan(prob(partition_tokens=64))["workspace_bytes"] == 4 * 8 * 5 * 66 * 4 + 5 * 4 * 2 * 4
    assert plan(num_seqs=0)[2] == 0
    assert pda.pda_workspace_bytes(llama()) == plan()[2]


def test_plan_partition_choice():
    # B * Hkv * chunk groups * max_len / 2 tokens over 768 concurrent
    # workgroups (x 1.3 for items of 16 or more query rows); above 4608 the
    # fewest equal pieces of at most 4608; rounded up to 256 tokens, at least 256
    assert plan()[:2] == (4096, 1)                        # share 5462 -> one piece of 4096
    assert plan(num_seqs=9000)[:2] == (4096, 1)
    assert plan(num_seqs=64)[:2] == (1536, 3)             # share 1366
    assert plan(num_seqs=32)[:2] == (768, 6)              # share 683
    assert plan(num_seqs=1)[:2] == (256, 16)              # share 22
    shard = dict(num_seqs=512, num_kv_heads=1, num_q_heads=8, max_context_len=8183)
    assert plan(**shard)[:2] == (2816, 3)                 # share 2728
    assert plan(**shard, num_query_tokens=2)[:2] == (3584, 3)  # 16 rows per item: 2728 * 1.3
    assert plan(**shard, num_query_tokens=8)[:2] == (3584, 3)  # 64 rows per item
    assert plan(num_seqs=64, max_context_len=15288)[:2] == (3840, 4)   # share 5096: 4 x 3822
    assert plan(num_seqs=64, max_context_len=16384)[:2] == (4096, 4)   # share 5462: 4 x 4096
    assert plan(num_q_heads=28, num_kv_heads=4, max_context_len=9216)[:2] == (4608, 2)  # share 6144
    # never longer than the longest context, rounded up to a whole block
    assert plan(num_seqs=9000, max_context_len=2001)[:2] == (2016, 1)
    assert plan(max_context_len=0)[:2] == (16, 1)
    # a forced size is kept
    assert plan(partition_tokens=16)[:2] == (16, 256)
    # a forced size beyond the longest context is one partition of that context
    assert plan(partition_tokens=2 ** 31 - 16)[:2] == (4096, 1)
    assert plan(max_context_len=0, partition_tokens=1024)[:2] == (16, 1)
    # sizes whose work estimate overflows 64 bits: the grid bound rejects them
    with pytest.raises(pda.PdaError) as e:
        plan(num_seqs=2 ** 20, num_q_heads=16, num_kv_heads=16, max_blocks_per_seq=2 ** 24,
             max_context_len=2 ** 28, num_blocks=10 ** 9)
    assert e.value.status == pda.pda.PDA_ERR_SHAPE
    # contexts beyond 2^28 tokens are refused (token sums stay far inside int32)
    for mcl in (2 ** 28 + 1, 2 ** 31 - 1):
        with pytest.raises(pda.PdaError) as e:
            plan(max_blocks_per_seq=2 ** 27, max_context_len=mcl)
        assert e.value.status == pda.pda.PDA_ERR_SHAPE
    # rows B * n * Hq beyond int32, with every factor alone in range (the product of
    # the three overflows even int64)
    with pytest.raises(pda.PdaError) as e:
        plan(num_seqs=2 ** 30, num_query_tokens=2 ** 30, num_q_heads=2 ** 30, num_kv_heads=2 ** 26)
    assert e.value.status == pda.pda.PDA_ERR_SHAPE


def call(fn, p, q=0x1000, k=0x1000, v=0x1000, bt=0x1000, lens=0x1000, scale=0.125, out=0x1000,
         ws=None, ws_bytes=0):
    lib = pda.load_library()
    return getattr(lib, fn)(ctypes.byref(p), q, k, v, bt, lens, ctypes.c_float(scale), out, ws, ws_bytes, None)


@pytest.mark.parametrize("fn", ["pda_decode", "pda_partition_attention", "pda_decode_reusing_order",
                                "pda_partition_attention_reusing_order"])
def test_step_validation(fn):
    lib = pda.load_library()
    assert call(fn, prob(), q=None) == pda.pda.PDA_ERR_NULL
    assert call(fn, prob(), lens=None) == pda.pda.PDA_ERR_NULL
    assert call(fn, prob(), out=None) == pda.pda.PDA_ERR_NULL
    assert call(fn, prob(), scale=float("nan")) == pda.pda.PDA_ERR_VALUE
    assert call(fn, prob(), scale=float("inf")) == pda.pda.PDA_ERR_VALUE
    assert call(fn, prob(), q=0x1008) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(fn, prob(), k=0x1004) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(fn, prob(), out=0x1002) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(fn, prob(), out=0x1004) == pda.pda.PDA_ERR_ALIGNMENT  # rows are written 16 bytes at a time
    assert call(fn, prob()) == pda.pda.PDA_ERR_WORKSPACE  # the work order always needs one
    split = prob(partition_tokens=64)
    assert call(fn, split) == pda.pda.PDA_ERR_WORKSPACE
    assert call(fn, split, ws=0x1000, ws_bytes=100) == pda.pda.PDA_ERR_WORKSPACE
    need = pda.pda_workspace_bytes(split)
    assert call(fn, split, ws=0x1008, ws_bytes=need) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(fn, prob(head_dim=80)) == pda.pda.PDA_ERR_UNSUPPORTED
    assert getattr(lib, fn)(None, None, None, None, None, None, ctypes.c_float(1), None, None, 0,
                            None) == pda.pda.PDA_ERR_NULL
    # an empty batch is valid and launches nothing, even with NULL pointers
    assert call(fn, prob(num_seqs=0), q=None, k=None, v=None, bt=None, lens=None, out=None) == pda.pda.PDA_OK


def test_work_order_validation():
    lib = pda.load_library()
    p = prob(partition_tokens=64)
    need = pda.pda_workspace_bytes(p)
    wo = lib.pda_work_order
    assert wo(None, 0x1000, 0x1000, need, None) == pda.pda.PDA_ERR_NULL
    assert wo(ctypes.byref(p), None, 0x1000, need, None) == pda.pda.PDA_ERR_NULL
    assert wo(ctypes.byref(p), 0x1000, None, 0, None) == pda.pda.PDA_ERR_WORKSPACE
    assert wo(ctypes.byref(p), 0x1000, 0x1000, need - 4, None) == pda.pda.PDA_ERR_WORKSPACE
    assert wo(ctypes.byref(p), 0x1000, 0x1008, need, None) == pda.pda.PDA_ERR_ALIGNMENT
    assert wo(ctypes.byref(prob(head_dim=80)), 0x1000, 0x1000, need, None) == pda.pda.PDA_ERR_UNSUPPORTED
    # nothing to order (an empty batch, or every item runs at once): no launch, no device access
    assert wo(ctypes.byref(prob(num_seqs=0)), None, None, 0, None) == pda.pda.PDA_OK
    assert pda.pda_plan(p)["num_partitions"] > 1


def test_merge_validation():
    lib = pda.load_library()
    split = prob(partition_tokens=64)
    need = pda.pda_workspace_bytes(split)
    f = lib.pda_merge_partitions
    assert f(ctypes.byref(split), None, 0x1000, 0x1000, need, None) == pda.pda.PDA_ERR_NULL
    assert f(ctypes.byref(split), 0x1000, 0x1000, 0x1000, need - 1, None) == pda.pda.PDA_ERR_WORKSPACE
    assert f(ctypes.byref(split), 0x1000, 0x1000, 0x1004, need, None) == pda.pda.PDA_ERR_ALIGNMENT
    assert f(ctypes.byref(split), 0x1000, 0x1004, 0x1000, need, None) == pda.pda.PDA_ERR_ALIGNMENT  # out
    # nothing split: nothing to merge, no launch
    single = prob(max_context_len=200, partition_tokens=208)
    assert f(ctypes.byref(single), 0x1000, 0x1000, None, 0, None) == pda.pda.PDA_OK


def test_logprob_validation():
    """Host validation of pda_token_logprobs (no launch)."""
    f = pda.load_library().pda_token_logprobs
    ok = dict(rows=4, vocab=1000, stride=1000, dtype=pda.pda.PDA_DTYPE_BF16, logits=0x1000, tokens=0x1000,
              inv_t=1.0, lp=0x1000, ent=0x1000)

    def call(ws=None, ws_bytes=0, **kw):
        a = dict(ok, **kw)
        return f(a["rows"], a["vocab"], a["stride"], a["dtype"], a["logits"], a["tokens"],
                 ctypes.c_float(a["inv_t"]), a["lp"], a["ent"], ws, ws_bytes, None)
    assert call(rows=-1) == pda.pda.PDA_ERR_SHAPE
    assert call(vocab=0) == pda.pda.PDA_ERR_SHAPE
    assert call(stride=999) == pda.pda.PDA_ERR_SHAPE
    assert call(vocab=2**30, stride=2**30) == pda.pda.PDA_ERR_SHAPE  # a row beyond one buffer descriptor
    assert call(dtype=7) == pda.pda.PDA_ERR_UNSUPPORTED
    assert call(logits=None) == pda.pda.PDA_ERR_NULL
    assert call(tokens=None) == pda.pda.PDA_ERR_NULL
    assert call(lp=None) == pda.pda.PDA_ERR_NULL
    assert call(inv_t=float("nan")) == pda.pda.PDA_ERR_VALUE
    assert call(inv_t=-1.0) == pda.pda.PDA_ERR_VALUE
    assert call(logits=0x1008) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(stride=1004) == pda.pda.PDA_ERR_ALIGNMENT          # rows of 2008 bytes
    assert call(stride=1002, dtype=pda.pda.PDA_DTYPE_F32) == pda.pda.PDA_ERR_ALIGNMENT
    assert call(rows=0, logits=None, tokens=None, lp=None) == pda.pda.PDA_OK  # nothing to do
    # the workspace: rows split over workgroups when it is given and the batch has fewer rows than compute
    # units (at most 16 per row, at least one 16-byte chunk per thread of each)
    need = pda.pda.pda_logprob_workspace_bytes(100, 128256, pda.pda.PDA_DTYPE_BF16)
    assert need == 100 * 3 * 16
    assert pda.pda.pda_logprob_workspace_bytes(8, 128256, pda.pda.PDA_DTYPE_BF16) == 8 * 15 * 16
    assert pda.pda.pda_logprob_workspace_bytes(256, 128256, pda.pda.PDA_DTYPE_BF16) == 0  # enough rows
    assert pda.pda.pda_logprob_workspace_bytes(4, 1000, pda.pda.PDA_DTYPE_BF16) == 0  # rows too short to split
    assert call(rows=100, vocab=128256, stride=128256, ws=0x1000, ws_bytes=need - 1) == pda.pda.PDA_ERR_WORKSPACE
    assert call(rows=100, vocab=128256, stride=128256, ws=0x1008, ws_bytes=need) == pda.pda.PDA_ERR_ALIGNMENT


def test_append_and_graph_validation():
    lib = pda.load_library()
    p = prob()
    args = [0x1000] * 6
    f = lib.pda_append_kv
    assert f(ctypes.byref(p), None, *args[1:], None) == pda.pda.PDA_ERR_NULL
    assert f(ctypes.byref(p), 0x1008, *args[1:], None) == pda.pda.PDA_ERR_ALIGNMENT
    assert f(ctypes.byref(prob(num_query_tokens=-1)), *args, None) == pda.pda.PDA_ERR_SHAPE
    assert f(ctypes.byref(prob(head_dim=96)), *args, None) == pda.pda.PDA_ERR_UNSUPPORTED
    assert f(ctypes.byref(prob(num_seqs=0)), *([None] * 6), None) == pda.pda.PDA_OK
    g = ctypes.c_void_p()
    c = lib.pda_step_graph_create
    assert c(ctypes.byref(p), *([0x1000] * 7), ctypes.c_float(0.1), 0x1000, None, 0,
             ctypes.byref(g)) == pda.pda.PDA_ERR_WORKSPACE
    assert c(ctypes.byref(p), None, *([0x1000] * 6), ctypes.c_float(0.1), 0x1000, None, 0,
             ctypes.byref(g)) == pda.pda.PDA_ERR_NULL
    assert c(ctypes.byref(p), *([0x1000] * 7), ctypes.c_float(0.1), 0x1000, None, 0, None) == pda.pda.PDA_ERR_NULL
    assert g.value is None
    assert lib.pda_step_graph_launch(None, None) == pda.pda.PDA_ERR_NULL
    assert lib.pda_step_graph_destroy(None) == pda.pda.PDA_OK
    # the append folded into the decode step: one new token per sequence only
    da = lib.pda_decode_append
    big = 1 << 30
    assert da(ctypes.byref(prob(num_query_tokens=2)), *([0x1000] * 7), ctypes.c_float(0.1), 0x1000, 0x1000, big,
              None) == pda.pda.PDA_ERR_UNSUPPORTED
    assert da(ctypes.byref(p), 0x1000, None, *([0x1000] * 5), ctypes.c_float(0.1), 0x1000, 0x1000, big,
              None) == pda.pda.PDA_ERR_NULL
    assert da(ctypes.byref(p), *([0x1000] * 7), ctypes.c_float(0.1), 0x1000, None, 0,
              None) == pda.pda.PDA_ERR_WORKSPACE
    assert da(ctypes.byref(prob(num_seqs=0)), *([None] * 7), ctypes.c_float(0.1), None, None, 0, None) == pda.pda.PDA_OK
    # the model-step graph validates every layer before capturing anything
    m = lib.pda_model_step_graph_create
    L = pda.pda.pda_layer_buffers
    two = (L * 2)(L(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000), L(0x1000, 0x1000, None, 0x1000, 0x1000, 0x1000))
    ws = pda.pda_workspace_bytes(p)
    assert m(ctypes.byref(p), 2, two, 0x1000, 0x1000, ctypes.c_float(0.1), 0x1000, ws,
             ctypes.byref(g)) == pda.pda.PDA_ERR_NULL  # layer 1's v_new
    assert m(ctypes.byref(p), 0, two, 0x1000, 0x1000, ctypes.c_float(0.1), 0x1000, ws,
             ctypes.byref(g)) == pda.pda.PDA_ERR_SHAPE
    assert m(ctypes.byref(p), 1, None, 0x1000, 0x1000, ctypes.c_float(0.1), 0x1000, ws,
             ctypes.byref(g)) == pda.pda.PDA_ERR_NULL
    bad = (L * 1)(L(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1004))  # out not 16-byte aligned
    assert m(ctypes.byref(p), 1, bad, 0x1000, 0x1000, ctypes.c_float(0.1), 0x1000, ws,
             ctypes.byref(g)) == pda.pda.PDA_ERR_ALIGNMENT
    assert g.value is None


def test_multi_token_plan():
    # n new tokens per sequence: query chunks of min(n, 16 // G) tokens; one
    # work item per (partition, sequence, KV head, group of chunks): up to 4,
    # up to 8 when there are more than 4, up to 16 when there are more than 8
    d = pda.pda_plan(llama(num_query_tokens=4, partition_tokens=4096))     # G = 4: one chunk
    assert d["workspace_bytes"] == 256 * 8 * 4
    d = pda.pda_plan(llama(num_query_tokens=7, partition_tokens=4096))     # two chunks, one item
    assert d["workspace_bytes"] == 256 * 8 * 4
    d = pda.pda_plan(llama(num_query_tokens=17, partition_tokens=4096))    # five chunks: one item of up to 8
    assert d["workspace_bytes"] == 256 * 8 * 4
    d = pda.pda_plan(llama(num_query_tokens=33, partition_tokens=4096))    # nine chunks: one item of up to 16
    assert d["workspace_bytes"] == 256 * 8 * 4
    d = pda.pda_plan(llama(num_query_tokens=68, partition_tokens=4096))    # seventeen chunks, two items
    assert d["workspace_bytes"] == 256 * 8 * 2 * 4
    d = pda.pda_plan(llama(num_query_tokens=4, partition_tokens=2048))     # 2 partitions: partials per row
    assert d["workspace_bytes"] == 256 * 4 * 32 * 2 * (128 + 2) * 4 + 2 * 256 * 8 * 4
    assert pda.pda_plan(llama(num_query_tokens=0)) == pda.pda_plan(llama(num_query_tokens=1))


def test_shared_prefix_validation():
    G = pda.pda.make_prefix_groups
    ok = dict(num_groups=3, max_group_size=8, max_prefix_len=256, group_start=0x1000, group_prefix_len=0x1000)

    def plan(p=None, **kw):
        return pda.pda.load_library().pda_plan_shared_prefix(
            ctypes.byref(p or llama()), ctypes.byref(G(**dict(ok, **kw))), ctypes.byref(pda.pda_plan_info()))
    assert plan() == pda.pda.PDA_OK
    assert plan(num_groups=-1) == pda.pda.PDA_ERR_SHAPE
    assert plan(max_group_size=0) == pda.pda.PDA_ERR_SHAPE
    assert plan(max_prefix_len=100) == pda.pda.PDA_ERR_SHAPE        # not a multiple of 16
    assert plan(max_prefix_len=8192) == pda.pda.PDA_ERR_SHAPE       # beyond max_context_len
    # groups of more than 64 / (n G) members take several row groups
    assert plan(max_group_size=17) == pda.pda.PDA_OK                # 17 x G=4 rows: 2 row groups of 16 members
    # huge bounds count at most B members per group (no wrap: 2^30 x 4 = 2^32 -> 0 in 32 bits)
    assert plan(max_group_size=1 << 30) == pda.pda.PDA_OK
    assert plan(llama(num_q_heads=16, num_kv_heads=1), max_group_size=(1 << 28) + 2) == pda.pda.PDA_OK
    # n new tokens per sequence: one member's n x G rows must fit the 64 of an item
    assert plan(llama(num_query_tokens=2)) == pda.pda.PDA_OK                        # 8 x 2 x 4 = 64
    assert plan(llama(num_query_tokens=3)) == pda.pda.PDA_OK                        # 5 members per row group
    assert plan(llama(num_query_tokens=16), max_group_size=4) == pda.pda.PDA_OK     # 16 x 4 = 64
    assert plan(llama(num_query_tokens=17), max_group_size=1) == pda.pda.PDA_ERR_UNSUPPORTED  # 68
    assert plan(llama(num_q_heads=16, num_kv_heads=1, num_query_tokens=5)) == pda.pda.PDA_ERR_UNSUPPORTED  # 80
    assert plan(llama(num_query_tokens=1 << 29), max_group_size=8) == pda.pda.PDA_ERR_SHAPE  # rows overflow
    # items beyond int32: groups x prefix partitions x row groups x KV heads
    big = llama(num_seqs=1 << 20, max_context_len=1 << 20, max_blocks_per_seq=1 << 16, partition_tokens=16)
    assert plan(big, num_groups=1 << 20, max_group_size=1 << 20, max_prefix_len=1 << 20) == pda.pda.PDA_ERR_SHAPE
    d = pda.pda_plan_shared_prefix(llama(num_query_tokens=2, partition_tokens=1024), G(**ok))
    assert d["workspace_bytes"] == (256 * 2 * 32 * (1 + 4) * (128 + 2) * 4 + (4 * 256 * 8 + 3 * 1 * 8) * 4 + 256 * 4)
    # 3 new tokens: 5 members per row group, 8 members -> 2 row groups of prefix items
    d = pda.pda_plan_shared_prefix(llama(num_query_tokens=3, partition_tokens=1024), G(**ok))
    assert d["workspace_bytes"] == (256 * 3 * 32 * (1 + 4) * (128 + 2) * 4 + (4 * 256 * 8 + 3 * 1 * 2 * 8) * 4
                                    + 256 * 4)
    assert plan(group_start=None) == pda.pda.PDA_OK  # planning reads the host bounds only
    assert plan(num_groups=0, group_start=None, group_prefix_len=None) == pda.pda.PDA_OK
    # workspace: (Pp + P) partial states per row, the work order (regular +
    # prefix items) and one int per sequence
    d = pda.pda_plan_shared_prefix(llama(partition_tokens=1024), G(**ok))
    assert d["workspace_bytes"] == (256 * 32 * (1 + 4) * (128 + 2) * 4 + (4 * 256 * 8 + 3 * 1 * 8) * 4 + 256 * 4)
    f = pda.pda.load_library().pda_decode_shared_prefix
    assert f(ctypes.byref(llama()), None, *([0x1000] * 5), ctypes.c_float(1), 0x1000, None, 0,
             None) == pda.pda.PDA_ERR_NULL
    no_arrays = G(**dict(ok, group_start=None))
    assert f(ctypes.byref(llama()), ctypes.byref(no_arrays), *([0x1000] * 5), ctypes.c_float(1), 0x1000, 0x1000,
             1 << 40, None) == pda.pda.PDA_ERR_NULL


def test_validate_host():
    st = W.make_structure("tiny")
    p = prob(num_blocks=st.num_blocks, max_blocks_per_seq=st.max_blocks_per_seq,
             max_context_len=st.max_context_len)
    assert pda.pda_validate_host(p, st.block_table, st.context_lens)[0] == pda.pda.PDA_OK
    bt = st.block_table.copy()
    b = int(np.argmax(st.context_lens))
    bt[b, 3] = st.num_blocks
    rc, bad = pda.pda_validate_host(p, bt, st.context_lens)
    assert rc == pda.pda.PDA_ERR_VALUE and bad == b * st.max_blocks_per_seq + 3
    lens = st.context_lens.copy()
    lens[2] = st.max_context_len + 1
    rc, bad = pda.pda_validate_host(p, st.block_table, lens)
    assert rc == pda.pda.PDA_ERR_VALUE and bad == 2
    # entries past ceil(L/16) are never read and may hold anything
    bt = st.block_table.copy()
    bt[bt < 0] = 999999
    assert pda.pda_validate_host(p, bt, st.context_lens)[0] == pda.pda.PDA_OK


def test_status_strings():
    for s in range(8):
        assert pda.pda_status_string(s).startswith("PDA_")
    assert "unknown" in pda.pda_status_string(99)


def test_binding_has_no_fallback(tmp_path):
    with pytest.raises(RuntimeError, match="no fallback"):
        pda.load_library(str(tmp_path / "missing.so"))


def test_plan_invariants_over_random_descriptors():
    """For seeded random valid descriptors, the library's own partition choice
    covers the longest context, is a multiple of 256 (or the whole context
    rounded to 16) and at most 4608 tokens unless its items hold 64 or more
    query rows (then it is not capped), and the workspace holds the partial
    states (when split) and one order entry per work item."""
    rng = np.random.default_rng(2405)
    for _ in range(400):
        G = int(rng.choice([1, 2, 4, 5, 7, 8, 16]))
        hkv = int(rng.integers(1, 9))
        n = int(rng.choice([1, 1, 2, 4, 8, 16, 33, 70, 512]))
        max_len = int(rng.integers(0, 40000))
        mb = max(1, -(-max_len // 16) + int(rng.integers(0, 4)))
        p = pda.make_problem(int(rng.integers(1, 600)), G * hkv, hkv, int(rng.choice([64, 128])), 1 << 20, mb,
                             max_len, 0, 16, n)
        info = pda.pda_plan(p)
        tp, parts = info["partition_tokens"], info["num_partitions"]
        qc = min(n, 16 // G)
        nqc = -(-n // qc)
        cpg = 16 if nqc > 8 else 8 if nqc > 4 else 4
        wide = min(nqc, cpg) * qc * G >= 64
        assert tp % 16 == 0 and 16 <= tp and (wide or tp <= 4608)
        assert tp % 256 == 0 or tp == -(-max(max_len, 1) // 16) * 16
        assert parts == (-(-max_len // tp) if max_len > 0 else 1)
        assert parts * tp >= max_len
        items = p.num_seqs * hkv * -(-nqc // cpg) * parts
        split = p.num_seqs * n * p.num_q_heads * parts * (p.head_dim + 2) * 4 if parts > 1 else 0
        assert info["workspace_bytes"] == split + items * 4
        assert pda.pda_workspace_bytes(p) == info["workspace_bytes"]


def test_noalloc_host_checks():
    """pda_decode_noalloc's host-side answers, which touch no GPU: descriptor
    errors as pda_decode's, PDA_ERR_SCRATCH for a step whose workspace exceeds
    the static scratch, and nothing to do for an empty batch."""
    f = pda.load_library().pda_decode_noalloc

    def call_na(p):
        return f(ctypes.byref(p), 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, ctypes.c_float(0.125), 0x1000, None)

    assert call_na(llama(head_dim=96)) == pda.pda.PDA_ERR_UNSUPPORTED
    assert call_na(llama(num_q_heads=30)) == pda.pda.PDA_ERR_SHAPE
    big = llama(num_query_tokens=64, partition_tokens=16)
    assert pda.pda_workspace_bytes(big) > pda.pda.PDA_NOALLOC_SCRATCH_BYTES
    assert call_na(big) == pda.pda.PDA_ERR_SCRATCH
    assert call_na(llama(num_seqs=0)) == pda.pda.PDA_OK
    assert "scratch" in pda.pda_status_string(pda.pda.PDA_ERR_SCRATCH)


def test_ceiling_host_checks():
    """The read-ceiling kernels' argument checks (no launch)."""
    lib = pda.load_library()
    g, st = lib.pda_gather_ceiling, lib.pda_stream_ceiling
    assert g(8, 96, 10, 0x1000, 0x1000, 0x1000, 5, 4, 0x1000, None) == pda.pda.PDA_ERR_SHAPE
    assert g(0, 128, 10, 0x1000, 0x1000, 0x1000, 5, 4, 0x1000, None) == pda.pda.PDA_ERR_SHAPE
    assert g(8, 128, 10, 0x1000, 0x1000, None, 5, 4, 0x1000, None) == pda.pda.PDA_ERR_NULL
    assert g(8, 128, 10, 0x1008, 0x1000, 0x1000, 5, 4, 0x1000, None) == pda.pda.PDA_ERR_ALIGNMENT
    assert st(0x1000, 24, 4, 0x1000, None) == pda.pda.PDA_ERR_SHAPE
    assert st(0x1000, 0, 4, 0x1000, None) == pda.pda.PDA_ERR_SHAPE
    assert st(None, 32, 4, 0x1000, None) == pda.pda.PDA_ERR_NULL
    assert st(0x1004, 32, 4, 0x1000, None) == pda.pda.PDA_ERR_ALIGNMENT
