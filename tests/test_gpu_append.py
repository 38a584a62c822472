"""GPU parity of the KV-cache append and of the captured step graph.

The append is byte work: the GPU caches must equal the oracle's bit for bit
(NaN poison included) after storing each sequence's n new tokens at positions
L - n .. L - 1.  The step graph (append + attention captured once) is replayed
several times with fresh inputs written between replays by ordinary eager
work; every replay must equal the same step run eagerly through the C ABI,
bit for bit, and the oracle within the attention tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from paper_2405_11143_amd import StepGraph, make_problem, pda_append_kv, pda_decode, pda_decode_append, pda_plan

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 8e-3, 1e-3


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def bits16(t):
    return W.bf16_bits(t)


@pytest.mark.parametrize("Hq,Hkv,D", [(32, 8, 128), (8, 2, 64), (16, 1, 128)], ids=str)
@pytest.mark.parametrize("n", [1, 3, 16])
def test_append_bit_exact(dev, Hq, Hkv, D, n):
    lens = [0, 1, 2, 15, 16, 17, 31, 32, 33, 200, -3, 1000]
    st = W.custom_structure(len(lens), Hq, Hkv, D, lens, seed=40 + n)
    _, k, v = W.fill_values(st, dev, fill="nan")
    kn, vn = W.fill_new_kv(st, n, dev)
    k_ref, v_ref = oracle.append(bits16(kn), bits16(vn), st.block_table, st.context_lens, bits16(k), bits16(v))
    bt = torch.from_numpy(st.block_table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    pda_append_kv(kn, vn, bt, ln, k, v, max_context_len=st.max_context_len, num_q_heads=Hq)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(k), k_ref), "K cache"
    assert np.array_equal(bits16(v), v_ref), "V cache"


def test_append_full_size(dev):
    """The Llama-3-8B step's append (one new token per sequence) at full size."""
    st = W.make_structure("llama3_8b")
    _, k, v = W.fill_values(st, dev, fill="nan")
    kn, vn = W.fill_new_kv(st, 1, dev)
    k_ref, v_ref = oracle.append(bits16(kn), bits16(vn), st.block_table, st.context_lens, bits16(k), bits16(v))
    pda_append_kv(kn, vn, torch.from_numpy(st.block_table).to(dev), torch.from_numpy(st.context_lens).to(dev),
                  k, v, max_context_len=st.max_context_len, num_q_heads=st.Hq)
    torch.cuda.synchronize()
    assert np.array_equal(bits16(k), k_ref) and np.array_equal(bits16(v), v_ref)


def check(got, ref, what):
    err = np.abs(got.astype(np.float64) - ref)
    print(f"{what}: max-abs {err.max():.3e} mean-abs {err.mean():.3e}", flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, what


GRAPH_CASES = {  # (Hq, Hkv, D, final context lengths, partition_tokens)
    # every work item runs at once: append + partition kernel only
    "small": (8, 2, 64, [50, 100, 17, 230], 0),
    # 64 sequences in 16-token partitions: append, work order, partition and merge kernels
    "split": (32, 8, 128, [int(x) for x in np.random.default_rng(3).integers(40, 700, 64)], 16),
}


@pytest.mark.parametrize("case", sorted(GRAPH_CASES))
@pytest.mark.parametrize("n", [1, 4])
def test_step_graph_replays(dev, n, case):
    """Replays of one captured step, each after new queries, new K/V rows and
    longer contexts were written by eager torch work, against the eager step
    (bitwise) and the oracle."""
    Hq, Hkv, D, final, tp = GRAPH_CASES[case]
    st = W.custom_structure(len(final), Hq, Hkv, D, final, seed=77)
    B = st.B
    growth = np.array([[(s + b) % 4 for b in range(B)] for s in range(4)], dtype=np.int32)  # per replay and sequence
    lens0 = (np.asarray(final) - growth.sum(axis=0)).astype(np.int32)  # every context stays in its blocks
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(lens0).to(dev)
    _, k_g, v_g = W.fill_values(st, dev, fill="nan")
    k_e, v_e = k_g.clone(), v_g.clone()
    q = torch.empty((B, n, st.Hq, st.D), dtype=torch.bfloat16, device=dev)
    kn = torch.empty((B, n, st.Hkv, st.D), dtype=torch.bfloat16, device=dev)
    vn = torch.empty_like(kn)
    graph = StepGraph(q, kn, vn, k_g, v_g, bt, lens, st.scale, max_context_len=st.max_context_len,
                      partition_tokens=tp)
    try:
        for step in range(4):
            # eager work between replays: new inputs, one more token per sequence
            for s_, t in enumerate((q, kn, vn)):
                t.copy_(W.normal_draw(t.shape, 500 + step, s_, dev).to(torch.bfloat16))
            lens.add_(torch.from_numpy(growth[step]).to(dev))
            torch.cuda.synchronize()
            out_g = graph.launch().clone()
            torch.cuda.synchronize()
            # the same step eagerly
            pda_append_kv(kn, vn, bt, lens, k_e, v_e, max_context_len=st.max_context_len, num_q_heads=st.Hq)
            out_e = pda_decode(q, k_e, v_e, bt, lens, st.scale, max_context_len=st.max_context_len,
                               partition_tokens=tp)
            torch.cuda.synchronize()
            assert torch.equal(k_g.view(torch.int16), k_e.view(torch.int16)), f"replay {step}: K cache"
            assert torch.equal(v_g.view(torch.int16), v_e.view(torch.int16)), f"replay {step}: V cache"
            assert torch.equal(out_g, out_e), f"replay {step}: output differs from the eager step"
            lens_h = lens.cpu().numpy()
            ref = oracle.decode_multi(bits16(q), bits16(k_g), bits16(v_g), st.block_table, lens_h, st.scale,
                                      threads=16)
            check(out_g.cpu().numpy(), ref, f"graph replay {step} n={n} {case}")
    finally:
        graph.close()


@pytest.mark.parametrize("case", sorted(GRAPH_CASES))
def test_model_step_graph_replays(dev, case):
    """A 4-layer decode step captured as one graph (per layer: append into its
    own cache, attention; the work order once): replays after eager work
    (new inputs, longer contexts), each against the same layers run eagerly
    (bitwise: caches and outputs of every layer) and layer 3 against the
    oracle."""
    from paper_2405_11143_amd import ModelStepGraph

    Hq, Hkv, D, final, tp = GRAPH_CASES[case]
    n, layers = 1, 4
    st = W.custom_structure(len(final), Hq, Hkv, D, final, seed=78)
    B = st.B
    growth = np.array([[(s + b) % 3 for b in range(B)] for s in range(3)], dtype=np.int32)
    lens0 = (np.asarray(final) - growth.sum(axis=0)).astype(np.int32)
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(lens0).to(dev)
    graph_bufs, eager_caches = [], []
    for l in range(layers):
        _, k, v = W.fill_values(st, dev, fill="nan")
        graph_bufs.append(dict(q=torch.empty((B, n, Hq, D), dtype=torch.bfloat16, device=dev),
                               k_new=torch.empty((B, n, Hkv, D), dtype=torch.bfloat16, device=dev),
                               v_new=torch.empty((B, n, Hkv, D), dtype=torch.bfloat16, device=dev),
                               k_cache=k, v_cache=v,
                               out=torch.empty((B, n, Hq, D), dtype=torch.float32, device=dev)))
        eager_caches.append((k.clone(), v.clone()))
    graph = ModelStepGraph(graph_bufs, bt, lens, st.scale, max_context_len=st.max_context_len, partition_tokens=tp)
    try:
        for step in range(3):
            for li, L in enumerate(graph_bufs):
                for s_, name in enumerate(("q", "k_new", "v_new")):
                    L[name].copy_(W.normal_draw(L[name].shape, 600 + step, 3 * li + s_, dev).to(torch.bfloat16))
            lens.add_(torch.from_numpy(growth[step]).to(dev))
            torch.cuda.synchronize()
            graph.launch()
            torch.cuda.synchronize()
            outs = [L["out"].clone() for L in graph_bufs]
            for l, L in enumerate(graph_bufs):
                k_e, v_e = eager_caches[l]
                pda_append_kv(L["k_new"], L["v_new"], bt, lens, k_e, v_e, max_context_len=st.max_context_len,
                              num_q_heads=Hq)
                out_e = pda_decode(L["q"], k_e, v_e, bt, lens, st.scale, max_context_len=st.max_context_len,
                                   partition_tokens=tp)
                torch.cuda.synchronize()
                assert torch.equal(L["k_cache"].view(torch.int16), k_e.view(torch.int16)), (step, l, "K")
                assert torch.equal(L["v_cache"].view(torch.int16), v_e.view(torch.int16)), (step, l, "V")
                assert torch.equal(outs[l], out_e), (step, l, "output")
            L = graph_bufs[-1]
            ref = oracle.decode_multi(bits16(L["q"]), bits16(L["k_cache"]), bits16(L["v_cache"]), st.block_table,
                                      lens.cpu().numpy(), st.scale, threads=16)
            check(outs[-1].cpu().numpy(), ref, f"model-step graph replay {step} {case}")
    finally:
        graph.close()


@pytest.mark.parametrize("case", ["edge", "split_small", "split_large", "llama3_8b"])
def test_decode_append_matches_two_calls(dev, case):
    """pda_decode_append against pda_append_kv + pda_decode on copies of the
    same caches: caches and outputs bitwise equal.  Small steps (every work
    item at once) fold the append into pass 1: empty and negative lengths, a
    new token that opens a block, a sequence whose new token's block id is
    outside the pool (its append is skipped, its rows are NaN in both), split
    contexts.  Larger steps (split_large, the full Llama-3-8B step) run the
    append kernel first."""
    if case == "llama3_8b":
        st, tp = W.make_structure("llama3_8b"), 0
    else:
        lens = {"edge": [0, 1, 16, 17, 33, -2, 700, 1000, 2049],
                "split_small": [1, 17, 64, 65, 300, 499, 500, 128],
                "split_large": [int(x) for x in np.random.default_rng(5).integers(1, 900, 40)]}[case]
        st = W.custom_structure(len(lens), 32, 8, 128, lens, seed=91)
        tp = 0 if case == "edge" else 64
    plan = pda_plan(make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq,
                                 st.max_context_len, tp))
    items = st.B * st.Hkv * plan["num_partitions"]
    print(f"decode_append {case}: {items} work items ({'folded' if items <= 768 else 'append kernel first'})")
    q, k, v = W.fill_values(st, dev, fill="nan")
    kn, vn = W.fill_new_kv(st, 1, dev)
    table = st.block_table.copy()
    if case == "edge":  # sequence 6's new token lands in a block outside the pool
        table[6, (700 - 1) // 16] = st.num_blocks + 3
    bt = torch.from_numpy(table).to(dev)
    ln = torch.from_numpy(st.context_lens).to(dev)
    k2, v2 = k.clone(), v.clone()
    kw = dict(max_context_len=st.max_context_len, partition_tokens=tp)
    pda_append_kv(kn, vn, bt, ln, k, v, max_context_len=st.max_context_len, num_q_heads=st.Hq)
    ref = pda_decode(q, k, v, bt, ln, st.scale, **kw)
    got = pda_decode_append(q[:, None].contiguous(), kn, vn, k2, v2, bt, ln, st.scale, **kw)
    torch.cuda.synchronize()
    assert torch.equal(k.view(torch.int16), k2.view(torch.int16)), "K cache"
    assert torch.equal(v.view(torch.int16), v2.view(torch.int16)), "V cache"
    got = got[:, 0]
    assert torch.equal(torch.isnan(got), torch.isnan(ref)), "NaN rows"
    assert torch.equal(torch.nan_to_num(got), torch.nan_to_num(ref)), "output"
    if case == "edge":
        assert torch.isnan(got[6]).all() and not torch.isnan(got[7]).any()
