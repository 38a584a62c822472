"""The seeded input generator (no GPU): determinism, shapes, block tables,
prefix sharing, poison fill, bf16 rounding, and the counter-based value draw
(SplitMix64 against an independent uint64 implementation and its published
first output, the normal quantile table, chunked draws)."""
import math

import numpy as np
import pytest
import torch

import workloads as W


@pytest.mark.parametrize("name", W.CONFIG_NAMES)
def test_structure_is_deterministic_and_valid(name):
    a, b = W.make_structure(name), W.make_structure(name)
    assert np.array_equal(a.context_lens, b.context_lens)
    assert np.array_equal(a.block_table, b.block_table)
    cfg = W.CONFIGS[name]
    kind, lo, hi = cfg["lens"]
    L = a.context_lens
    if "prefix_len" in cfg:
        assert L.min() >= cfg["prefix_len"] + lo and L.max() <= cfg["prefix_len"] + hi
    else:
        assert L.min() >= lo and L.max() <= hi
    assert a.max_context_len <= 16 * a.max_blocks_per_seq
    nb = a.blocks_used()
    for s in range(a.B):
        row = a.block_table[s]
        assert np.all(row[:nb[s]] >= 0) and np.all(row[:nb[s]] < a.num_blocks)
        assert np.all(row[nb[s]:] == -1)
    c = W.make_structure(name, seed=a.seed + 1000)
    assert not np.array_equal(a.context_lens, c.context_lens)


@pytest.mark.parametrize("name", ["llama3_8b", "long_cot", "llama3_70b_tp8"])
def test_private_pools_have_ten_percent_slack(name):
    st = W.make_structure(name)
    used = st.block_table[st.block_table >= 0]
    assert len(np.unique(used)) == used.size  # no block referenced twice
    assert st.num_blocks == math.ceil(1.1 * used.size)


def test_tiny_pool_is_fixed():
    st = W.make_structure("tiny")
    assert st.num_blocks == 128 and (st.B, st.Hq, st.Hkv, st.D) == (4, 8, 2, 64)


def test_shared_prefix_pattern():
    st = W.make_structure("shared_prefix")
    pre = 1024 // 16
    t = st.block_table
    prefixes = []
    for p in range(32):
        rows = t[p * 8:(p + 1) * 8, :pre]
        assert np.all(rows == rows[0])  # the prompt's 8 samples share its prefix
        prefixes.append(rows[0])
    prefixes = np.concatenate(prefixes)
    assert len(np.unique(prefixes)) == prefixes.size  # prompts do not share
    priv = np.concatenate([t[b, pre:st.blocks_used()[b]] for b in range(st.B)])
    assert len(np.unique(priv)) == priv.size
    assert not set(priv.tolist()) & set(prefixes.tolist())
    unique_blocks = prefixes.size + priv.size
    assert st.num_blocks == math.ceil(1.1 * unique_blocks)
    # unique bytes count each shared prefix row once
    assert st.unique_tokens == st.logical_tokens - 7 * 32 * 1024


def test_values_are_deterministic_and_poisoned():
    st = W.make_structure("tiny")
    q1, k1, v1 = W.fill_values(st, "cpu")
    q2, k2, v2 = W.fill_values(st, "cpu")
    for a, b in ((q1, q2), (k1, k2), (v1, v2)):
        assert a.dtype == torch.bfloat16
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    mask = torch.from_numpy(W.unread_slot_mask(st))
    assert k1.shape == (st.num_blocks, 2, 8, 16, 8) and v1.shape == (st.num_blocks, 2, 16, 64)
    assert torch.isnan(k1.float()).any(dim=(1, 2, 4)).eq(mask).all()
    assert torch.isnan(v1.float()).all(dim=(1, 3)).eq(mask).all()
    # read slots hold N(0,1) draws
    read = W.k_cache_to_rows(k1).float().permute(0, 2, 1, 3)[~mask]
    assert torch.isfinite(read).all() and abs(read.mean().item()) < 0.1 and abs(read.std().item() - 1) < 0.1


def _splitmix64_uint64(key: int, n: int) -> np.ndarray:
    """SplitMix64 outputs 1..n from `key`, in numpy uint64 arithmetic (which
    wraps modulo 2^64): state += gamma, then the two xor-shift-multiply
    rounds and a final xor-shift."""
    out = np.empty(n, dtype=np.uint64)
    state = np.uint64(key)
    with np.errstate(over="ignore"):
        for i in range(n):
            state = state + np.uint64(0x9E3779B97F4A7C15)
            z = state
            z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
            z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
            out[i] = z ^ (z >> np.uint64(31))
    return out


def test_splitmix64_matches_uint64_reference():
    # the first output of SplitMix64 seeded with 0, as its reference code prints it
    assert int(W.splitmix64(0, torch.tensor([0])).numpy().view(np.uint64)[0]) == 0xE220A8397B1DCDAF
    for key in (0, 1, 2**63 + 12345, W._stream_key(2406, 4)):
        got = W.splitmix64(key, torch.arange(300, dtype=torch.int64)).numpy().view(np.uint64)
        assert np.array_equal(got, _splitmix64_uint64(key, 300))


def test_normal_table_is_the_quantiles():
    t = W.normal_table()
    n = t.size
    assert n == 1 << 20 and t.dtype == np.float32
    assert np.all(np.diff(t) > 0) and np.array_equal(t, -t[::-1])  # increasing, symmetric
    from statistics import NormalDist
    for j in (0, 1, 1000, n // 2 - 1, n - 5):
        assert abs(float(t[j]) - NormalDist().inv_cdf((j + 0.5) / n)) < 1e-6 * max(1.0, abs(float(t[j])))
    assert abs(float(t.astype(np.float64).mean())) < 1e-9
    assert abs(float((t.astype(np.float64) ** 2).mean()) - 1) < 2e-4  # the discrete draw's variance


def test_normal_draw_chunks_and_streams():
    full = W.normal_draw((7, 300), 11, 4)
    part = W.normal_draw((3, 300), 11, 4, first=4 * 300)
    assert torch.equal(full[4:], part)  # element i of a stream does not depend on the chunking
    other = W.normal_draw((7, 300), 11, 5)
    assert not torch.equal(full, other)
    x = W.normal_draw((1 << 18,), 1, 3).double()
    assert abs(x.mean().item()) < 0.01 and abs(x.std().item() - 1) < 0.01


def test_bf16_rounds_to_nearest_even():
    x = torch.tensor([1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-8 + 2**-20, -(1 + 2**-8)], dtype=torch.float32)
    got = x.to(torch.bfloat16).float().tolist()
    assert got == [1.0, 1 + 2**-6, 1 + 2**-7, -1.0]


def test_k_layout_round_trip():
    rows = np.arange(3 * 2 * 16 * 24, dtype=np.float32).reshape(3, 2, 16, 24)
    cache = W.k_rows_to_cache(rows)
    assert cache.shape == (3, 2, 3, 16, 8)
    # key d of slot o of block p, head g sits at [p][g][d // 8][o][d % 8]
    for (p, g, o, d) in [(0, 0, 0, 0), (2, 1, 15, 23), (1, 0, 7, 9), (1, 1, 3, 16)]:
        assert cache[p, g, d // 8, o, d % 8] == rows[p, g, o, d]
    assert np.array_equal(W.k_cache_to_rows(cache), rows)
    t = torch.from_numpy(rows)
    assert torch.equal(W.k_rows_to_cache(t), torch.from_numpy(cache))
    assert torch.equal(W.k_cache_to_rows(W.k_rows_to_cache(t)), t)


def test_permute_pool_moves_blocks():
    st = W.custom_structure(2, 2, 1, 8, [20, 33], seed=3)
    q, k, v = W.fill_values(st, "cpu")
    st2, k2, v2 = W.permute_pool(st, k, v, seed=5)
    for b in range(2):
        for j in range(st.blocks_used()[b]):
            a = k[st.block_table[b, j]].view(torch.int16)
            c = k2[st2.block_table[b, j]].view(torch.int16)
            assert torch.equal(a, c)


def test_algorithmic_bytes_llama3_8b():
    st = W.make_structure("llama3_8b")
    kv = st.logical_tokens * 8 * 128 * 2 * 2
    assert st.algorithmic_bytes() == kv + 256 * 32 * 128 * 6 + int(st.blocks_used().sum()) * 4 + 256 * 4
    assert 2.2e9 < st.algorithmic_bytes() < 2.7e9
