"""Seeded synthetic inputs for paged decode attention.

This module only draws inputs; it holds none of the attention arithmetic.  It
is the one piece shared by the GPU tests, the benchmark and the oracle tests.

A workload has two parts:

* the *structure*, drawn on the host with numpy's counter-based Philox
  generator: context lengths, the block table and the physical block pool;
* the *values* q, K, V, drawn by a counter-based generator written out
  with torch integer ops, so that the same seed gives the same bits on any
  device (``cpu`` for the CPU tests, ``cuda`` for the large configurations,
  where only the device is fast enough): element i of stream (seed, s) is
  the i-th output of SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014) started from a 64-bit key
  of (seed, s), and its top 20 bits pick one of 2^20 equally likely
  standard-normal quantiles (inverse-CDF sampling; |z| <= 4.9).  The
  normal values are rounded to bf16 to nearest even by
  ``Tensor.to(torch.bfloat16)``.

The five named configurations are the rollout decode steps the build is
measured on: the paper's long chain-of-thought rollouts (Section 4.1 uses
inputs of at most 1024 tokens and generations up to 8K tokens, Section 3.2
describes vLLM's PagedAttention with block sharing for parallel sampling)
stand in as Llama-3-shaped synthetic batches, since no model weights or
datasets are available.

Streams of the Philox generator (seed, stream):
    1 lengths, 2 pool permutation, 3 q, 4 K, 5 V, 6 per-head K offset,
    7 multi-token q, 8 new K rows, 9 new V rows, 10 logits, 11 logit
    structure (likely tokens, sampled tokens).

Besides the attention inputs it draws the inputs of the steps around
attention: the new tokens' K/V rows that a step stores in the cache, the
queries of several new tokens per sequence, and LM-head logits with the
sampled token of each row.
Pool blocks that no sequence references, and the slots of a block beyond the
longest context that references it, can be filled with bf16 NaN ("poison")
so that any read of them shows up in the output.

Cache layouts (the library's): V is [num_blocks][Hkv][16][D], one row of D
values per token slot; K is [num_blocks][Hkv][D/8][16][8], each block's keys
split into D/8 chunks of 16 slots x 8 consecutive elements.  Keys are drawn
as rows [num_blocks][Hkv][16][D] and stored through `k_rows_to_cache`.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional, Sequence

import numpy as np

BLOCK_SIZE = 16
_STREAM_LENS, _STREAM_POOL, _STREAM_Q, _STREAM_K, _STREAM_V, _STREAM_KOFF = 1, 2, 3, 4, 5, 6
_STREAM_QMULTI, _STREAM_KNEW, _STREAM_VNEW, _STREAM_LOGITS, _STREAM_LOGIT_STRUCT = 7, 8, 9, 10, 11
_POOL_CHUNK_BLOCKS = 4096  # the value draw walks the pool in fixed chunks (deterministic)


# Named configurations.  `lens` is (kind, lo, hi); `pool` is either a fixed block
# count or the slack factor over the referenced (unique) blocks.
CONFIGS: Dict[str, dict] = {
    "tiny": dict(index=0, B=4, Hq=8, Hkv=2, D=64, lens=("uniform", 1, 257), pool_fixed=128,
                 desc="tiny: B=4, 8 q / 2 kv heads, D=64, L~U[1,257], 128-block pool"),
    "llama3_8b": dict(index=1, B=256, Hq=32, Hkv=8, D=128, lens=("uniform", 512, 4096), pool_slack=1.1,
                      desc="Llama-3-8B decode: B=256, 32 q / 8 kv heads, D=128, L~U[512,4096]"),
    "long_cot": dict(index=2, B=64, Hq=32, Hkv=8, D=128, lens=("loguniform", 1024, 16384), pool_slack=1.1,
                     k_offset_std=0.5,
                     desc="long CoT decode: B=64, 32/8 heads, D=128, L log-uniform [1024,16384], "
                          "per-KV-head K mean offset N(0, 0.5^2)"),
    "llama3_70b_tp8": dict(index=3, B=512, Hq=8, Hkv=1, D=128, lens=("uniform", 1024, 8192), pool_slack=1.1,
                           desc="Llama-3-70B TP=8 one-GPU share: B=512, 8 q / 1 kv head, D=128, L~U[1024,8192]"),
    "shared_prefix": dict(index=4, B=256, Hq=32, Hkv=8, D=128, prompts=32, samples=8, prefix_len=1024,
                          lens=("uniform", 256, 8192), pool_slack=1.1,
                          desc="shared-prefix rollouts: 32 prompts x 8 samples, 1024-token shared prefix "
                               "+ response ~U[256,8192], 32/8 heads, D=128"),
    # The attention shapes of the distilled Qwen models the paper trains on
    # (Table 1): a prompt of up to 1024 tokens plus up to 8K generated ones.
    "r1_qwen7b": dict(index=5, B=256, Hq=28, Hkv=4, D=128, lens=("uniform", 1024, 9216), pool_slack=1.1,
                      desc="long-CoT rollout, DeepSeek-R1-Distill-Qwen-7B attention shape: B=256, "
                           "28 q / 4 kv heads (G=7), D=128, L~U[1024,9216]"),
    "r1_qwen14b": dict(index=6, B=256, Hq=40, Hkv=8, D=128, lens=("uniform", 1024, 9216), pool_slack=1.1,
                       desc="long-CoT rollout, DeepSeek-R1-Distill-Qwen-14B attention shape: B=256, "
                            "40 q / 8 kv heads (G=5), D=128, L~U[1024,9216]"),
    # Chunked prefill (Section 3.2 names it among vLLM's features): a chunk of
    # a prompt's tokens (bench.py --tokens, e.g. 512) attends over the
    # cached context plus itself, causally.
    "chunked_prefill": dict(index=7, B=32, Hq=32, Hkv=8, D=128, lens=("uniform", 1024, 8192), pool_slack=1.1,
                            desc="chunked prefill: B=32, 32 q / 8 kv heads, D=128, contexts L~U[1024,8192] "
                                 "whose last n tokens are the chunk"),
}
CONFIG_NAMES = sorted(CONFIGS, key=lambda n: CONFIGS[n]["index"])


def default_seed(name: str) -> int:
    return 2405 + CONFIGS[name]["index"]


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([int(seed), int(stream)])))


@dataclasses.dataclass
class Structure:
    """Host-side shape of one decode step (everything except q/K/V values)."""
    name: str
    seed: int
    B: int
    Hq: int
    Hkv: int
    D: int
    num_blocks: int
    max_blocks_per_seq: int
    context_lens: np.ndarray   # int32 [B]
    block_table: np.ndarray    # int32 [B][max_blocks_per_seq]; -1 where unused
    k_offset_std: float = 0.0
    block_size: int = BLOCK_SIZE
    # Shared-prefix groups (parallel samples of one prompt), or None: members of
    # group i are sequences [group_start[i], group_start[i+1]), whose first
    # group_prefix_len[i] tokens sit in the same blocks.
    group_start: Optional[np.ndarray] = None       # int32 [num_groups + 1]
    group_prefix_len: Optional[np.ndarray] = None  # int32 [num_groups]

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def scale(self) -> float:
        return float(np.float32(1.0 / math.sqrt(self.D)))

    @property
    def max_context_len(self) -> int:
        return int(max(int(self.context_lens.max(initial=0)), 0))

    def blocks_used(self) -> np.ndarray:
        """Number of block-table entries each sequence reads: ceil(L/16)."""
        L = np.maximum(self.context_lens.astype(np.int64), 0)
        return (L + self.block_size - 1) // self.block_size

    def valid_slots(self) -> np.ndarray:
        """Per physical block, the number of leading slots some sequence reads."""
        valid = np.zeros(self.num_blocks, dtype=np.int64)
        nb = self.blocks_used()
        for b in range(self.B):
            n = int(nb[b])
            if n == 0:
                continue
            j = np.arange(n)
            cnt = np.minimum(self.block_size, int(self.context_lens[b]) - self.block_size * j)
            np.maximum.at(valid, self.block_table[b, :n].astype(np.int64), cnt)
        return valid

    @property
    def logical_tokens(self) -> int:
        return int(np.maximum(self.context_lens.astype(np.int64), 0).sum())

    @property
    def unique_tokens(self) -> int:
        return int(self.valid_slots().sum())

    def algorithmic_bytes(self, unique: bool = True, query_tokens: int = 1) -> int:
        """Bytes an attention step must move: K and V rows of the context (each
        shared physical row once when ``unique``), q and the fp32 output of
        ``query_tokens`` new tokens per sequence, the block-table entries read
        and the context lengths."""
        tokens = self.unique_tokens if unique else self.logical_tokens
        kv = tokens * self.Hkv * self.D * 2 * 2
        q = self.B * query_tokens * self.Hq * self.D * 2
        out = self.B * query_tokens * self.Hq * self.D * 4
        bt = int(self.blocks_used().sum()) * 4
        return int(kv + q + out + bt + self.B * 4)

    def algorithmic_flops(self, query_tokens: int = 1) -> int:
        """Multiply-add work of an attention step, 2 flops each: q.k and p.v
        (D multiply-adds each) per query head and visible context token.  New
        token i of n sees the first L - n + 1 + i tokens of a context of L."""
        n = int(query_tokens)
        lens = np.maximum(self.context_lens.astype(np.int64), 0)
        i = np.arange(n, dtype=np.int64)
        vis = np.clip(lens[:, None] - n + 1 + i[None, :], 0, None).sum()
        return int(vis * self.Hq * 2 * self.D * 2)

    def append_bytes(self, new_tokens: int = 1) -> int:
        """Bytes a KV-cache append must move: the new K and V rows read and
        written once, the block-table entry of each new token, the lengths."""
        rows = self.B * new_tokens * self.Hkv * self.D * 2
        return int(2 * 2 * rows + self.B * new_tokens * 4 + self.B * 4)


def _draw_lens(rng: np.random.Generator, kind: str, lo: int, hi: int, n: int) -> np.ndarray:
    if kind == "uniform":
        return rng.integers(lo, hi, size=n, endpoint=True).astype(np.int32)
    if kind == "loguniform":
        x = np.exp(rng.uniform(math.log(lo), math.log(hi), size=n))
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    raise ValueError(kind)


def make_structure(name: str, seed: Optional[int] = None) -> Structure:
    """The block table, pool size and context lengths of a named configuration."""
    cfg = CONFIGS[name]
    seed = default_seed(name) if seed is None else int(seed)
    B, BS = cfg["B"], BLOCK_SIZE
    kind, lo, hi = cfg["lens"]
    rl = _rng(seed, _STREAM_LENS)
    rp = _rng(seed, _STREAM_POOL)
    if "prompts" in cfg:
        P, S, prefix = cfg["prompts"], cfg["samples"], cfg["prefix_len"]
        assert P * S == B and prefix % BS == 0
        resp = _draw_lens(rl, kind, lo, hi, B)
        lens = (prefix + resp).astype(np.int32)
        mbs = (prefix + hi + BS - 1) // BS
        pre_blocks = prefix // BS
        priv = (resp.astype(np.int64) + BS - 1) // BS
        unique = P * pre_blocks + int(priv.sum())
        num_blocks = int(math.ceil(cfg["pool_slack"] * unique))
        perm = rp.permutation(num_blocks).astype(np.int32)
        table = np.full((B, mbs), -1, dtype=np.int32)
        cur = 0
        for p in range(P):  # each prompt's prefix blocks, shared by its S samples
            ids = perm[cur:cur + pre_blocks]
            cur += pre_blocks
            table[p * S:(p + 1) * S, :pre_blocks] = ids
        for b in range(B):  # private response blocks
            n = int(priv[b])
            table[b, pre_blocks:pre_blocks + n] = perm[cur:cur + n]
            cur += n
        assert cur == unique
        group_start = (np.arange(P + 1) * S).astype(np.int32)
        group_prefix_len = np.full(P, prefix, dtype=np.int32)
    else:
        group_start = group_prefix_len = None
        lens = _draw_lens(rl, kind, lo, hi, B)
        mbs = (hi + BS - 1) // BS
        nblk = (lens.astype(np.int64) + BS - 1) // BS
        total = int(nblk.sum())
        num_blocks = cfg["pool_fixed"] if "pool_fixed" in cfg else int(math.ceil(cfg["pool_slack"] * total))
        assert num_blocks >= total
        perm = rp.permutation(num_blocks).astype(np.int32)
        table = np.full((B, mbs), -1, dtype=np.int32)
        cur = 0
        for b in range(B):
            n = int(nblk[b])
            table[b, :n] = perm[cur:cur + n]
            cur += n
    return Structure(name=name, seed=seed, B=B, Hq=cfg["Hq"], Hkv=cfg["Hkv"], D=cfg["D"],
                     num_blocks=num_blocks, max_blocks_per_seq=int(mbs), context_lens=lens,
                     block_table=table, k_offset_std=float(cfg.get("k_offset_std", 0.0)),
                     group_start=group_start, group_prefix_len=group_prefix_len)


def custom_shared_structure(Hq: int, Hkv: int, D: int, groups: Sequence, loner_lens: Sequence[int] = (),
                            seed: int = 0, pool_slack: float = 1.25, name: str = "custom_shared") -> Structure:
    """Sequences in shared-prefix groups, then sequences in none.  `groups` is
    a list of (prefix_len, [context lengths of the members]): each group's
    prefix_len tokens (a multiple of 16, at most every member's length) sit in
    blocks that all its members' tables share; the rest of every context is
    private.  Blocks are placed by a random permutation of the pool."""
    BS = BLOCK_SIZE
    lens, pre_blocks, group_start, group_prefix = [], [], [0], []
    for prefix_len, members in groups:
        assert prefix_len % BS == 0 and all(L >= prefix_len for L in members) and len(members) > 0
        lens += list(members)
        pre_blocks += [prefix_len // BS] * len(members)
        group_start.append(group_start[-1] + len(members))
        group_prefix.append(prefix_len)
    lens += list(loner_lens)
    pre_blocks += [0] * len(loner_lens)
    B = len(lens)
    lens = np.asarray(lens, dtype=np.int32)
    nblk = (np.maximum(lens.astype(np.int64), 0) + BS - 1) // BS
    unique = sum(prefix_len // BS for prefix_len, _ in groups) + int(sum(nblk - np.asarray(pre_blocks, np.int64)))
    mbs = max(1, int(nblk.max(initial=1)))
    num_blocks = max(1, int(math.ceil(pool_slack * max(unique, 1))))
    perm = _rng(seed, _STREAM_POOL).permutation(num_blocks).astype(np.int32)
    table = np.full((B, mbs), -1, dtype=np.int32)
    cur, b = 0, 0
    for prefix_len, members in groups:
        ids = perm[cur:cur + prefix_len // BS]
        cur += prefix_len // BS
        for _ in members:
            table[b, :len(ids)] = ids
            b += 1
    for b in range(B):
        n0, n = pre_blocks[b], int(nblk[b])
        table[b, n0:n] = perm[cur:cur + n - n0]
        cur += n - n0
    assert cur == unique
    return Structure(name=name, seed=seed, B=B, Hq=Hq, Hkv=Hkv, D=D, num_blocks=num_blocks,
                     max_blocks_per_seq=mbs, context_lens=lens, block_table=table,
                     group_start=np.asarray(group_start, dtype=np.int32),
                     group_prefix_len=np.asarray(group_prefix, dtype=np.int32))


def custom_structure(B: int, Hq: int, Hkv: int, D: int, lens: Sequence[int], seed: int = 0,
                     pool_slack: float = 1.25, max_blocks_per_seq: Optional[int] = None,
                     name: str = "custom") -> Structure:
    """Independent sequences with the given context lengths, each logical block
    mapped to a random physical block of a pool with `pool_slack` spare room."""
    BS = BLOCK_SIZE
    lens = np.asarray(lens, dtype=np.int32)
    assert lens.shape == (B,)
    nblk = (np.maximum(lens.astype(np.int64), 0) + BS - 1) // BS
    total = int(nblk.sum())
    mbs = int(max_blocks_per_seq or max(1, int(nblk.max(initial=1))))
    assert mbs >= int(nblk.max(initial=0))
    num_blocks = max(1, int(math.ceil(pool_slack * max(total, 1))))
    perm = _rng(seed, _STREAM_POOL).permutation(num_blocks).astype(np.int32)
    table = np.full((B, mbs), -1, dtype=np.int32)
    cur = 0
    for b in range(B):
        n = int(nblk[b])
        table[b, :n] = perm[cur:cur + n]
        cur += n
    return Structure(name=name, seed=seed, B=B, Hq=Hq, Hkv=Hkv, D=D, num_blocks=num_blocks,
                     max_blocks_per_seq=mbs, context_lens=lens, block_table=table)


def k_rows_to_cache(k_rows):
    """[NB][Hkv][16][D] key rows -> the cache layout [NB][Hkv][D/8][16][8]
    (numpy array or torch tensor)."""
    NB, H, S, D = k_rows.shape
    x = k_rows.reshape(NB, H, S, D // 8, 8)
    if hasattr(x, "permute"):
        return x.permute(0, 1, 3, 2, 4).contiguous()
    return np.ascontiguousarray(x.transpose(0, 1, 3, 2, 4))


def k_cache_to_rows(k_cache):
    """The cache layout [NB][Hkv][D/8][16][8] -> key rows [NB][Hkv][16][D]."""
    NB, H, C, S, E = k_cache.shape
    if hasattr(k_cache, "permute"):
        return k_cache.permute(0, 1, 3, 2, 4).reshape(NB, H, S, C * E).contiguous()
    return np.ascontiguousarray(k_cache.transpose(0, 1, 3, 2, 4).reshape(NB, H, S, C * E))


# ---- counter-based normal draws (the same bits on every device) ----
_U64 = (1 << 64) - 1
_SM_GAMMA = 0x9E3779B97F4A7C15  # SplitMix64's increment
_SM_M1, _SM_M2 = 0xBF58476D1CE4E5B9, 0x94D049BB133111EB
_NORMAL_BITS = 20
_NORMAL_TABLES: Dict[str, object] = {}


def _i64(c: int) -> int:
    """A 64-bit pattern as the signed int64 torch stores."""
    c &= _U64
    return c - (1 << 64) if c >= (1 << 63) else c


def _lsr(z, k: int):
    """Logical right shift of int64 bit patterns (torch's >> is arithmetic)."""
    return (z >> k) & ((1 << (64 - k)) - 1)


def splitmix64(key: int, index):
    """Output number index + 1 of SplitMix64 started at `key`: mix(key +
    (index + 1) * gamma), on int64 tensors whose bits are the uint64 values
    (multiplications wrap modulo 2^64)."""
    z = (index + 1) * _i64(_SM_GAMMA) + _i64(key)
    z = (z ^ _lsr(z, 30)) * _i64(_SM_M1)
    z = (z ^ _lsr(z, 27)) * _i64(_SM_M2)
    return z ^ _lsr(z, 31)


def normal_table():
    """The 2^20 standard-normal quantiles Phi^-1((j + 1/2) / 2^20) in fp32
    (computed in fp64 on the host)."""
    from scipy.special import ndtri

    n = 1 << _NORMAL_BITS
    return ndtri((np.arange(n, dtype=np.float64) + 0.5) / n).astype(np.float32)


def _table_on(device):
    import torch

    dev = torch.device(device)
    key = str(dev)
    if key not in _NORMAL_TABLES:
        _NORMAL_TABLES[key] = torch.from_numpy(normal_table()).to(dev)
    return _NORMAL_TABLES[key]


def _stream_key(seed: int, stream: int) -> int:
    return int(np.random.SeedSequence([int(seed), int(stream)]).generate_state(1, np.uint64)[0])


def normal_draw(shape, seed: int, stream: int, device="cpu", first: int = 0):
    """fp32 standard-normal values of stream (seed, stream), elements first ..
    first + prod(shape) - 1 in row-major order, the same bits on any device."""
    import torch

    dev = torch.device(device)
    n = int(np.prod(shape, dtype=np.int64))
    idx = torch.arange(first, first + n, dtype=torch.int64, device=dev)
    z = splitmix64(_stream_key(seed, stream), idx)
    return _table_on(dev)[_lsr(z, 64 - _NORMAL_BITS)].reshape(shape)


def fill_values(st: Structure, device="cpu", fill: Optional[str] = "nan"):
    """Draw q [B][Hq][D], the K pool [num_blocks][Hkv][D/8][16][8] and the V pool
    [num_blocks][Hkv][16][D] (bf16) on `device`.  `fill` is 'nan', 'zero' or
    None: what to write into pool slots no sequence reads."""
    import torch

    dev = torch.device(device)
    q = normal_draw((st.B, st.Hq, st.D), st.seed, _STREAM_Q, dev).to(torch.bfloat16)
    mu = None
    if st.k_offset_std:
        mu = normal_draw((st.Hkv, 1, st.D), st.seed, _STREAM_KOFF, dev) * st.k_offset_std
    shape = (st.num_blocks, st.Hkv, st.block_size, st.D)
    per_block = st.Hkv * st.block_size * st.D
    k = torch.empty((st.num_blocks, st.Hkv, st.D // 8, st.block_size, 8), dtype=torch.bfloat16, device=dev)
    v = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    for c0 in range(0, st.num_blocks, _POOL_CHUNK_BLOCKS):
        c1 = min(st.num_blocks, c0 + _POOL_CHUNK_BLOCKS)
        sub = (c1 - c0,) + shape[1:]
        kf = normal_draw(sub, st.seed, _STREAM_K, dev, first=c0 * per_block)
        if mu is not None:
            kf += mu
        k[c0:c1] = k_rows_to_cache(kf.to(torch.bfloat16))
        del kf
        v[c0:c1] = normal_draw(sub, st.seed, _STREAM_V, dev, first=c0 * per_block).to(torch.bfloat16)
    if fill is not None:
        apply_fill(st, k, v, fill)
    return q, k, v


def unread_slot_mask(st: Structure) -> np.ndarray:
    """bool [num_blocks][16]: True for pool slots that no sequence reads."""
    valid = st.valid_slots()
    return np.arange(st.block_size)[None, :] >= valid[:, None]


def apply_fill(st: Structure, k, v, fill: str = "nan"):
    """Overwrite every unread pool slot of k and v (in place) with NaN or zero."""
    import torch

    value = {"nan": float("nan"), "zero": 0.0}[fill]
    mask = torch.from_numpy(unread_slot_mask(st)).to(k.device)
    k.masked_fill_(mask[:, None, None, :, None], value)
    v.masked_fill_(mask[:, None, :, None], value)


def permute_pool(st: Structure, k, v, seed: int):
    """Move every physical block p to pi(p) (new_pool[pi(p)] = pool[p]) and
    rewrite the block table through pi; returns (structure, k, v)."""
    import torch

    pi = _rng(seed, 99).permutation(st.num_blocks).astype(np.int64)
    inv = np.empty_like(pi)
    inv[pi] = np.arange(st.num_blocks)
    idx = torch.from_numpy(inv).to(k.device)
    k2 = k.index_select(0, idx)
    v2 = v.index_select(0, idx)
    table = st.block_table.copy()
    used = table >= 0
    table[used] = pi[table[used]].astype(np.int32)
    return dataclasses.replace(st, block_table=table), k2, v2


def bf16_bits(t) -> np.ndarray:
    """Raw uint16 bit patterns of a bf16 tensor, on the host."""
    import torch

    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def sample_rows(st: Structure, n: int, seed: int = 7) -> np.ndarray:
    """(b, h) pairs for spot checks at full size: the longest and shortest
    sequences, every query head of one sequence, and random pairs."""
    r = _rng(seed, 100)
    L = st.context_lens
    picks = [(int(np.argmax(L)), 0), (int(np.argmax(L)), st.Hq - 1),
             (int(np.argmin(L)), 0), (int(np.argmin(L)), st.Hq - 1)]
    b0 = int(r.integers(0, st.B))
    picks += [(b0, h) for h in range(st.Hq)]
    while len(picks) < n:
        picks.append((int(r.integers(0, st.B)), int(r.integers(0, st.Hq))))
    return np.asarray(picks[:max(n, len(picks))], dtype=np.int32)


def fill_multi_q(st: Structure, n: int, device="cpu"):
    """Queries of n new tokens per sequence: bf16 [B][n][Hq][D], N(0, 1)."""
    import torch

    return normal_draw((st.B, n, st.Hq, st.D), st.seed, _STREAM_QMULTI, device).to(torch.bfloat16)


def fill_new_kv(st: Structure, n: int, device="cpu"):
    """K and V rows of n new tokens per sequence: bf16 [B][n][Hkv][D] each, N(0, 1)."""
    import torch

    shape = (st.B, n, st.Hkv, st.D)
    k = normal_draw(shape, st.seed, _STREAM_KNEW, device)
    v = normal_draw(shape, st.seed, _STREAM_VNEW, device)
    return k.to(torch.bfloat16), v.to(torch.bfloat16)


# LM-head outputs of one decode step (one row per sequence).  The paper's
# rollouts use DeepSeek-R1-distilled Qwen models (Section 4.1); the
# attention configurations above are Llama-3-shaped, so both vocabularies
# appear.
LOGIT_CONFIGS: Dict[str, dict] = {
    "llama3_vocab": dict(index=10, B=256, V=128256,
                         desc="LM-head logits of a Llama-3 decode step: B=256 rows x 128256 vocabulary"),
    "qwen_vocab": dict(index=11, B=256, V=151936,
                       desc="LM-head logits of a Qwen decode step: B=256 rows x 151936 vocabulary"),
    "tiny_vocab": dict(index=12, B=5, V=1000, desc="tiny: 5 rows x 1000 vocabulary"),
    "llama3_vocab_b32": dict(index=13, B=32, V=128256,
                             desc="LM-head logits of a small Llama-3 decode batch: B=32 rows x 128256 vocabulary"),
}


def make_logits(B: int, V: int, seed: int, device="cpu", dtype=None, likely: int = 32,
                background_std: float = 2.0, boost=(6.0, 14.0), p_likely: float = 0.7):
    """Synthetic LM-head logits [B][V] and sampled tokens [B] (int32, host).

    Each row is N(0, background_std^2) noise plus, on `likely` random tokens,
    a boost drawn from U(boost): a peaked distribution with a long flat tail
    like a language model's.  The sampled token is one of the likely tokens
    with probability p_likely, else uniform over the vocabulary.  `dtype` is
    torch.bfloat16 (default) or torch.float32."""
    import torch

    dtype = torch.bfloat16 if dtype is None else dtype
    r = _rng(seed, _STREAM_LOGIT_STRUCT)
    likely_ids = np.stack([r.choice(V, size=min(likely, V), replace=False) for _ in range(B)]) if B else \
        np.zeros((0, min(likely, V)), dtype=np.int64)
    boosts = r.uniform(boost[0], boost[1], size=likely_ids.shape)
    pick_likely = r.random(B) < p_likely
    tokens = np.where(pick_likely, likely_ids[np.arange(B), r.integers(0, likely_ids.shape[1], B)]
                      if B else np.zeros(0, np.int64), r.integers(0, V, B)).astype(np.int32)
    dev = torch.device(device)
    x = normal_draw((B, V), seed, _STREAM_LOGITS, dev) * background_std
    if B:
        rows = torch.arange(B, device=dev)[:, None].expand(B, likely_ids.shape[1])
        x[rows, torch.from_numpy(likely_ids).to(dev)] += torch.from_numpy(boosts).float().to(dev)
    return x.to(dtype), tokens


def logits_for(name: str, device="cpu", dtype=None):
    """make_logits for a named logit configuration (seed 2405 + index)."""
    cfg = LOGIT_CONFIGS[name]
    return make_logits(cfg["B"], cfg["V"], 2405 + cfg["index"], device, dtype)
