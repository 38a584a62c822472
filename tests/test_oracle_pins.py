"""Pins for the fp64 CPU oracle (no GPU).

The oracle is the plain definition of single-query attention over a paged KV
cache (the decode step of the rollout phase the paper runs through vLLM's
PagedAttention: Section 3.2 and Appendix C).  Before it may judge the GPU
path it is pinned here to facts that do not come from its own code:

* hand-worked examples with closed-form answers (tests/golden/hand_worked.json);
* a brute-force dense computation (numpy gather + matrix softmax) on tiny inputs;
* special cases with closed forms: one token returns its V row exactly,
  identical keys or a zero scale give the mean of V, a dominant key returns
  its V row, per-KV-head constant V reveals the query-to-KV head mapping;
* invariants: softmax weights are a probability vector whose ratios are
  exp(score differences), permuting physical blocks leaves the output
  bit-identical, permuting tokens jointly in K and V or shifting every score of
  a head by one constant leaves it unchanged, unread slots never matter,
  the output is linear in V.

Every pin is a function of an oracle object, so ``test_oracle_mutants.py``
can run the same pins against deliberately broken copies of the oracle.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")
TIGHT = 1e-12


# ----------------------------------------------------------------- helpers --

def bits_of(x) -> np.ndarray:
    """bf16 bit patterns of float values that must be exactly representable."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32))
    b = t.to(torch.bfloat16)
    assert torch.equal(b.float(), t) or bool(((b.float() == t) | (t.isnan() & b.float().isnan())).all()), \
        "fixture value not exact in bf16"
    return b.view(torch.int16).numpy().view(np.uint16)


def widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64 (independent of the oracle's C widening)."""
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()


class Case:
    """A decode problem with host bf16 bit arrays."""

    def __init__(self, st: W.Structure, q, k, v, scale=None):
        self.st, self.q, self.k, self.v = st, q, k, v
        self.bt = st.block_table
        self.lens = st.context_lens
        self.scale = st.scale if scale is None else scale

    @classmethod
    def random(cls, B, Hq, Hkv, D, lens, seed=0, fill="nan", **kw):
        st = W.custom_structure(B, Hq, Hkv, D, lens, seed=seed, **kw)
        q, k, v = W.fill_values(st, "cpu", fill=fill)
        return cls(st, W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v))

    def args(self):
        return (self.q, self.k, self.v, self.bt, self.lens, self.scale)

    def run(self, O, threads=1):
        return O.decode(*self.args(), threads=threads)


def dense_reference(case: Case) -> np.ndarray:
    """Brute force: gather each sequence's K/V densely, softmax(scale q K^T) V."""
    q, k, v = widen(case.q), W.k_cache_to_rows(widen(case.k)), widen(case.v)
    B, Hq, D = q.shape
    G = Hq // k.shape[1]
    out = np.zeros((B, Hq, D))
    for b in range(B):
        L = int(case.lens[b])
        if L <= 0:
            continue
        t = np.arange(L)
        phys = case.bt[b][t // 16]
        slot = t % 16
        for h in range(Hq):
            K = k[phys, h // G, slot]   # [L][D]
            V = v[phys, h // G, slot]
            s = case.scale * (K @ q[b, h])
            w = np.exp(s - s.max())
            out[b, h] = (w / w.sum()) @ V
    return out


def load_golden():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def golden_case(c) -> tuple:
    B, Hq, Hkv, D, NB = c["B"], c["Hq"], c["Hkv"], c["D"], c["num_blocks"]
    k = np.full((NB, Hkv, 16, D), np.nan, dtype=np.float32)
    v = np.full((NB, Hkv, 16, D), np.nan, dtype=np.float32)
    for r in c["rows"]:
        k[r["block"], r["head"], r["slot"]] = r["k"]
        v[r["block"], r["head"], r["slot"]] = r["v"]
    q = bits_of(c["q"])
    expected = np.array([[[eval(e, {"__builtins__": {}}, {"e": math.e}) for e in row]
                          for row in seq] for seq in c["expected"]], dtype=np.float64)
    bt = np.asarray(c["block_table"], dtype=np.int32)
    lens = np.asarray(c["context_lens"], dtype=np.int32)
    return (q, bits_of(W.k_rows_to_cache(k)), bits_of(v), bt, lens, float(np.float32(c["scale"]))), expected


# -------------------------------------------------------------------- pins --
# Each pin raises AssertionError (or any exception) when the oracle is wrong.

def pin_golden(O):
    for c in load_golden():
        args, expected = golden_case(c)
        got = O.decode(*args)
        np.testing.assert_allclose(got, expected, rtol=0, atol=1e-15, err_msg=c["name"])


def pin_bruteforce(O):
    shapes = [(1, 1, 1, 8, [37]), (3, 4, 1, 8, [1, 16, 40]), (4, 8, 2, 64, [15, 17, 33, 64]),
              (2, 6, 2, 16, [31, 48]), (2, 16, 2, 64, [64, 5]), (3, 8, 8, 32, [2, 47, 20])]
    for i, (B, Hq, Hkv, D, lens) in enumerate(shapes):
        c = Case.random(B, Hq, Hkv, D, lens, seed=11 + i)
        np.testing.assert_allclose(c.run(O), dense_reference(c), rtol=0, atol=TIGHT,
                                   err_msg=str((B, Hq, Hkv, D, lens)))


def pin_length_one_is_v(O):
    c = Case.random(5, 8, 2, 64, [1] * 5, seed=3)
    out = c.run(O)
    v = widen(c.v)
    for b in range(5):
        p = c.bt[b, 0]
        for h in range(8):
            assert np.array_equal(out[b, h], v[p, h // 4, 0]), (b, h)


def pin_identical_keys_mean(O):
    c = Case.random(3, 4, 2, 16, [5, 16, 33], seed=4)
    k = W.k_cache_to_rows(c.k)
    for b in range(3):  # every key row of (b, g) equal to the first one of (b, g)
        L = int(c.lens[b])
        first = k[c.bt[b, 0], :, 0].copy()
        for t in range(L):
            k[c.bt[b, t // 16], :, t % 16] = first
    c.k = W.k_rows_to_cache(k)
    out = c.run(O)
    v = widen(c.v)
    for b in range(3):
        L = int(c.lens[b])
        t = np.arange(L)
        for h in range(4):
            rows = v[c.bt[b][t // 16], h // 2, t % 16]
            np.testing.assert_allclose(out[b, h], rows.sum(axis=0) / L, rtol=0, atol=TIGHT)


def pin_scale_zero_mean(O):
    c = Case.random(2, 4, 4, 16, [20, 7], seed=5)
    c.scale = 0.0
    out = c.run(O)
    v = widen(c.v)
    for b in range(2):
        L = int(c.lens[b])
        t = np.arange(L)
        for h in range(4):
            np.testing.assert_allclose(out[b, h], v[c.bt[b][t // 16], h, t % 16].mean(axis=0),
                                       rtol=0, atol=TIGHT)


def pin_weights_probability(O):
    c = Case.random(2, 4, 2, 32, [45, 3], seed=6)
    q, k = widen(c.q), W.k_cache_to_rows(widen(c.k))
    for b in range(2):
        for h in range(4):
            w = O.weights(*c.args(), b, h)
            L = int(c.lens[b])
            assert w.shape == (L,) and np.all(w >= 0)
            assert abs(w.sum() - 1.0) <= TIGHT
            # ratio of two weights is exp of the score difference
            t0, t1 = 0, L - 1
            s0 = c.scale * float(np.dot(q[b, h], k[c.bt[b, t0 // 16], h // 2, t0 % 16]))
            s1 = c.scale * float(np.dot(q[b, h], k[c.bt[b, t1 // 16], h // 2, t1 % 16]))
            assert math.isclose(w[t1] / w[t0], math.exp(s1 - s0), rel_tol=1e-12)


def pin_dominant_key(O):
    """A key whose score exceeds the rest by ~1000 takes all the weight (and an
    implementation that skips the max subtraction overflows here)."""
    c = Case.random(1, 1, 1, 8, [21], seed=7)
    q = np.zeros((1, 1, 8), np.float32)
    q[0, 0, 0] = 64.0
    k = np.zeros((c.st.num_blocks, 1, 16, 8), np.float32)
    t_hot = 13
    k[c.bt[0, t_hot // 16], 0, t_hot % 16, 0] = 128.0
    c.q, c.k, c.scale = bits_of(q), bits_of(W.k_rows_to_cache(k)), 0.125
    out = c.run(O)
    assert np.array_equal(out[0, 0], widen(c.v)[c.bt[0, t_hot // 16], 0, t_hot % 16])


def pin_gqa_mapping(O):
    for (Hq, Hkv) in [(8, 2), (6, 3), (8, 1), (4, 4)]:
        c = Case.random(2, Hq, Hkv, 16, [19, 40], seed=8)
        v = np.zeros((c.st.num_blocks, Hkv, 16, 16), np.float32)
        for g in range(Hkv):
            v[:, g] = g + 1
        c.v = bits_of(v)
        out = c.run(O)
        G = Hq // Hkv
        for h in range(Hq):
            np.testing.assert_allclose(out[:, h], h // G + 1, rtol=0, atol=TIGHT)


def pin_block_shuffle(O):
    st = W.custom_structure(3, 8, 2, 64, [30, 64, 7], seed=9)
    q, k, v = W.fill_values(st, "cpu", fill="nan")
    st2, k2, v2 = W.permute_pool(st, k, v, seed=1)
    assert not np.array_equal(st.block_table, st2.block_table)
    a = Case(st, W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)).run(O)
    b = Case(st2, W.bf16_bits(q), W.bf16_bits(k2), W.bf16_bits(v2)).run(O)
    assert np.array_equal(a, b)


def pin_token_permutation(O):
    c = Case.random(1, 4, 2, 16, [37], seed=10)
    out = c.run(O)
    L = 37
    perm = np.random.default_rng(0).permutation(L)
    k0 = W.k_cache_to_rows(c.k)
    k, v = k0.copy(), c.v.copy()
    for t in range(L):  # token t takes the K/V row of token perm[t]
        s = perm[t]
        k[c.bt[0, t // 16], :, t % 16] = k0[c.bt[0, s // 16], :, s % 16]
        v[c.bt[0, t // 16], :, t % 16] = c.v[c.bt[0, s // 16], :, s % 16]
    c.k, c.v = W.k_rows_to_cache(k), v
    np.testing.assert_allclose(c.run(O), out, rtol=0, atol=TIGHT)


def pin_uniform_shift(O):
    """Adding one vector mu to every key of a KV head shifts all scores of each
    of its query heads by scale*q.mu, which the softmax cancels.  Keys and mu
    are multiples of 1/8 so that k + mu stays exact in bf16."""
    st = W.custom_structure(2, 4, 2, 16, [29, 50], seed=12)
    r = np.random.default_rng(1)
    k = r.integers(-32, 33, size=(st.num_blocks, 2, 16, 16)).astype(np.float32) / 8
    mu = r.integers(-16, 17, size=(1, 2, 1, 16)).astype(np.float32) / 8
    q, _, v = W.fill_values(st, "cpu", fill=None)
    base = Case(st, W.bf16_bits(q), bits_of(W.k_rows_to_cache(k)), W.bf16_bits(v)).run(O)
    shifted = Case(st, W.bf16_bits(q), bits_of(W.k_rows_to_cache(k + mu)), W.bf16_bits(v)).run(O)
    np.testing.assert_allclose(shifted, base, rtol=0, atol=1e-9)


def pin_unread_slots(O):
    st = W.custom_structure(3, 4, 2, 32, [17, 1, 40], seed=13)
    outs = []
    for fill in ("nan", "zero", None):
        q, k, v = W.fill_values(st, "cpu", fill=fill)
        outs.append(Case(st, W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)).run(O))
    assert np.all(np.isfinite(outs[0]))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def pin_nonpositive_length(O):
    c = Case.random(3, 2, 1, 8, [0, 5, -3], seed=14)
    out = c.run(O)
    assert np.all(out[0] == 0) and np.all(out[2] == 0) and np.any(out[1] != 0)


def pin_linear_in_v(O):
    st = W.custom_structure(2, 4, 2, 16, [23, 9], seed=15)
    r = np.random.default_rng(2)
    v1 = r.integers(-64, 65, size=(st.num_blocks, 2, 16, 16)).astype(np.float32) / 16
    v2 = r.integers(-64, 65, size=(st.num_blocks, 2, 16, 16)).astype(np.float32) / 16
    q, k, _ = W.fill_values(st, "cpu", fill=None)
    mk = lambda vv: Case(st, W.bf16_bits(q), W.bf16_bits(k), bits_of(vv)).run(O)
    np.testing.assert_allclose(mk(v1 + v2), mk(v1) + mk(v2), rtol=0, atol=1e-12)


def pin_rows_and_threads(O):
    c = Case.random(4, 8, 2, 64, [3, 100, 57, 16], seed=16)
    full = c.run(O, threads=1)
    assert np.array_equal(full, c.run(O, threads=3))
    rows = np.array([[1, 7], [0, 0], [3, 4], [1, 0]], np.int32)
    part = O.decode_rows(*c.args(), rows)
    for i, (b, h) in enumerate(rows):
        assert np.array_equal(part[i], full[b, h])


PINS = [pin_golden, pin_bruteforce, pin_length_one_is_v, pin_identical_keys_mean,
        pin_scale_zero_mean, pin_weights_probability, pin_dominant_key, pin_gqa_mapping,
        pin_block_shuffle, pin_token_permutation, pin_uniform_shift, pin_unread_slots,
        pin_nonpositive_length, pin_linear_in_v, pin_rows_and_threads]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle._load())


def test_rejects_bad_block_ids():
    c = Case.random(2, 2, 1, 8, [20, 4], seed=17)
    bt = c.bt.copy()
    bt[0, 1] = c.st.num_blocks  # out of the pool
    with pytest.raises(ValueError):
        oracle.decode(c.q, c.k, c.v, bt, c.lens, c.scale)
    bt = c.bt.copy()
    bt[1, 0] = -1
    with pytest.raises(ValueError):
        oracle.decode(c.q, c.k, c.v, bt, c.lens, c.scale)
    lens = c.lens.copy()
    lens[1] = 16 * c.bt.shape[1] + 1  # beyond the block table
    with pytest.raises(ValueError):
        oracle.decode(c.q, c.k, c.v, c.bt, lens, c.scale)
