"""Pins for the fp64 CPU oracle (no GPU).

The oracle is the plain definition of attention over a paged KV cache (the
decode step of the rollout phase the paper runs through vLLM's
PagedAttention: Section 3.2 and Appendix C), also with several causal query
tokens per sequence, of storing new tokens in the cache, and of token
log-probabilities and entropies.  Before it may judge the GPU path it is
pinned here to facts that do not come from its own code:

* hand-worked examples with closed-form answers (tests/golden/hand_worked.json);
* a brute-force dense computation (numpy gather + matrix softmax) on tiny inputs;
* special cases with closed forms: one token returns its V row exactly,
  identical keys or a zero scale give the mean of V, a dominant key returns
  its V row, per-KV-head constant V reveals the query-to-KV head mapping;
* invariants: softmax weights are a probability vector whose ratios are
  exp(score differences), permuting physical blocks leaves the output
  bit-identical, permuting tokens jointly in K and V or shifting every score of
  a head by one constant leaves it unchanged, unread slots never matter,
  the output is linear in V;
* several query tokens: a dense causal brute force, each row equals the
  one-token step over its visible prefix, keys after a row's position never
  reach it;
* append: rows land where the generator's own layout conversion says, nothing
  else changes, appending a context token by token rebuilds the pool, a
  one-token context then decodes to the new V row exactly;
* log-probabilities: uniform and two-point closed forms, numpy's logaddexp
  and -sum p log p, probabilities summing to one, shift invariance, no
  overflow, masked tokens.

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


# ------------------------------------------- several query tokens per step --

def multi_case(B, Hq, Hkv, D, lens, n, seed, fill="nan"):
    c = Case.random(B, Hq, Hkv, D, lens, seed=seed, fill=fill)
    c.q = W.bf16_bits(W.fill_multi_q(c.st, n))
    return c


def dense_multi_reference(case: Case) -> np.ndarray:
    """Brute force: new token i of a sequence with L tokens sits at position
    L - n + i and sees positions 0 .. L - n + i (a causal mask over the dense
    gathered K/V)."""
    q, k, v = widen(case.q), W.k_cache_to_rows(widen(case.k)), widen(case.v)
    B, n, Hq, D = q.shape
    G = Hq // k.shape[1]
    out = np.zeros((B, n, Hq, D))
    for b in range(B):
        L = int(case.lens[b])
        t = np.arange(max(L, 0))
        phys, slot = case.bt[b][t // 16], t % 16
        for i in range(n):
            visible = t <= L - n + i
            if L <= 0 or not visible.any():
                continue
            for h in range(Hq):
                K, V = k[phys, h // G, slot], v[phys, h // G, slot]
                s = case.scale * (K @ q[b, i, h])
                s = np.where(visible, s, -np.inf)
                w = np.exp(s - s.max())
                out[b, i, h] = (w / w.sum()) @ V
    return out


def pin_multi_bruteforce(O):
    for j, (B, Hq, Hkv, D, lens, n) in enumerate([(3, 4, 1, 16, [5, 16, 40], 4), (2, 8, 2, 64, [33, 17], 2),
                                                   (2, 2, 2, 8, [3, 20], 5), (1, 16, 1, 32, [64], 1)]):
        c = multi_case(B, Hq, Hkv, D, lens, n, seed=40 + j)
        got = O.decode_multi(*c.args())
        np.testing.assert_allclose(got, dense_multi_reference(c), rtol=0, atol=TIGHT,
                                   err_msg=str((B, Hq, Hkv, D, lens, n)))


def pin_multi_rows_are_decode_steps(O):
    """Row i of a step with n new tokens is exactly the one-token decode step
    of the same query over the first L - n + 1 + i tokens (bitwise), and n = 1
    is the decode step itself."""
    c = multi_case(3, 8, 2, 32, [9, 31, 50], 3, seed=44)
    multi = O.decode_multi(*c.args())
    for i in range(3):
        lens_i = c.lens - 3 + 1 + i
        one = O.decode(np.ascontiguousarray(c.q[:, i]), c.k, c.v, c.bt, lens_i, c.scale)
        assert np.array_equal(multi[:, i], one), i
    single = multi_case(3, 8, 2, 32, [9, 31, 50], 1, seed=44)
    assert np.array_equal(O.decode_multi(*single.args())[:, 0],
                          O.decode(np.ascontiguousarray(single.q[:, 0]), *single.args()[1:]))


def pin_multi_causal(O):
    """Keys and values after a token's own position never reach its row:
    NaN there leaves rows before it bit-identical and finite."""
    c = multi_case(2, 4, 2, 16, [20, 37], 4, seed=45, fill=None)
    base = O.decode_multi(*c.args())
    k, v = W.k_cache_to_rows(widen(c.k)), widen(c.v)
    for b in range(2):
        L = int(c.lens[b])
        t = L - 1  # the last new token's position: only row n-1 may see it
        k[c.bt[b, t // 16], :, t % 16] = np.nan
        v[c.bt[b, t // 16], :, t % 16] = np.nan
    c.k, c.v = bits_of(W.k_rows_to_cache(k)), bits_of(v)
    got = O.decode_multi(*c.args())
    assert np.array_equal(got[:, :3], base[:, :3]) and np.all(np.isfinite(got[:, :3]))
    assert np.all(np.isnan(got[:, 3]))


def pin_multi_rows_subset(O):
    c = multi_case(3, 4, 2, 16, [7, 30, 2], 3, seed=46)
    full = O.decode_multi(*c.args(), threads=2)
    rows = np.array([[1, 2, 3], [0, 0, 0], [2, 0, 1], [2, 2, 2]], np.int32)
    part = O.decode_multi_rows(*c.args(), rows)
    for r, (b, i, h) in enumerate(rows):
        assert np.array_equal(part[r], full[b, i, h])
    # sequence 2 has L = 2 < n = 3: its first new token sees nothing
    assert np.all(full[2, 0] == 0) and np.any(full[2, 1] != 0)


# ------------------------------------------------------- KV-cache append --

def append_case(B, Hkv, D, lens, n, seed):
    st = W.custom_structure(B, 2 * Hkv, Hkv, D, lens, seed=seed)
    _, k, v = W.fill_values(st, "cpu", fill="nan")
    kn, vn = W.fill_new_kv(st, n)
    return st, W.bf16_bits(k), W.bf16_bits(v), W.bf16_bits(kn), W.bf16_bits(vn)


def pin_append_places_rows(O):
    """Each new row lands at position L - n + i: read back through the
    generator's own layout conversion it equals the input row, and every
    other element of both pools is unchanged (bitwise)."""
    for (B, Hkv, D, lens, n) in [(4, 2, 64, [1, 16, 17, 40], 1), (3, 1, 16, [5, 32, 33], 3),
                                 (2, 4, 32, [2, 20], 4)]:
        st, k, v, kn, vn = append_case(B, Hkv, D, lens, n, seed=50 + n)
        k2, v2 = O.append(kn, vn, st.block_table, st.context_lens, k, v)
        kr, kr2 = W.k_cache_to_rows(k), W.k_cache_to_rows(k2)
        touched = np.zeros((st.num_blocks, 16), bool)
        for b in range(B):
            for i in range(n):
                t = int(st.context_lens[b]) - n + i
                if t < 0:
                    continue
                p, o = st.block_table[b, t // 16], t % 16
                assert np.array_equal(kr2[p, :, o], kn[b, i]) and np.array_equal(v2[p, :, o], vn[b, i])
                touched[p, o] = True
        same = ~touched[:, None, :, None]
        assert np.array_equal(np.where(same, kr2, 0), np.where(same, kr, 0))
        assert np.array_equal(np.where(same, v2, 0), np.where(same, v, 0))
        assert np.array_equal(np.isnan(widen(kr2)) & same, np.isnan(widen(kr)) & same)


def pin_append_builds_the_cache(O):
    """Appending a context token by token (n = 1) or chunk by chunk (n = 5)
    into an all-NaN pool rebuilds the generator's pool on every slot a
    sequence uses."""
    st = W.custom_structure(3, 4, 2, 32, [23, 40, 9], seed=55)
    _, k, v = W.fill_values(st, "cpu", fill="nan")
    kb, vb = W.bf16_bits(k), W.bf16_bits(v)
    krows = W.k_cache_to_rows(kb)
    for n in (1, 5):
        k_cur = np.full_like(kb, 0x7FC0)
        v_cur = np.full_like(vb, 0x7FC0)
        Lmax = int(st.context_lens.max())
        for end in range(n, ((Lmax + n - 1) // n) * n + 1, n):
            lens = np.minimum(st.context_lens, end).astype(np.int32)
            kn = np.zeros((st.B, n, st.Hkv, st.D), np.uint16)
            vn = np.zeros_like(kn)
            for b in range(st.B):
                for i in range(n):
                    t = int(lens[b]) - n + i
                    if t >= 0:
                        p, o = st.block_table[b, t // 16], t % 16
                        kn[b, i], vn[b, i] = krows[p, :, o], vb[p, :, o]
            k_cur, v_cur = O.append(kn, vn, st.block_table, lens, k_cur, v_cur)
        mask = ~W.unread_slot_mask(st)
        assert np.array_equal(W.k_cache_to_rows(k_cur)[mask.nonzero()[0], :, mask.nonzero()[1]],
                              krows[mask.nonzero()[0], :, mask.nonzero()[1]]), n
        assert np.array_equal(v_cur[mask.nonzero()[0], :, mask.nonzero()[1]],
                              vb[mask.nonzero()[0], :, mask.nonzero()[1]]), n


def pin_append_then_decode(O):
    """After storing a one-token context, the decode step returns the new V row
    exactly (closed form)."""
    st, k, v, kn, vn = append_case(4, 2, 64, [1, 1, 1, 1], 1, seed=56)
    k2, v2 = O.append(kn, vn, st.block_table, st.context_lens, k, v)
    q = W.bf16_bits(W.fill_multi_q(st, 1)[:, 0].contiguous())
    out = O.decode(q, k2, v2, st.block_table, st.context_lens, st.scale)
    for b in range(4):
        for h in range(st.Hq):
            assert np.array_equal(out[b, h], widen(vn[b, 0, h // st.G]))


def pin_append_skips_and_rejects(O):
    st, k, v, kn, vn = append_case(3, 1, 16, [0, 2, -4], 3, seed=57)
    k2, v2 = O.append(kn, vn, st.block_table, st.context_lens, k, v)
    # only sequence 1's tokens 1 and 2 have positions 0 and 1
    p = st.block_table[1, 0]
    assert np.array_equal(W.k_cache_to_rows(k2)[p, :, 0], kn[1, 1])
    assert np.array_equal(v2[p, :, 1], vn[1, 2])
    changed = (k2 != k) & ~(np.isnan(widen(k2)) & np.isnan(widen(k)))
    assert changed.sum() <= 2 * 16
    bt = st.block_table.copy()
    bt[1, 0] = st.num_blocks
    try:
        O.append(kn, vn, bt, st.context_lens, k, v)
    except ValueError:
        return
    raise AssertionError("an out-of-pool block id was accepted")


# ---------------------------------------------------- token log-probabilities --

def np_log_softmax_entropy(x64):
    """Independent fp64 reference: numpy's logaddexp reduction and the entropy
    as -sum p log p."""
    lse = np.logaddexp.reduce(x64, axis=-1)
    logp = x64 - lse[..., None]
    p = np.exp(logp)
    ent = -np.sum(np.where(p > 0, p * logp, 0.0), axis=-1)
    return logp, ent


def pin_logprob_uniform(O):
    for V in (1, 7, 1000):
        x = np.full((3, V), 1.5, np.float32)
        lp, ent = O.logprob(x, np.array([0, V - 1, V // 2], np.int32))
        np.testing.assert_allclose(lp, -math.log(V), rtol=0, atol=TIGHT)
        np.testing.assert_allclose(ent, math.log(V), rtol=0, atol=TIGHT)
        lp0, _ = O.logprob(np.random.default_rng(V).normal(size=(3, V)).astype(np.float32),
                           np.zeros(3, np.int32), inv_temperature=0.0)
        np.testing.assert_allclose(lp0, -math.log(V), rtol=0, atol=TIGHT)


def pin_logprob_two_point(O):
    a, b = 0.25, 3.0
    x = np.array([[a, b], [a, b]], np.float32)
    lp, ent = O.logprob(x, np.array([0, 1], np.int32))
    p0 = 1.0 / (1.0 + math.exp(b - a))
    assert math.isclose(lp[0], math.log(p0), rel_tol=0, abs_tol=TIGHT)
    assert math.isclose(lp[1], math.log(1 - p0), rel_tol=0, abs_tol=TIGHT)
    h = -(p0 * math.log(p0) + (1 - p0) * math.log(1 - p0))
    assert math.isclose(ent[0], h, rel_tol=0, abs_tol=TIGHT)


def pin_logprob_bruteforce(O):
    for j, (B, V, T) in enumerate([(5, 1000, 1.0), (3, 4099, 0.5), (2, 64, 1.75)]):
        x, tok = W.make_logits(B, V, seed=60 + j)
        bits = W.bf16_bits(x)
        lp, ent = O.logprob(bits, tok, inv_temperature=T)
        logp, ref_ent = np_log_softmax_entropy(widen(bits) * T)
        np.testing.assert_allclose(lp, logp[np.arange(B), tok], rtol=0, atol=1e-11)
        np.testing.assert_allclose(ent, ref_ent, rtol=0, atol=1e-11)
        # every token of a row: the probabilities sum to one
        row = np.repeat(bits[:1], V, axis=0)
        all_lp, _ = O.logprob(row, np.arange(V, dtype=np.int32), inv_temperature=T, entropy=False)
        assert abs(np.exp(all_lp).sum() - 1.0) <= 1e-12


def pin_logprob_invariants(O):
    """A shift of every logit by one constant changes nothing; huge logits do
    not overflow; bf16 and float32 inputs of the same values agree; masked
    (-inf) tokens get probability zero and drop out of the entropy."""
    x, tok = W.make_logits(4, 500, seed=63)
    xf = x.float().numpy()
    lp, ent = O.logprob(xf, tok)
    lp2, ent2 = O.logprob(xf + np.float32(64.0), tok)  # exact: |x| < 64 and x has bf16 precision
    np.testing.assert_allclose(lp2, lp, rtol=0, atol=1e-12)
    # the entropy is lse - E[x]: both grow by 64, and the fp64 sum over V terms
    # of size ~64 leaves a few 1e-12 of cancellation error
    np.testing.assert_allclose(ent2, ent, rtol=0, atol=1e-10)
    big = np.array([[30000.0, 29990.0, -30000.0]], np.float32)
    lpb, entb = O.logprob(big, np.array([1], np.int32))
    assert math.isclose(lpb[0], -10 - math.log1p(math.exp(-10)), abs_tol=1e-12) and np.isfinite(entb[0])
    lpf, entf = O.logprob(W.bf16_bits(x), tok)
    assert np.array_equal(lpf, lp) and np.array_equal(entf, ent)
    xm = xf.copy()
    xm[:, 250:] = -np.inf
    tok_in = np.minimum(tok, 249)
    lpm, entm = O.logprob(xm, tok_in)
    lpr, entr = O.logprob(np.ascontiguousarray(xf[:, :250]), tok_in)
    np.testing.assert_allclose(lpm, lpr, rtol=0, atol=1e-12)
    np.testing.assert_allclose(entm, entr, rtol=0, atol=1e-12)


PINS = [pin_golden, pin_bruteforce, pin_length_one_is_v, pin_identical_keys_mean,
        pin_scale_zero_mean, pin_weights_probability, pin_dominant_key, pin_gqa_mapping,
        pin_block_shuffle, pin_token_permutation, pin_uniform_shift, pin_unread_slots,
        pin_nonpositive_length, pin_linear_in_v, pin_rows_and_threads,
        pin_multi_bruteforce, pin_multi_rows_are_decode_steps, pin_multi_causal, pin_multi_rows_subset,
        pin_append_places_rows, pin_append_builds_the_cache, pin_append_then_decode,
        pin_append_skips_and_rejects,
        pin_logprob_uniform, pin_logprob_two_point, pin_logprob_bruteforce, pin_logprob_invariants]


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
