"""GPU parity of the token log-probability / entropy kernel against the fp64
oracle, through the C ABI.

Bar: max-abs error <= 1e-4 on both log-probabilities and entropies (natural
log units).  The kernel works in fp32 on d = logit / T * log2(e) - mk, mk a
per-thread reference at most 2^64 (in probability) below the running max:
- the difference is taken on the raw values, so a large common offset costs
  nothing; rounding d costs at most |d| * 2^-24 (< 3e-6 here);
- each thread sums about 130 terms in order and 16 + 64 partial states are
  merged, so the relative error of the sums stays below ~1e-5, i.e. ~1e-5
  after the logarithm;
- the entropy is formed from sum p d relative to the reference, so its error
  scales with the entropy and the reference's distance from the max (at most
  64 in log2 units), not with |y|.
1e-4 leaves several times that margin.  PDA_RANDOM_LOGPROB_CASES sets the
number of seeded random calls (24 by default).
"""
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from paper_2405_11143_amd import pda_token_logprobs

pytestmark = pytest.mark.gpu

TOL = 1e-4


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def host_values(x):
    """What the oracle reads: bf16 bit patterns or float32 values."""
    return W.bf16_bits(x) if x.dtype == torch.bfloat16 else x.float().cpu().numpy()


def compare(lp, ent, ref_lp, ref_ent, what):
    lp, ent = lp.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64)
    e1, e2 = np.abs(lp - ref_lp).max(), np.abs(ent - ref_ent).max()
    print(f"{what}: logprob max-abs {e1:.2e}, entropy max-abs {e2:.2e}", flush=True)
    assert e1 <= TOL and e2 <= TOL, what


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("inv_t", [1.0, 1 / 0.7, 0.5, 0.0])
def test_small_vocab(dev, dtype, inv_t):
    x, tok = W.make_logits(5, 1000, seed=3, device=dev, dtype=dtype)
    lp, ent = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), inv_t)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(host_values(x), tok, np.float32(inv_t))
    compare(lp, ent, ref_lp, ref_ent, f"V=1000 {dtype} 1/T={inv_t:.3f}")


@pytest.mark.parametrize("name", ["llama3_vocab", "qwen_vocab"])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_full_size(dev, name, dtype):
    """One decode step's LM-head logits (256 rows x the full vocabulary)."""
    x, tok = W.logits_for(name, dev, dtype)
    lp, ent = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), 1.0)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(host_values(x), tok, 1.0)
    compare(lp, ent, ref_lp, ref_ent, f"{name} {dtype}")
    lp2, ent2 = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), 1.0)
    assert torch.equal(lp, lp2) and torch.equal(ent, ent2), "run-to-run"
    # the log-probabilities-only kernel sums the same terms in the same order
    lp3, none = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), 1.0, entropy=False)
    torch.cuda.synchronize()
    assert none is None and torch.equal(lp, lp3), "without entropies"


@pytest.mark.parametrize("V,stride", [(1001, 1008), (7, 8), (1, 8), (33000, 33024)])
def test_ragged_vocab_and_padded_rows(dev, V, stride):
    """Vocabularies that are not a multiple of the 16-byte load, and rows with
    padding past the vocabulary that holds NaN (never read into the result)."""
    x, tok = W.make_logits(6, V, seed=V, device=dev, dtype=torch.bfloat16)
    padded = torch.full((6, stride), float("nan"), dtype=torch.bfloat16, device=dev)
    padded[:, :V] = x
    lp, ent = pda_token_logprobs(padded, torch.from_numpy(tok).to(dev), 1.0, vocab=V)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(W.bf16_bits(x), tok, 1.0)
    compare(lp, ent, ref_lp, ref_ent, f"V={V} stride={stride}")


def test_masked_huge_and_bad_tokens(dev):
    """-inf logits drop out; logits of +-30000 do not overflow; a token id
    outside the vocabulary gives NaN for its row only."""
    x, tok = W.make_logits(4, 4096, seed=9, device=dev, dtype=torch.float32)
    x[0, 2048:] = float("-inf")
    tok[0] = min(int(tok[0]), 2047)
    x[1] = x[1] * 0
    x[1, 5], x[1, 6], x[1, 7] = 30000.0, 29990.0, -30000.0
    tok[1] = 6
    lp, ent = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), 1.0)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(x.cpu().numpy(), tok, 1.0)
    compare(lp, ent, ref_lp, ref_ent, "masked / huge logits")
    bad = tok.copy()
    bad[2] = 4096
    bad[3] = -1
    lp_b, ent_b = pda_token_logprobs(x, torch.from_numpy(bad).to(dev), 1.0)
    torch.cuda.synchronize()
    lp_b = lp_b.cpu().numpy()
    assert np.isnan(lp_b[2]) and np.isnan(lp_b[3]) and np.isfinite(lp_b[:2]).all()
    assert np.array_equal(ent_b.cpu().numpy(), ent.cpu().numpy())  # the entropy does not depend on the token


def test_no_entropy_output(dev):
    x, tok = W.make_logits(3, 5000, seed=11, device=dev)
    lp, ent = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), 1.0, entropy=False)
    torch.cuda.synchronize()
    assert ent is None
    ref_lp, _ = oracle.logprob(W.bf16_bits(x), tok, 1.0, entropy=False)
    assert np.abs(lp.cpu().numpy() - ref_lp).max() <= TOL


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_rising_logits_retake_passes(dev, dtype):
    """Rows whose logits outgrow each thread's reference within a pass (a
    ramp, a jump from -1e4 to +1e4, -inf before the only finite logit, a
    sharp temperature), so that passes are taken again against their max,
    and a row whose first logit is its max (never)."""
    V = 40000
    x, tok = W.make_logits(6, V, seed=21, device=dev, dtype=torch.float32)
    x[0] = torch.arange(V, device=dev, dtype=torch.float32) * 0.01
    x[1, : V // 2], x[1, V // 2:] = -1e4, 1e4
    x[2] = float("-inf")
    x[2, V - 3] = 5.0
    tok[2] = V - 3
    x[3, 0] = 60.0
    x[4] = x[4] * 8
    x = x.to(dtype)
    for inv_t in (1.0, 25.0):
        lp, ent = pda_token_logprobs(x, torch.from_numpy(tok).to(dev), inv_t)
        torch.cuda.synchronize()
        ref_lp, ref_ent = oracle.logprob(host_values(x), tok, np.float32(inv_t))
        # log-probabilities down to -2e5 here: an fp32 result of that size
        # carries a rounding of 2^-24 of itself (d is rounded once, then the
        # log is subtracted), so their bar grows with |log p|
        lp, ent = lp.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64)
        e_lp = np.abs(lp - ref_lp) / (TOL + 4 * 2.0 ** -24 * np.abs(ref_lp))
        e_ent = np.abs(ent - ref_ent)
        print(f"rising logits {dtype} 1/T={inv_t}: logprob error / bar {e_lp.max():.2f}, "
              f"entropy max-abs {e_ent.max():.2e}", flush=True)
        assert e_lp.max() <= 1.0 and e_ent.max() <= TOL, (dtype, inv_t)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_neg_inf_rows_take_entropy_again_alone(dev, dtype):
    """A row with -inf logits has its entropy sum taken again in a second,
    guarded pass; rows without any keep their one-pass results bit for bit,
    and the log-probabilities (which never depend on that pass) are the same
    bits with or without it."""
    x, tok = W.make_logits(8, 128256, seed=21, device=dev, dtype=dtype)
    tt = torch.from_numpy(tok).to(dev)
    lp0, ent0 = pda_token_logprobs(x, tt, 1.0)
    y = x.clone()
    y[3, 1000:90000] = float("-inf")   # a wide masked band
    y[5, ::7] = float("-inf")          # scattered masked tokens
    tok2 = tok.copy()
    tok2[3], tok2[5] = 17, 1
    tt2 = torch.from_numpy(tok2).to(dev)
    lp1, ent1 = pda_token_logprobs(y, tt2, 1.0)
    torch.cuda.synchronize()
    keep = [0, 1, 2, 4, 6, 7]
    assert torch.equal(ent1[keep], ent0[keep]) and torch.equal(lp1[keep], lp0[keep])
    ref_lp, ref_ent = oracle.logprob(host_values(y), tok2, 1.0)
    compare(lp1, ent1, ref_lp, ref_ent, f"-inf rows {dtype}")
    assert np.isfinite(ent1.cpu().numpy()).all()
    lp_only, none = pda_token_logprobs(y, tt2, 1.0, entropy=False)
    torch.cuda.synchronize()
    assert none is None and torch.equal(lp_only, lp1)


@pytest.mark.parametrize("rows,V,dtype", [(100, 128256, torch.bfloat16), (8, 128256, torch.bfloat16),
                                          (3, 151936, torch.float32), (40, 33000, torch.bfloat16)],
                         ids=str)
def test_rows_split_over_workgroups(dev, rows, V, dtype):
    """A batch with fewer rows than compute units, given a workspace, has each
    row streamed by several workgroups whose states a second kernel merges in
    slice order: results agree with one workgroup per row to fp32 rounding,
    match the oracle and repeat bit for bit, whatever the workspace held
    before (NaN bytes, or another call's states)."""
    from paper_2405_11143_amd.pda import PDA_DTYPE_BF16, PDA_DTYPE_F32, pda_logprob_workspace_bytes

    x, tok = W.make_logits(rows, V, seed=rows + V, device=dev, dtype=dtype)
    tt = torch.from_numpy(tok).to(dev)
    need = pda_logprob_workspace_bytes(rows, V, PDA_DTYPE_BF16 if dtype == torch.bfloat16 else PDA_DTYPE_F32)
    assert need > 0
    ws = torch.full((need + 4096,), 0xff, dtype=torch.uint8, device=dev)  # NaN patterns; larger than needed
    lp, ent = pda_token_logprobs(x, tt, 1.0, workspace=ws)
    lp1, ent1 = pda_token_logprobs(x, tt, 1.0, workspace=None)  # one workgroup per row
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(host_values(x), tok, 1.0)
    compare(lp, ent, ref_lp, ref_ent, f"split rows={rows} V={V} {dtype}")
    compare(lp1, ent1, ref_lp, ref_ent, f"one workgroup per row rows={rows} V={V} {dtype}")
    d_lp = (lp - lp1).abs().max().item()
    d_ent = (ent - ent1).abs().max().item()
    print(f"split vs one workgroup: logprob {d_lp:.2e}, entropy {d_ent:.2e}", flush=True)
    assert d_lp <= 2e-5 and d_ent <= 2e-5
    for _ in range(2):
        lp2, ent2 = pda_token_logprobs(x, tt, 1.0, workspace=ws)
        assert torch.equal(lp, lp2) and torch.equal(ent, ent2), "run-to-run"
    lp3, none = pda_token_logprobs(x, tt, 1.0, entropy=False, workspace=ws)
    torch.cuda.synchronize()
    assert none is None and torch.equal(lp, lp3), "without entropies"
    # the same workspace for a call of another shape, then this one again
    xs, toks = W.make_logits(2, 50000, seed=5, device=dev, dtype=torch.bfloat16)
    lps, ents = pda_token_logprobs(xs, torch.from_numpy(toks).to(dev), 1.0, workspace=ws)
    ref_lps, ref_ents = oracle.logprob(W.bf16_bits(xs), toks, 1.0)
    compare(lps, ents, ref_lps, ref_ents, "another shape on the same workspace")
    lp4, ent4 = pda_token_logprobs(x, tt, 1.0, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(lp, lp4) and torch.equal(ent, ent4)


def test_split_rows_with_neg_inf(dev):
    """-inf logits in some slices of split rows: each slice takes its entropy
    sum again, guarded, against its own reference before the merge."""
    x, tok = W.make_logits(8, 128256, seed=33, device=dev, dtype=torch.bfloat16)
    x[1, 5000:70000] = float("-inf")   # spans several slices
    x[4, ::11] = float("-inf")
    x[6, 127000:] = float("-inf")      # the partial chunk's slice only
    tok[1], tok[4], tok[6] = 3, 1, 5
    tt = torch.from_numpy(tok).to(dev)
    lp, ent = pda_token_logprobs(x, tt, 1.0)
    lp1, ent1 = pda_token_logprobs(x, tt, 1.0, workspace=None)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(W.bf16_bits(x), tok, 1.0)
    compare(lp, ent, ref_lp, ref_ent, "split rows with -inf logits")
    compare(lp1, ent1, ref_lp, ref_ent, "one workgroup per row with -inf logits")
    assert np.isfinite(ent.cpu().numpy()).all()


def draw_logprob_case(case: int):
    r = np.random.default_rng(7000 + case)
    dtype = torch.bfloat16 if r.random() < 0.6 else torch.float32
    rows = int(r.choice([1, 2, 7, 31, 100, 255, 256, 300]))
    V = int(r.choice([1, 7, 8, 9, 1000, 4097, 33000, 128256, 151936]))
    per16 = 8 if dtype == torch.bfloat16 else 4  # elements per 16 bytes
    stride = (V + per16 - 1) // per16 * per16 + per16 * int(r.choice([0, 0, 1, 8]))
    inv_t = float(r.choice([1.0, 1 / 0.7, 0.5, 2.0, 0.0]))
    workspace = "auto" if r.random() < 0.7 else None
    entropy = bool(r.random() < 0.8)
    # -inf spans in some rows (with a positive inverse temperature), never over
    # the row's token and never the whole row
    spans = []
    for row in range(rows):
        if V > 2 and inv_t > 0 and r.random() < 0.2:
            a = int(r.integers(0, V - 1))
            spans.append((row, a, int(r.integers(a + 1, V + 1))))
    return dtype, rows, V, stride, inv_t, workspace, entropy, spans


@pytest.mark.parametrize("case", range(int(os.environ.get("PDA_RANDOM_LOGPROB_CASES", "24"))))
def test_random_logprob_case(dev, case):
    """Seeded random calls: bf16 and fp32, 1-300 rows (so both one workgroup
    per row and rows split over workgroups), vocabularies from 1 to 151936
    (ragged ones), rows padded past the vocabulary with NaN, temperatures
    (0 included), -inf spans, with and without a workspace and the entropy;
    the same bar against the oracle, and the log-probabilities bitwise the
    same with and without the entropy."""
    dtype, rows, V, stride, inv_t, workspace, entropy, spans = draw_logprob_case(case)
    what = f"case {case}: {dtype} rows={rows} V={V} stride={stride} 1/T={inv_t:.3f} ws={workspace} ent={entropy}"
    print(what, flush=True)
    x, tok = W.make_logits(rows, V, seed=case, device=dev, dtype=dtype)
    for row, a, b in spans:
        if a == 0 and b == V:  # keep one finite logit
            b = V - 1
        x[row, a:b] = float("-inf")
        t = int(tok[row])
        if a <= t < b:  # the sampled token keeps a finite logit
            tok[row] = a - 1 if a > 0 else b
    padded = torch.full((rows, stride), float("nan"), dtype=dtype, device=dev)
    padded[:, :V] = x
    tt = torch.from_numpy(tok).to(dev)
    lp, ent = pda_token_logprobs(padded, tt, inv_t, entropy=entropy, vocab=V, workspace=workspace)
    torch.cuda.synchronize()
    ref_lp, ref_ent = oracle.logprob(host_values(x), tok, np.float32(inv_t), entropy=entropy)
    e1 = np.abs(lp.cpu().numpy().astype(np.float64) - ref_lp).max()
    assert e1 <= TOL, (what, e1)
    if entropy:
        e2 = np.abs(ent.cpu().numpy().astype(np.float64) - ref_ent).max()
        assert e2 <= TOL, (what, e2)
        lp2, none = pda_token_logprobs(padded, tt, inv_t, entropy=False, vocab=V, workspace=workspace)
        torch.cuda.synchronize()
        assert none is None and torch.equal(lp, lp2), what
    else:
        assert ent is None
