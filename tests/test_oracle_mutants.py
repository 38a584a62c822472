"""The oracle pins must catch plausible mistakes (no GPU).

Each case below plants one mistake in a copy of the oracle's C source (a
dropped term, a wrong sign, a wrong index, a transposed layout), builds it
with gcc into a temporary directory, and runs every pin of
``test_oracle_pins.py`` against it in a child process (a mistake may crash).
At least one pin must fail for every mutant; the unmodified source must pass
all of them.
"""
import os
import subprocess
import sys
import textwrap

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "pda_oracle.c")

MUTANTS = {
    "kv head = h mod Hkv": ("int g = h / G;", "int g = h % P->Hkv;"),
    "K block and slot swapped": ("const int32_t p = bt[t / P->BS];\n    const int o = t % P->BS;",
                                 "const int32_t p = bt[t % P->BS];\n    const int o = t / P->BS;"),
    "V block and slot swapped": ("bt[t / P->BS], g, t % P->BS", "bt[t % P->BS], g, t / P->BS"),
    "no max subtraction": ("exp(scores[t] - m)", "exp(scores[t])"),
    "exp sign flipped": ("exp(scores[t] - m)", "exp(m - scores[t])"),
    "scale dropped": ("scores[t] = P->scale * dot;", "scores[t] = dot;"),
    "no normalisation": ("for (int t = 0; t < L; ++t) scores[t] /= Z;", ""),
    "sum starts at one": ("double Z = 0.0;", "double Z = 1.0;"),
    "V layout [p][o][g]": ("(((size_t)p * P->Hkv + g) * P->BS + o) * P->D",
                           "(((size_t)p * P->BS + o) * P->Hkv + g) * P->D"),
    "K layout read as rows": ("((((size_t)p * P->Hkv + g) * (P->D / 8) + d / 8) * P->BS + o) * 8 + d % 8",
                              "(((size_t)p * P->Hkv + g) * P->BS + o) * P->D + d"),
    "K chunk element order": ("* P->BS + o) * 8 + d % 8", "* P->BS + o) * 8 + (7 - d % 8)"),
    "q row of the kv head": ("(((size_t)b * P->nq + i) * P->Hq + h) * P->D",
                             "(((size_t)b * P->nq + i) * P->Hq + g) * P->D"),
    "V read from K": ("const uint16_t *vrow = P->v +", "const uint16_t *vrow = P->k +"),
    "bf16 widened wrongly": ("(uint32_t)bits << 16", "(uint32_t)bits << 15"),
    "last token dropped from V sum": ("for (int t = 0; t < L; ++t) {\n    const uint16_t *vrow",
                                      "for (int t = 0; t + 1 < L; ++t) {\n    const uint16_t *vrow"),
    "min instead of max": ("if (scores[t] > m) m = scores[t];", "if (scores[t] < m || t == 0) m = scores[t];"),
    "table row stride = B": ("P->block_table + (size_t)b * P->max_blocks_per_seq",
                             "P->block_table + (size_t)b * P->B"),
    "zero length not zeroed": ("for (int d = 0; d < P->D; ++d) out_row[d] = 0.0;\n  int L",
                               "int L"),
    # several query tokens per sequence
    "visible length off by one": ("int n = L - P->nq + 1 + i;", "int n = L - P->nq + i;"),
    "no causal mask": ("int n = L - P->nq + 1 + i;", "int n = L;"),
    "same q row for every new token": ("(((size_t)b * P->nq + i) * P->Hq + h) * P->D",
                                       "(((size_t)b * P->nq) * P->Hq + h) * P->D"),
    "new-token index not decoded": ("i = (r / J->P->Hq) % J->P->nq;", "i = 0;"),
    # KV-cache append
    "append order reversed": ("const int t = L - n + i;\n      if (t < 0) continue;\n      const int32_t p = bt[",
                              "const int t = L - 1 - i;\n      if (t < 0) continue;\n      const int32_t p = bt["),
    "append K stored as rows": ("k_cache[k_elem(&P, p, g, o, d)] = k_new[src + d];",
                                "k_cache[v_row(&P, p, g, o) + d] = k_new[src + d];"),
    "append V taken from K": ("v_cache[v_row(&P, p, g, o) + d] = v_new[src + d];",
                              "v_cache[v_row(&P, p, g, o) + d] = k_new[src + d];"),
    "append source [b][g][i]": ("(((size_t)b * n + i) * Hkv + g) * D", "(((size_t)b * Hkv + g) * n + i) * D"),
    "append no id check": ("if (p < 0 || p >= num_blocks) return -5;\n    }\n  }\n  for (int b = 0; b < B; ++b) {\n    const int L",
                           "}\n  }\n  for (int b = 0; b < B; ++b) {\n    const int L"),
    # log-probabilities
    "temperature dropped": ("x[j] = raw * inv_temperature;", "x[j] = raw;"),
    "lse without the max": ("const double lse = m + log(Z);", "const double lse = log(Z);"),
    "no max subtraction in lse": [("Z += exp(x[j] - m);", "Z += exp(x[j]);"),
                                  ("const double lse = m + log(Z);", "const double lse = log(Z);")],
    "entropy sign": ("entropy[b] = lse - mean_x;", "entropy[b] = mean_x - lse;"),
    "entropy unnormalised": ("mean_x += e / Z * x[j];", "mean_x += e * x[j];"),
    "token off by one": ("logprob[b] = x[tokens[b]] - lse;", "logprob[b] = x[tokens[b] > 0 ? tokens[b] - 1 : 1] - lse;"),
    "bf16 logits widened as f32 bits": ("raw = bf16_to_double(((const uint16_t *)logits)[base + j]);",
                                        "raw = (double)((const uint16_t *)logits)[base + j];"),
}

RUNNER = textwrap.dedent("""
    import sys, traceback
    sys.path[:0] = [{root!r}, {tests!r}]
    import numpy as np
    np.seterr(all="ignore")
    import oracle, test_oracle_pins as T
    O = oracle.Oracle({lib!r})
    failed = []
    for pin in T.PINS:
        try:
            pin(O)
        except BaseException:
            failed.append(pin.__name__)
    print("FAILED:" + ",".join(failed))
""")


def run_pins_in_child(lib_path):
    code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib_path)
    p = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    lines = [l for l in p.stdout.splitlines() if l.startswith("FAILED:")]
    if p.returncode != 0 or not lines:
        return None  # crashed: the mistake is caught, loudly
    return [f for f in lines[-1][len("FAILED:"):].split(",") if f]


def build_variant(tmp_path, edits):
    """`edits` is one (old, new) pair or a list of them (one mistake that
    needs consistent edits in several places)."""
    src = open(SRC).read()
    for old, new in ([edits] if isinstance(edits, tuple) else edits):
        assert old in src, f"mutation anchor not found: {old!r}"
        src = src.replace(old, new)
    path = tmp_path / "pda_oracle_mut.c"
    path.write_text(src)
    lib = str(tmp_path / "libpda_oracle_mut.so")
    oracle.build(src=str(path), lib=lib)
    return lib


def test_unmodified_source_passes_all_pins(tmp_path):
    lib = str(tmp_path / "libpda_oracle_copy.so")
    oracle.build(lib=lib)
    assert run_pins_in_child(lib) == []


@pytest.mark.parametrize("name", list(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    failed = run_pins_in_child(build_variant(tmp_path, MUTANTS[name]))
    assert failed is None or len(failed) > 0, f"no pin caught mutant {name!r}"
