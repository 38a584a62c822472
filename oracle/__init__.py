"""CPU oracle for the rollout decode step (fp64) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never does, and this
package imports nothing from it: the two share no code.

What ``pda_oracle.c`` writes out, plainly and in fp64 (the rollout phase the
paper runs through vLLM, Section 3.2 and Appendix C):

* attention of each sequence's new query token over its paged KV cache
  (PagedAttention), and of several new causal query tokens per sequence
  (speculative decoding, chunked prefill);
* storing the new tokens' keys and values in the paged cache;
* the log-probability of each sampled token and the entropy of its
  distribution.

This module only compiles that file with gcc and marshals numpy arrays into
it.  bf16 inputs are passed as their raw bit patterns (``numpy.uint16``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pda_oracle.c")
_LIB = os.path.join(_HERE, "libpda_oracle.so")
_lib = None


def build(verbose: bool = False, src: str = _SRC, lib: str = _LIB) -> str:
    """Compile ``pda_oracle.c`` (or an edited copy) into a shared library with gcc -O2."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-o", lib + ".tmp", src, "-lm", "-lpthread"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


class Oracle:
    """ctypes binding of one build of ``pda_oracle.c`` (the default build, or a
    variant compiled from an edited copy of the source by the mutation tests)."""

    def __init__(self, lib_path: str):
        lib = ctypes.CDLL(lib_path)
        i32, i64, dbl, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        common = [i32] * 7 + [vp] * 5 + [dbl]
        lib.pda_oracle_decode.argtypes = common + [vp, i32]
        lib.pda_oracle_decode_multi.argtypes = common + [i32, vp, i32]
        lib.pda_oracle_decode_rows.argtypes = common + [i32, vp, i32, vp, i32]
        lib.pda_oracle_weights.argtypes = common + [i32, i32, vp]
        lib.pda_oracle_append.argtypes = [i32] * 7 + [vp] * 6
        lib.pda_oracle_logprob.argtypes = [i32, i32, i64, vp, i32, vp, dbl, vp, vp]
        for f in (lib.pda_oracle_decode, lib.pda_oracle_decode_multi, lib.pda_oracle_decode_rows,
                  lib.pda_oracle_weights, lib.pda_oracle_append, lib.pda_oracle_logprob):
            f.restype = i32
        self.lib = lib

    # ---- attention ----

    def decode(self, q, k_cache, v_cache, block_table, context_lens, scale, threads: int = 1):
        """Decode step, one query token per sequence: float64 ``[B][Hq][D]``."""
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens, 1)
        out = np.full((dims[0], dims[1], dims[3]), np.nan)  # unwritten rows would show
        rc = self.lib.pda_oracle_decode(*dims, *ptrs, float(scale), out.ctypes.data, int(threads))
        _check(rc, "decode")
        del keep
        return out

    def decode_multi(self, q, k_cache, v_cache, block_table, context_lens, scale, threads: int = 1):
        """``q`` is ``[B][n][Hq][D]``: n causal query tokens per sequence, the
        last n of its context.  Returns float64 ``[B][n][Hq][D]``."""
        n = np.asarray(q).shape[1]
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens, n)
        out = np.full((dims[0], n, dims[1], dims[3]), np.nan)
        rc = self.lib.pda_oracle_decode_multi(*dims, *ptrs, float(scale), n, out.ctypes.data, int(threads))
        _check(rc, "decode_multi")
        del keep
        return out

    def decode_rows(self, q, k_cache, v_cache, block_table, context_lens, scale, rows,
                    threads: int = 1):
        """Decode-step output for the listed (b, h) pairs only: float64 ``[n][D]``."""
        rows = np.asarray(rows, dtype=np.int32).reshape(-1, 2)
        triples = np.stack([rows[:, 0], np.zeros_like(rows[:, 0]), rows[:, 1]], axis=1)
        return self._rows(q, k_cache, v_cache, block_table, context_lens, scale, 1, triples, threads)

    def decode_multi_rows(self, q, k_cache, v_cache, block_table, context_lens, scale, rows,
                          threads: int = 1):
        """Multi-token output for the listed (b, i, h) triples only: float64 ``[n][D]``."""
        n = np.asarray(q).shape[1]
        return self._rows(q, k_cache, v_cache, block_table, context_lens, scale, n,
                          np.asarray(rows, dtype=np.int32).reshape(-1, 3), threads)

    def _rows(self, q, k_cache, v_cache, block_table, context_lens, scale, n, triples, threads):
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens, n)
        triples = np.ascontiguousarray(triples, dtype=np.int32)
        out = np.full((triples.shape[0], dims[3]), np.nan)
        rc = self.lib.pda_oracle_decode_rows(*dims, *ptrs, float(scale), n, triples.ctypes.data,
                                             triples.shape[0], out.ctypes.data, int(threads))
        _check(rc, "decode_rows")
        del keep
        return out

    def weights(self, q, k_cache, v_cache, block_table, context_lens, scale, b: int, h: int):
        """The softmax weights of decode row (b, h) over its context: float64 ``[L]``."""
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens, 1)
        L = max(int(np.asarray(context_lens)[b]), 0)
        w = np.zeros(max(L, 1), dtype=np.float64)
        rc = self.lib.pda_oracle_weights(*dims, *ptrs, float(scale), int(b), int(h), w.ctypes.data)
        _check(rc, "weights")
        del keep
        return w[:rc]

    # ---- KV-cache append ----

    def append(self, k_new, v_new, block_table, context_lens, k_cache, v_cache):
        """Store ``k_new``/``v_new`` (bf16 bits ``[B][n][Hkv][D]``) at positions
        L - n .. L - 1 of every sequence.  Returns new (k_cache, v_cache) arrays;
        the inputs are not modified."""
        k_new = np.ascontiguousarray(k_new, dtype=np.uint16)
        v_new = np.ascontiguousarray(v_new, dtype=np.uint16)
        block_table = np.ascontiguousarray(block_table, dtype=np.int32)
        context_lens = np.ascontiguousarray(context_lens, dtype=np.int32)
        k_out = np.array(k_cache, dtype=np.uint16, copy=True, order="C")
        v_out = np.array(v_cache, dtype=np.uint16, copy=True, order="C")
        if k_new.ndim != 4 or v_new.shape != k_new.shape or k_out.ndim != 5 or v_out.ndim != 4:
            raise ValueError("k_new/v_new must be [B][n][Hkv][D], k_cache [NB][Hkv][D/8][BS][8], "
                             "v_cache [NB][Hkv][BS][D]")
        B, n, Hkv, D = k_new.shape
        NB, _, BS, _ = v_out.shape
        if (v_out.shape != (NB, Hkv, BS, D) or k_out.shape != (NB, Hkv, D // 8, BS, 8)
                or block_table.ndim != 2 or block_table.shape[0] != B or context_lens.shape != (B,)):
            raise ValueError("inconsistent shapes")
        rc = self.lib.pda_oracle_append(B, Hkv, D, BS, NB, block_table.shape[1], n, k_new.ctypes.data,
                                        v_new.ctypes.data, block_table.ctypes.data, context_lens.ctypes.data,
                                        k_out.ctypes.data, v_out.ctypes.data)
        _check(rc, "append")
        return k_out, v_out

    # ---- log-probabilities ----

    def logprob(self, logits, tokens, inv_temperature=1.0, entropy: bool = True):
        """``logits`` [B][V] as bf16 bits (uint16) or float32.  Returns
        (logprob float64 [B], entropy float64 [B] or None)."""
        logits = np.ascontiguousarray(logits)
        if logits.dtype not in (np.uint16, np.float32) or logits.ndim != 2:
            raise ValueError("logits must be a [B][V] array of bf16 bits (uint16) or float32")
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        B, V = logits.shape
        if tokens.shape != (B,):
            raise ValueError("tokens must be [B]")
        lp = np.full(B, np.nan)
        ent = np.full(B, np.nan) if entropy else None
        rc = self.lib.pda_oracle_logprob(B, V, V, logits.ctypes.data, int(logits.dtype == np.float32),
                                         tokens.ctypes.data, float(inv_temperature), lp.ctypes.data,
                                         ent.ctypes.data if entropy else None)
        _check(rc, "logprob")
        return lp, ent


def _load() -> Oracle:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = Oracle(_LIB)
    return _lib


def _prep(q, k_cache, v_cache, block_table, context_lens, n):
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k_cache = np.ascontiguousarray(k_cache, dtype=np.uint16)
    v_cache = np.ascontiguousarray(v_cache, dtype=np.uint16)
    block_table = np.ascontiguousarray(block_table, dtype=np.int32)
    context_lens = np.ascontiguousarray(context_lens, dtype=np.int32)
    want_q = 3 if n == 1 and q.ndim == 3 else 4
    if q.ndim != want_q or k_cache.ndim != 5 or v_cache.ndim != 4:
        raise ValueError("q must be [B][Hq][D] (or [B][n][Hq][D]), k_cache [num_blocks][Hkv][D/8][BS][8], "
                         "v_cache [num_blocks][Hkv][BS][D]")
    B, Hq, D = q.shape[0], q.shape[-2], q.shape[-1]
    NB, Hkv, BS, Dv = v_cache.shape
    if (k_cache.shape != (NB, Hkv, D // 8, BS, 8) or Dv != D or block_table.ndim != 2
            or block_table.shape[0] != B or context_lens.shape != (B,)):
        raise ValueError("inconsistent shapes")
    dims = [B, Hq, Hkv, D, BS, NB, block_table.shape[1]]
    ptrs = [a.ctypes.data for a in (q, k_cache, v_cache, block_table, context_lens)]
    keep = (q, k_cache, v_cache, block_table, context_lens)
    return dims, ptrs, keep


def _check(rc: int, what: str):
    if rc < 0:
        raise ValueError(f"oracle {what} rejected its arguments (code {rc})")


def decode(q, k_cache, v_cache, block_table, context_lens, scale, threads: int = 1) -> np.ndarray:
    """Decode step, one query token per sequence: float64 ``[B][Hq][D]``."""
    return _load().decode(q, k_cache, v_cache, block_table, context_lens, scale, threads)


def decode_multi(q, k_cache, v_cache, block_table, context_lens, scale, threads: int = 1) -> np.ndarray:
    """n causal query tokens per sequence (``q`` [B][n][Hq][D]): float64 ``[B][n][Hq][D]``."""
    return _load().decode_multi(q, k_cache, v_cache, block_table, context_lens, scale, threads)


def decode_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows,
                threads: int = 1) -> np.ndarray:
    """Decode-step output for the listed (b, h) pairs only: float64 ``[n][D]``."""
    return _load().decode_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows, threads)


def decode_multi_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows,
                      threads: int = 1) -> np.ndarray:
    """Multi-token output for the listed (b, i, h) triples only: float64 ``[n][D]``."""
    return _load().decode_multi_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows, threads)


def weights(q, k_cache, v_cache, block_table, context_lens, scale, b: int, h: int) -> np.ndarray:
    """The softmax weights of decode row (b, h) over its context: float64 ``[L]``."""
    return _load().weights(q, k_cache, v_cache, block_table, context_lens, scale, b, h)


def append(k_new, v_new, block_table, context_lens, k_cache, v_cache):
    """New (k_cache, v_cache) with each sequence's n new tokens stored at L - n .. L - 1."""
    return _load().append(k_new, v_new, block_table, context_lens, k_cache, v_cache)


def logprob(logits, tokens, inv_temperature=1.0, entropy: bool = True):
    """(log-probability of tokens[b], entropy) of softmax(logits[b] * inv_temperature)."""
    return _load().logprob(logits, tokens, inv_temperature, entropy)
