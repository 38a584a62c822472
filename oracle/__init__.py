"""CPU oracle for paged decode attention (fp64) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never does, and this
package imports nothing from it: the two share no code.

The computation is the plain definition of single-query scaled dot-product
attention over a paged KV cache (the rollout decode step that the paper runs
through vLLM's PagedAttention, Section 3.2 and Appendix C), written out in
``pda_oracle.c``.  This module only compiles that file with gcc and marshals
numpy arrays into it.

bf16 inputs are passed as their raw bit patterns (``numpy.uint16``).
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
        i32, dbl, vp = ctypes.c_int, ctypes.c_double, ctypes.c_void_p
        common = [i32] * 7 + [vp] * 5 + [dbl]
        lib.pda_oracle_decode.argtypes = common + [vp, i32]
        lib.pda_oracle_decode_rows.argtypes = common + [vp, i32, vp, i32]
        lib.pda_oracle_weights.argtypes = common + [i32, i32, vp]
        for f in (lib.pda_oracle_decode, lib.pda_oracle_decode_rows, lib.pda_oracle_weights):
            f.restype = i32
        self.lib = lib

    def decode(self, q, k_cache, v_cache, block_table, context_lens, scale, threads: int = 1):
        """Attention output for every (b, h): float64 ``[B][Hq][D]``."""
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens)
        out = np.full((dims[0], dims[1], dims[3]), np.nan)  # unwritten rows would show
        rc = self.lib.pda_oracle_decode(*dims, *ptrs, float(scale), out.ctypes.data, int(threads))
        _check(rc, "decode")
        del keep
        return out

    def decode_rows(self, q, k_cache, v_cache, block_table, context_lens, scale, rows,
                    threads: int = 1):
        """Attention output for the listed (b, h) pairs only: float64 ``[n][D]``."""
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens)
        rows = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 2)
        out = np.full((rows.shape[0], dims[3]), np.nan)
        rc = self.lib.pda_oracle_decode_rows(*dims, *ptrs, float(scale), rows.ctypes.data,
                                             rows.shape[0], out.ctypes.data, int(threads))
        _check(rc, "decode_rows")
        del keep
        return out

    def weights(self, q, k_cache, v_cache, block_table, context_lens, scale, b: int, h: int):
        """The softmax weights of (b, h) over its context: float64 ``[L]``."""
        dims, ptrs, keep = _prep(q, k_cache, v_cache, block_table, context_lens)
        L = max(int(np.asarray(context_lens)[b]), 0)
        w = np.zeros(max(L, 1), dtype=np.float64)
        rc = self.lib.pda_oracle_weights(*dims, *ptrs, float(scale), int(b), int(h), w.ctypes.data)
        _check(rc, "weights")
        del keep
        return w[:rc]


def _load() -> Oracle:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = Oracle(_LIB)
    return _lib


def _prep(q, k_cache, v_cache, block_table, context_lens):
    q = np.ascontiguousarray(q, dtype=np.uint16)
    k_cache = np.ascontiguousarray(k_cache, dtype=np.uint16)
    v_cache = np.ascontiguousarray(v_cache, dtype=np.uint16)
    block_table = np.ascontiguousarray(block_table, dtype=np.int32)
    context_lens = np.ascontiguousarray(context_lens, dtype=np.int32)
    if q.ndim != 3 or k_cache.ndim != 5 or v_cache.ndim != 4:
        raise ValueError("q must be [B][Hq][D], k_cache [num_blocks][Hkv][D/8][BS][8], "
                         "v_cache [num_blocks][Hkv][BS][D]")
    B, Hq, D = q.shape
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
    """Attention output for every (b, h): float64 ``[B][Hq][D]``."""
    return _load().decode(q, k_cache, v_cache, block_table, context_lens, scale, threads)


def decode_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows,
                threads: int = 1) -> np.ndarray:
    """Attention output for the listed (b, h) pairs only: float64 ``[n][D]``."""
    return _load().decode_rows(q, k_cache, v_cache, block_table, context_lens, scale, rows, threads)


def weights(q, k_cache, v_cache, block_table, context_lens, scale, b: int, h: int) -> np.ndarray:
    """The softmax weights of (b, h) over its context: float64 ``[L]``."""
    return _load().weights(q, k_cache, v_cache, block_table, context_lens, scale, b, h)
