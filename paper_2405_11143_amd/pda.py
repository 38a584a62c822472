"""Python binding of the paged decode-attention C ABI (include/pda.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of libpda.so.  The library must have been built in-tree
(``paper_2405_11143_amd/build.py``); if it is missing, loading fails with an
error -- there is no fallback implementation.  PyTorch supplies device
memory and streams.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpda.so")

PDA_OK, PDA_ERR_NULL, PDA_ERR_SHAPE, PDA_ERR_UNSUPPORTED = 0, 1, 2, 3
PDA_ERR_WORKSPACE, PDA_ERR_ALIGNMENT, PDA_ERR_VALUE, PDA_ERR_HIP = 4, 5, 6, 7

# Every symbol include/pda.h declares.
EXPORTED = ("pda_plan", "pda_workspace_bytes", "pda_decode", "pda_partition_attention",
            "pda_merge_partitions", "pda_validate_host", "pda_status_string")


class pda_problem(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "num_seqs", "num_q_heads", "num_kv_heads", "head_dim", "block_size", "num_blocks",
        "max_blocks_per_seq", "max_context_len", "partition_tokens")]


class pda_plan_info(ctypes.Structure):
    _fields_ = [("partition_tokens", ctypes.c_int32), ("num_partitions", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class PdaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {pda_status_string(status)} (status {status})")


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libpda.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2405_11143_amd/build.py "
                           "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(pda_problem)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.pda_plan.argtypes = [P, ctypes.POINTER(pda_plan_info)]
    lib.pda_workspace_bytes.argtypes = [P, ctypes.POINTER(sz)]
    step = [P, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, sz, vp]
    lib.pda_decode.argtypes = step
    lib.pda_partition_attention.argtypes = step
    lib.pda_merge_partitions.argtypes = [P, vp, vp, vp, sz, vp]
    lib.pda_validate_host.argtypes = [P, vp, vp, ctypes.POINTER(ctypes.c_int64)]
    lib.pda_status_string.argtypes = [i32]
    lib.pda_status_string.restype = ctypes.c_char_p
    for name in EXPORTED[:-1]:
        getattr(lib, name).restype = i32
    if path == LIB_PATH:
        _lib = lib
    return lib


def pda_status_string(status: int) -> str:
    return load_library().pda_status_string(int(status)).decode()


def make_problem(num_seqs, num_q_heads, num_kv_heads, head_dim, num_blocks, max_blocks_per_seq,
                 max_context_len, partition_tokens=0, block_size=16) -> pda_problem:
    return pda_problem(int(num_seqs), int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size),
                       int(num_blocks), int(max_blocks_per_seq), int(max_context_len), int(partition_tokens))


def pda_plan(prob: pda_problem) -> dict:
    """The plan of a problem: partition_tokens, num_partitions, workspace_bytes."""
    info = pda_plan_info()
    rc = load_library().pda_plan(ctypes.byref(prob), ctypes.byref(info))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_plan")
    return info.as_dict()


def pda_workspace_bytes(prob: pda_problem) -> int:
    ws = ctypes.c_size_t()
    rc = load_library().pda_workspace_bytes(ctypes.byref(prob), ctypes.byref(ws))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_workspace_bytes")
    return ws.value


def pda_validate_host(prob: pda_problem, block_table, context_lens) -> Tuple[int, int]:
    """Check host copies of the device contents; returns (status, first_bad_index)."""
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    lens = np.ascontiguousarray(context_lens, dtype=np.int32)
    bad = ctypes.c_int64(-1)
    rc = load_library().pda_validate_host(ctypes.byref(prob), bt.ctypes.data, lens.ctypes.data,
                                          ctypes.byref(bad))
    return rc, bad.value


def _problem_from(q, k_cache, block_table, max_context_len, partition_tokens) -> pda_problem:
    import torch

    if q.dim() != 3 or k_cache.dim() != 5 or block_table.dim() != 2:
        raise ValueError("q [B][Hq][D], k_cache [num_blocks][Hkv][D/8][16][8], block_table [B][max_blocks]")
    B, Hq, D = q.shape
    NB, Hkv, C, BS, E = k_cache.shape
    if C * E != D or E != 8 or block_table.shape[0] != B:
        raise ValueError("q, k_cache and block_table shapes disagree")
    if max_context_len is None:
        raise ValueError("max_context_len must be given (the host bound on context_lens)")
    return make_problem(B, Hq, Hkv, D, NB, block_table.shape[1], max_context_len, partition_tokens, BS)


def _check_tensors(q, k_cache, v_cache, block_table, context_lens, out):
    import torch

    for name, t, dt in (("q", q, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                        ("v_cache", v_cache, torch.bfloat16), ("block_table", block_table, torch.int32),
                        ("context_lens", context_lens, torch.int32), ("out", out, torch.float32)):
        if t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    NB, Hkv, C, BS, E = k_cache.shape
    if tuple(v_cache.shape) != (NB, Hkv, BS, C * E):
        raise ValueError("v_cache must be [num_blocks][Hkv][16][D] (k_cache is [num_blocks][Hkv][D/8][16][8])")
    if out.shape != q.shape:
        raise ValueError("out must have the shape of q")
    if context_lens.shape != (q.shape[0],):
        raise ValueError("context_lens must be [B]")


def _stream_handle(stream, device):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _step(fn_name, q, k_cache, v_cache, block_table, context_lens, scale, out, max_context_len,
          partition_tokens, workspace, stream):
    import torch

    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
    need = pda_workspace_bytes(prob)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    rc = getattr(load_library(), fn_name)(
        ctypes.byref(prob), q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
        context_lens.data_ptr(), ctypes.c_float(scale), out.data_ptr(), ws_ptr, ws_bytes,
        _stream_handle(stream, q.device))
    if rc != PDA_OK:
        raise PdaError(rc, fn_name)
    return out


def pda_decode(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
               max_context_len: int, partition_tokens: int = 0, workspace=None, stream=None):
    """One decode-attention step (both passes).  Tensors on the GPU:
    q bf16 [B][Hq][D], k_cache bf16 [num_blocks][Hkv][D/8][16][8] (each block's
    keys as D/8 chunks of 16 slots x 8 elements), v_cache bf16 [num_blocks][Hkv][16][D],
    block_table int32 [B][max_blocks], context_lens int32 [B], out fp32 [B][Hq][D].
    `workspace` (uint8, >= pda_workspace_bytes) is allocated when not given;
    partition_tokens > 0 fixes the split-K partition size."""
    return _step("pda_decode", q, k_cache, v_cache, block_table, context_lens, scale, out, max_context_len,
                 partition_tokens, workspace, stream)


def pda_partition_attention(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                            max_context_len: int, partition_tokens: int = 0, workspace=None, stream=None):
    """Pass 1 only (see pda_decode)."""
    return _step("pda_partition_attention", q, k_cache, v_cache, block_table, context_lens, scale, out,
                 max_context_len, partition_tokens, workspace, stream)


def pda_merge_partitions(prob: pda_problem, context_lens, out, workspace, stream=None):
    """Pass 2 only: merge the partial states pass 1 left in `workspace`."""
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    rc = load_library().pda_merge_partitions(ctypes.byref(prob), context_lens.data_ptr(), out.data_ptr(),
                                             ws_ptr, ws_bytes, _stream_handle(stream, out.device))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_merge_partitions")
    return out
