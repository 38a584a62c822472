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
from typing import Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpda.so")

PDA_OK, PDA_ERR_NULL, PDA_ERR_SHAPE, PDA_ERR_UNSUPPORTED = 0, 1, 2, 3
PDA_ERR_WORKSPACE, PDA_ERR_ALIGNMENT, PDA_ERR_VALUE, PDA_ERR_HIP, PDA_ERR_SCRATCH = 4, 5, 6, 7, 8
PDA_NOALLOC_SCRATCH_BYTES = 64 << 20  # the static scratch of pda_decode_noalloc

# Every function include/pda.h declares.
EXPORTED = ("pda_plan", "pda_workspace_bytes", "pda_decode", "pda_partition_attention",
            "pda_merge_partitions", "pda_plan_shared_prefix", "pda_decode_shared_prefix", "pda_append_kv",
            "pda_step_graph_create", "pda_step_graph_launch", "pda_step_graph_destroy", "pda_token_logprobs",
            "pda_logprob_workspace_bytes",
            "pda_validate_host", "pda_work_order", "pda_decode_reusing_order",
            "pda_partition_attention_reusing_order", "pda_decode_noalloc",
            "pda_gather_ceiling", "pda_stream_ceiling", "pda_model_step_graph_create", "pda_decode_append",
            "pda_status_string")
PDA_DTYPE_BF16, PDA_DTYPE_F32 = 0, 1


class pda_problem(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "num_seqs", "num_q_heads", "num_kv_heads", "head_dim", "block_size", "num_blocks",
        "max_blocks_per_seq", "max_context_len", "partition_tokens", "num_query_tokens")]


class pda_plan_info(ctypes.Structure):
    _fields_ = [("partition_tokens", ctypes.c_int32), ("num_partitions", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class pda_prefix_groups(ctypes.Structure):
    _fields_ = [("num_groups", ctypes.c_int32), ("max_group_size", ctypes.c_int32),
                ("max_prefix_len", ctypes.c_int32), ("group_start", ctypes.c_void_p),
                ("group_prefix_len", ctypes.c_void_p)]


class pda_layer_buffers(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p),
                ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p), ("out", ctypes.c_void_p)]


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
    lib.pda_decode_reusing_order.argtypes = step
    lib.pda_partition_attention_reusing_order.argtypes = step
    lib.pda_decode_noalloc.argtypes = [P, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp]
    lib.pda_gather_ceiling.argtypes = [i32, i32, i32, vp, vp, vp, i32, i32, vp, vp]
    lib.pda_stream_ceiling.argtypes = [vp, sz, i32, vp, vp]
    lib.pda_work_order.argtypes = [P, vp, vp, sz, vp]
    lib.pda_merge_partitions.argtypes = [P, vp, vp, vp, sz, vp]
    G = ctypes.POINTER(pda_prefix_groups)
    lib.pda_plan_shared_prefix.argtypes = [P, G, ctypes.POINTER(pda_plan_info)]
    lib.pda_decode_shared_prefix.argtypes = [P, G, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, sz, vp]
    lib.pda_append_kv.argtypes = [P, vp, vp, vp, vp, vp, vp, vp]
    lib.pda_decode_append.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, sz, vp]
    lib.pda_step_graph_create.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, sz,
                                          ctypes.POINTER(vp)]
    lib.pda_step_graph_launch.argtypes = [vp, vp]
    lib.pda_model_step_graph_create.argtypes = [P, ctypes.c_int32, ctypes.POINTER(pda_layer_buffers), vp, vp,
                                                ctypes.c_float, vp, sz, ctypes.POINTER(vp)]
    lib.pda_step_graph_destroy.argtypes = [vp]
    lib.pda_token_logprobs.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, ctypes.c_int32, vp, vp,
                                       ctypes.c_float, vp, vp, vp, sz, vp]
    lib.pda_logprob_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(sz)]
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
                 max_context_len, partition_tokens=0, block_size=16, num_query_tokens=1) -> pda_problem:
    return pda_problem(int(num_seqs), int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size),
                       int(num_blocks), int(max_blocks_per_seq), int(max_context_len), int(partition_tokens),
                       int(num_query_tokens))


def pda_plan(prob: pda_problem) -> dict:
    """The plan of a problem: partition_tokens, num_partitions, workspace_bytes."""
    info = pda_plan_info()
    rc = load_library().pda_plan(ctypes.byref(prob), ctypes.byref(info))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_plan")
    return info.as_dict()


def make_prefix_groups(num_groups, max_group_size, max_prefix_len, group_start=None,
                       group_prefix_len=None) -> pda_prefix_groups:
    """Host bounds plus the two device arrays (torch int32 tensors or raw pointers)."""
    ptr = lambda t: (t.data_ptr() if hasattr(t, "data_ptr") else t)
    return pda_prefix_groups(int(num_groups), int(max_group_size), int(max_prefix_len), ptr(group_start),
                             ptr(group_prefix_len))


def pda_plan_shared_prefix(prob: pda_problem, groups: pda_prefix_groups) -> dict:
    info = pda_plan_info()
    rc = load_library().pda_plan_shared_prefix(ctypes.byref(prob), ctypes.byref(groups), ctypes.byref(info))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_plan_shared_prefix")
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


def _query_shape(q):
    """(B, n, Hq, D) of q [B][Hq][D] (n = 1) or [B][n][Hq][D]."""
    if q.dim() == 3:
        return q.shape[0], 1, q.shape[1], q.shape[2]
    if q.dim() == 4:
        return tuple(q.shape)
    raise ValueError("q must be [B][Hq][D] or [B][n][Hq][D]")


def _problem_from(q, k_cache, block_table, max_context_len, partition_tokens) -> pda_problem:
    if k_cache.dim() != 5 or block_table.dim() != 2:
        raise ValueError("k_cache [num_blocks][Hkv][D/8][16][8], block_table [B][max_blocks]")
    B, n, Hq, D = _query_shape(q)
    NB, Hkv, C, BS, E = k_cache.shape
    if C * E != D or E != 8 or block_table.shape[0] != B:
        raise ValueError("q, k_cache and block_table shapes disagree")
    if max_context_len is None:
        raise ValueError("max_context_len must be given (the host bound on context_lens)")
    return make_problem(B, Hq, Hkv, D, NB, block_table.shape[1], max_context_len, partition_tokens, BS, n)


def _require(name, t, dtype):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_tensors(q, k_cache, v_cache, block_table, context_lens, out):
    import torch

    for name, t, dt in (("q", q, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                        ("v_cache", v_cache, torch.bfloat16), ("block_table", block_table, torch.int32),
                        ("context_lens", context_lens, torch.int32), ("out", out, torch.float32)):
        _require(name, t, dt)
    NB, Hkv, C, BS, E = k_cache.shape
    if tuple(v_cache.shape) != (NB, Hkv, BS, C * E):
        raise ValueError("v_cache must be [num_blocks][Hkv][16][D] (k_cache is [num_blocks][Hkv][D/8][16][8])")
    if out.shape != q.shape:
        raise ValueError("out must have the shape of q")
    if context_lens.shape != (q.shape[0],):
        raise ValueError("context_lens must be [B]")


def _check_new_kv(k_new, v_new, q_shape, k_cache):
    import torch

    _require("k_new", k_new, torch.bfloat16)
    _require("v_new", v_new, torch.bfloat16)
    B, n, _, D = q_shape
    Hkv = k_cache.shape[1]
    if tuple(k_new.shape) != (B, n, Hkv, D) or tuple(v_new.shape) != (B, n, Hkv, D):
        raise ValueError(f"k_new and v_new must be [B][n][Hkv][D] = {(B, n, Hkv, D)}")


def _stream_handle(stream, device):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _workspace(prob, workspace, device):
    import torch

    need = pda_workspace_bytes(prob)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    return workspace, ws_ptr, ws_bytes


def _step(fn_name, q, k_cache, v_cache, block_table, context_lens, scale, out, max_context_len,
          partition_tokens, workspace, stream):
    return bind_decode(q, k_cache, v_cache, block_table, context_lens, scale, out, max_context_len=max_context_len,
                       partition_tokens=partition_tokens, workspace=workspace, stream=stream,
                       pass1_only=fn_name == "pda_partition_attention")()


def pda_decode(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
               max_context_len: int, partition_tokens: int = 0, workspace=None, stream=None):
    """One attention step (both passes).  Tensors on the GPU: q bf16
    [B][Hq][D] (a decode step) or [B][n][Hq][D] (n new tokens per sequence,
    the last n of its context, attending causally), k_cache bf16
    [num_blocks][Hkv][D/8][16][8] (each block's keys as D/8 chunks of 16 slots
    x 8 elements), v_cache bf16 [num_blocks][Hkv][16][D], block_table int32
    [B][max_blocks], context_lens int32 [B], out fp32 shaped like q.
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


def pda_append_kv(k_new, v_new, block_table, context_lens, k_cache, v_cache, *, max_context_len: int,
                  num_q_heads: int = None, stream=None):
    """Store the K/V rows of each sequence's n new tokens (bf16 [B][n][Hkv][D])
    at positions L - n .. L - 1 of its paged cache, in place."""
    bind_append_kv(k_new, v_new, block_table, context_lens, k_cache, v_cache, max_context_len=max_context_len,
                   num_q_heads=num_q_heads, stream=stream)()


class BoundCall:
    """One entry point with its arguments bound once, for a serving loop that
    runs the same step on the same buffers again and again: the Python checks,
    the problem descriptor, the workspace and the stream are prepared when the
    call is built, and each call is then a single foreign-function call (the
    library still validates the descriptor, plans the step and launches its
    kernels every time).  The bound tensors are kept alive and must keep their
    storage; their contents may change between calls."""

    def __init__(self, fn_name, args, keep, result=None):
        self._fn = getattr(load_library(), fn_name)
        self._name = fn_name
        self._args = args
        self._keep = keep
        self.result = result

    def __call__(self):
        rc = self._fn(*self._args)
        if rc != PDA_OK:
            raise PdaError(rc, self._name)
        return self.result


def bind_decode(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *, max_context_len: int,
                partition_tokens: int = 0, workspace=None, stream=None, pass1_only: bool = False,
                reuse_order: bool = False) -> BoundCall:
    """pda_decode (or, with pass1_only, pda_partition_attention; with
    reuse_order, pda_decode_reusing_order; with both,
    pda_partition_attention_reusing_order) bound to these tensors and the
    given (else the current) stream; call it to run a step.  The arguments
    are those of pda_decode."""
    import torch

    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
    workspace, ws_ptr, ws_bytes = _workspace(prob, workspace, q.device)
    args = (ctypes.byref(prob), q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
            context_lens.data_ptr(), ctypes.c_float(scale), out.data_ptr(), ws_ptr, ws_bytes,
            _stream_handle(stream, q.device))
    keep = (prob, q, k_cache, v_cache, block_table, context_lens, out, workspace)
    name = {(False, False): "pda_decode", (True, False): "pda_partition_attention",
            (False, True): "pda_decode_reusing_order",
            (True, True): "pda_partition_attention_reusing_order"}[(bool(pass1_only), bool(reuse_order))]
    return BoundCall(name, args, keep, out)


def bind_decode_append(q, k_new, v_new, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                       max_context_len: int, partition_tokens: int = 0, workspace=None, stream=None) -> BoundCall:
    """pda_decode_append bound to these tensors: the append of each sequence's
    new token (k_new/v_new bf16 [B][1][Hkv][D]) folded into the decode step."""
    import torch

    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    _check_new_kv(k_new, v_new, _query_shape(q), k_cache)
    prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
    workspace, ws_ptr, ws_bytes = _workspace(prob, workspace, q.device)
    args = (ctypes.byref(prob), q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(),
            v_cache.data_ptr(), block_table.data_ptr(), context_lens.data_ptr(), ctypes.c_float(scale),
            out.data_ptr(), ws_ptr, ws_bytes, _stream_handle(stream, q.device))
    keep = (prob, q, k_new, v_new, k_cache, v_cache, block_table, context_lens, out, workspace)
    return BoundCall("pda_decode_append", args, keep, out)


def pda_decode_append(q, k_new, v_new, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                      max_context_len: int, partition_tokens: int = 0, workspace=None, stream=None):
    """pda_append_kv + pda_decode in the launches of pda_decode alone (one new
    token per sequence)."""
    return bind_decode_append(q, k_new, v_new, k_cache, v_cache, block_table, context_lens, scale, out,
                              max_context_len=max_context_len, partition_tokens=partition_tokens,
                              workspace=workspace, stream=stream)()


def pda_work_order(prob: pda_problem, context_lens, workspace, stream=None):
    """The step's work order into `workspace` (see include/pda.h): computed
    once per decode step, reused by every layer's pda_decode_reusing_order."""
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    rc = load_library().pda_work_order(ctypes.byref(prob), context_lens.data_ptr(),
                                       workspace.data_ptr() if workspace is not None else None, ws_bytes,
                                       _stream_handle(stream, context_lens.device))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_work_order")


def pda_decode_reusing_order(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                             max_context_len: int, partition_tokens: int = 0, workspace, stream=None):
    """pda_decode with the work order already in `workspace` (pda_work_order
    or an earlier pda_decode on it, same descriptor)."""
    return bind_decode(q, k_cache, v_cache, block_table, context_lens, scale, out, max_context_len=max_context_len,
                       partition_tokens=partition_tokens, workspace=workspace, stream=stream, reuse_order=True)()


def bind_decode_noalloc(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                        max_context_len: int, partition_tokens: int = 0, stream=None) -> BoundCall:
    """pda_decode_noalloc bound to these tensors and the given (else the
    current) stream: the step of pda_decode with its workspace in the
    library's static scratch, so no call allocates (`out` is allocated here,
    once, when not given)."""
    import torch

    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
    args = (ctypes.byref(prob), q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
            context_lens.data_ptr(), ctypes.c_float(scale), out.data_ptr(), _stream_handle(stream, q.device))
    return BoundCall("pda_decode_noalloc", args, (prob, q, k_cache, v_cache, block_table, context_lens, out), out)


def pda_decode_noalloc(q, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                       max_context_len: int, partition_tokens: int = 0, stream=None):
    """pda_decode without a workspace argument (see include/pda.h): raises
    PdaError with PDA_ERR_SCRATCH when the step needs more than
    PDA_NOALLOC_SCRATCH_BYTES of workspace."""
    return bind_decode_noalloc(q, k_cache, v_cache, block_table, context_lens, scale, out,
                               max_context_len=max_context_len, partition_tokens=partition_tokens, stream=stream)()


def bind_append_kv(k_new, v_new, block_table, context_lens, k_cache, v_cache, *, max_context_len: int,
                   num_q_heads: int = None, stream=None) -> BoundCall:
    """pda_append_kv bound to these tensors and the given (else the current)
    stream; the arguments are those of pda_append_kv."""
    import torch

    if k_new.dim() != 4:
        raise ValueError("k_new must be [B][n][Hkv][D]")
    B, n, Hkv, D = k_new.shape
    for name, t, dt in (("k_cache", k_cache, torch.bfloat16), ("v_cache", v_cache, torch.bfloat16),
                        ("block_table", block_table, torch.int32), ("context_lens", context_lens, torch.int32)):
        _require(name, t, dt)
    q_shape = (B, n, Hkv if num_q_heads is None else num_q_heads, D)
    _check_new_kv(k_new, v_new, q_shape, k_cache)
    NB, Hkv_c, C, BS, E = k_cache.shape
    if Hkv_c != Hkv or C * E != D or tuple(v_cache.shape) != (NB, Hkv, BS, D):
        raise ValueError("k_new/v_new and the caches disagree")
    if block_table.dim() != 2 or block_table.shape[0] != B or context_lens.shape != (B,):
        raise ValueError("block_table [B][max_blocks], context_lens [B]")
    prob = make_problem(B, q_shape[2], Hkv, D, NB, block_table.shape[1], max_context_len, 0, BS, n)
    args = (ctypes.byref(prob), k_new.data_ptr(), v_new.data_ptr(), block_table.data_ptr(), context_lens.data_ptr(),
            k_cache.data_ptr(), v_cache.data_ptr(), _stream_handle(stream, k_cache.device))
    keep = (prob, k_new, v_new, block_table, context_lens, k_cache, v_cache)
    return BoundCall("pda_append_kv", args, keep)


class ModelStepGraph:
    """pda_model_step_graph_create: a model's decode step over `layers` (a list
    of dicts with q, k_new, v_new, k_cache, v_cache and out tensors, one per
    layer) captured as one HIP graph -- per layer the KV append and the
    attention step, the work order computed once.  launch() replays it on a
    stream and reads the buffers' current contents."""

    def __init__(self, layers, block_table, context_lens, scale: float, *, max_context_len: int,
                 partition_tokens: int = 0, workspace=None):
        import torch

        if not layers:
            raise ValueError("at least one layer")
        arr = (pda_layer_buffers * len(layers))()
        for i, L in enumerate(layers):
            _check_tensors(L["q"], L["k_cache"], L["v_cache"], block_table, context_lens, L["out"])
            _check_new_kv(L["k_new"], L["v_new"], _query_shape(L["q"]), L["k_cache"])
            arr[i] = pda_layer_buffers(L["q"].data_ptr(), L["k_new"].data_ptr(), L["v_new"].data_ptr(),
                                       L["k_cache"].data_ptr(), L["v_cache"].data_ptr(), L["out"].data_ptr())
        L0 = layers[0]
        self.prob = _problem_from(L0["q"], L0["k_cache"], block_table, max_context_len, partition_tokens)
        workspace, ws_ptr, ws_bytes = _workspace(self.prob, workspace, L0["q"].device)
        self.workspace, self._device = workspace, L0["q"].device
        self._keep = (layers, block_table, context_lens, arr)
        handle = ctypes.c_void_p()
        rc = load_library().pda_model_step_graph_create(
            ctypes.byref(self.prob), len(layers), arr, block_table.data_ptr(), context_lens.data_ptr(),
            ctypes.c_float(scale), ws_ptr, ws_bytes, ctypes.byref(handle))
        if rc != PDA_OK:
            raise PdaError(rc, "pda_model_step_graph_create")
        self._handle = handle

    def launch(self, stream=None):
        rc = load_library().pda_step_graph_launch(self._handle, _stream_handle(stream, self._device))
        if rc != PDA_OK:
            raise PdaError(rc, "pda_step_graph_launch")

    def close(self):
        if getattr(self, "_handle", None) is not None:
            rc = load_library().pda_step_graph_destroy(self._handle)
            self._handle = None
            if rc != PDA_OK:
                raise PdaError(rc, "pda_step_graph_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class StepGraph:
    """pda_step_graph: append + attention captured once as a HIP graph over
    fixed buffers.  launch() replays it on a stream and reads the buffers'
    current contents.  The tensors are kept alive for the graph's lifetime."""

    def __init__(self, q, k_new, v_new, k_cache, v_cache, block_table, context_lens, scale: float, out=None, *,
                 max_context_len: int, partition_tokens: int = 0, workspace=None):
        import torch

        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
        _check_new_kv(k_new, v_new, _query_shape(q), k_cache)
        self.prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
        workspace, ws_ptr, ws_bytes = _workspace(self.prob, workspace, q.device)
        self.out, self.workspace = out, workspace
        self._keep = (q, k_new, v_new, k_cache, v_cache, block_table, context_lens)
        handle = ctypes.c_void_p()
        rc = load_library().pda_step_graph_create(
            ctypes.byref(self.prob), q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(),
            v_cache.data_ptr(), block_table.data_ptr(), context_lens.data_ptr(), ctypes.c_float(scale),
            out.data_ptr(), ws_ptr, ws_bytes, ctypes.byref(handle))
        if rc != PDA_OK:
            raise PdaError(rc, "pda_step_graph_create")
        self._handle = handle

    def launch(self, stream=None):
        rc = load_library().pda_step_graph_launch(self._handle, _stream_handle(stream, self.out.device))
        if rc != PDA_OK:
            raise PdaError(rc, "pda_step_graph_launch")
        return self.out

    def close(self):
        if getattr(self, "_handle", None) is not None:
            rc = load_library().pda_step_graph_destroy(self._handle)
            self._handle = None
            if rc != PDA_OK:
                raise PdaError(rc, "pda_step_graph_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def pda_logprob_workspace_bytes(rows: int, vocab: int, dtype: int) -> int:
    ws = ctypes.c_size_t()
    rc = load_library().pda_logprob_workspace_bytes(int(rows), int(vocab), int(dtype), ctypes.byref(ws))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_logprob_workspace_bytes")
    return ws.value


def bind_token_logprobs(logits, tokens, inv_temperature: float = 1.0, entropy: bool = True, vocab: int = None,
                        logprobs=None, entropies=None, stream=None, workspace="auto") -> BoundCall:
    """pda_token_logprobs bound to these tensors and the given (else the
    current) stream; calling it returns (logprobs, entropies or None).  The
    arguments are those of pda_token_logprobs; `workspace` is "auto" (a uint8
    tensor of pda_logprob_workspace_bytes, allocated here once), None (one
    workgroup per row) or a caller's uint8 device tensor."""
    import torch

    if logits.dim() != 2 or logits.stride(1) != 1:
        raise ValueError("logits must be [rows][row_stride] with unit element stride")
    if logits.dtype == torch.bfloat16:
        dtype = PDA_DTYPE_BF16
    elif logits.dtype == torch.float32:
        dtype = PDA_DTYPE_F32
    else:
        raise TypeError("logits must be bfloat16 or float32")
    _require("tokens", tokens, torch.int32)
    if not logits.is_cuda:
        raise ValueError("logits must be a device tensor")
    rows = logits.shape[0]
    vocab = logits.shape[1] if vocab is None else int(vocab)
    if tokens.shape != (rows,):
        raise ValueError("tokens must be [rows]")
    if logprobs is None:
        logprobs = torch.empty(rows, dtype=torch.float32, device=logits.device)
    if entropy and entropies is None:
        entropies = torch.empty(rows, dtype=torch.float32, device=logits.device)
    if isinstance(workspace, str):
        need = pda_logprob_workspace_bytes(rows, vocab, dtype) if vocab >= 1 else 0
        workspace = torch.empty(need, dtype=torch.uint8, device=logits.device) if need > 0 else None
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    args = (rows, vocab, logits.stride(0), dtype, logits.data_ptr(), tokens.data_ptr(),
            ctypes.c_float(inv_temperature), logprobs.data_ptr(), entropies.data_ptr() if entropy else None,
            ws_ptr, ws_bytes, _stream_handle(stream, logits.device))
    keep = (logits, tokens, logprobs, entropies, workspace)
    return BoundCall("pda_token_logprobs", args, keep, (logprobs, entropies if entropy else None))


def pda_token_logprobs(logits, tokens, inv_temperature: float = 1.0, entropy: bool = True, vocab: int = None,
                       logprobs=None, entropies=None, stream=None, workspace="auto"):
    """Log-probability of tokens[r] under softmax(logits[r][:vocab] * inv_temperature),
    and the entropy of that distribution (natural-log units).  logits: a device
    tensor [rows][row_stride] of bf16 or float32 (16-byte aligned rows); tokens
    int32 [rows].  Returns (logprobs fp32 [rows], entropies fp32 [rows] or None)."""
    return bind_token_logprobs(logits, tokens, inv_temperature, entropy, vocab, logprobs, entropies, stream,
                               workspace)()


def pda_decode_shared_prefix(q, k_cache, v_cache, block_table, context_lens, scale: float, group_start,
                             group_prefix_len, out=None, *, max_context_len: int, max_group_size: int,
                             max_prefix_len: int, partition_tokens: int = 0, workspace=None, stream=None):
    """The decode step with each shared-prefix group's prefix attended once for
    all its members.  group_start int32 [num_groups + 1] and group_prefix_len
    int32 [num_groups] are device tensors; max_group_size and max_prefix_len
    are their host bounds (n * G <= 64; groups larger than 64 / (n G) members
    read the prefix once per 64 / (n G) members).  Other arguments
    as pda_decode (q [B][Hq][D], or [B][n][Hq][D] for n new tokens)."""
    import torch

    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_tensors(q, k_cache, v_cache, block_table, context_lens, out)
    _require("group_start", group_start, torch.int32)
    _require("group_prefix_len", group_prefix_len, torch.int32)
    num_groups = group_prefix_len.shape[0]
    if group_start.shape != (num_groups + 1,):
        raise ValueError("group_start must be [num_groups + 1]")
    prob = _problem_from(q, k_cache, block_table, max_context_len, partition_tokens)
    groups = make_prefix_groups(num_groups, max_group_size, max_prefix_len, group_start, group_prefix_len)
    need = pda_plan_shared_prefix(prob, groups)["workspace_bytes"]
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    rc = load_library().pda_decode_shared_prefix(
        ctypes.byref(prob), ctypes.byref(groups), q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
        block_table.data_ptr(), context_lens.data_ptr(), ctypes.c_float(scale), out.data_ptr(), ws_ptr, ws_bytes,
        _stream_handle(stream, q.device))
    if rc != PDA_OK:
        raise PdaError(rc, "pda_decode_shared_prefix")
    return out


def bind_gather_ceiling(block_ids, k_cache, v_cache, workgroups: int, sink=None, stream=None) -> BoundCall:
    """pda_gather_ceiling (include/pda_ceiling.h) bound to these tensors: read
    the K and V tiles of every KV head of the listed physical blocks (device
    int32 [n]) with the attention kernel's loads and no arithmetic."""
    import torch

    _require("block_ids", block_ids, torch.int32)
    _require("k_cache", k_cache, torch.bfloat16)
    _require("v_cache", v_cache, torch.bfloat16)
    if sink is None:
        sink = torch.empty(4 * workgroups, dtype=torch.int32, device=k_cache.device)
    NB, Hkv, C, BS, E = k_cache.shape
    args = (int(Hkv), int(C * E), int(NB), k_cache.data_ptr(), v_cache.data_ptr(), block_ids.data_ptr(),
            int(block_ids.numel()), int(workgroups), sink.data_ptr(), _stream_handle(stream, k_cache.device))
    return BoundCall("pda_gather_ceiling", args, (block_ids, k_cache, v_cache, sink), sink)


def bind_stream_ceiling(buf, workgroups: int, sink=None, stream=None) -> BoundCall:
    """pda_stream_ceiling bound to a contiguous device tensor: read all its
    bytes with 16-byte non-temporal loads."""
    import torch

    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    if sink is None:
        sink = torch.empty(4 * workgroups, dtype=torch.int32, device=buf.device)
    nbytes = buf.numel() * buf.element_size() // 16 * 16
    args = (buf.data_ptr(), ctypes.c_size_t(nbytes), int(workgroups), sink.data_ptr(),
            _stream_handle(stream, buf.device))
    return BoundCall("pda_stream_ceiling", args, (buf, sink), sink)
