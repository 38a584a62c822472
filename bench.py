"""Benchmark of the rollout decode step's hot path on one MI355X.

Default (--op decode): a step is one pda_decode call (work order + pass 1 +
merge pass) over a whole batch: every sequence's new query token attends over
its paged KV cache.  The timed calls are bound once (bind_decode), as a
serving loop issues them: each step is one call into the library, which
validates the descriptor, plans the step and launches its kernels;
`ms_per_step_per_call_binding` gives the same step through the per-call
Python function (its tensor checks every step), and
`ms_per_step_order_reused` the step as a model's later layers run it
(pda_decode_reusing_order: the work order of the step's first layer
reused).  The default workload is the Llama-3-8B-shaped rollout step
(B=256, 32 query / 8 KV heads, head_dim 128, contexts uniform in [512,
4096], random block placement in a pool of the used blocks + 10%); inputs
are synthetic and already resident in HBM when the timed region
starts.

Prints one JSON line:
  value      algorithmic HBM bytes per step / step time, in GB/s
             (K and V rows of every context token -- shared rows once --
             plus q, the fp32 output, the block-table entries and lengths)
  roofline   the attention kernel (partition_kernel) alone: the same
             algorithmic bytes / its time (HIP events on its stream around
             pda_partition_attention_reusing_order, the step's pass 1 on the
             work order the step leaves in its workspace), against the 8 TB/s
             HBM peak; `ms_pass1_with_order` is pass 1 with the order kernel;
             `traffic` is the measured HBM bytes per launch from rocprofv3
             counters when they were taken on this kernel source;
             `ceiling_gbs` / `ceiling_frac`: the same K/V tiles read by a bare
             gather kernel with the same loads and no arithmetic (the practical
             read ceiling of this access pattern) and pass-1 time over it;
             `stream_read_gbs`: a contiguous read of the K and V pools
             (both read ceilings at the best of 256-8192 workgroups)
  cpu_baseline  the fp64 oracle on the host cores, same workload (and, as
             one_thread, on one core over the batch's first 16 sequences)
  ms_per_step_median / _min  single steps timed one by one (a separate pass)

Other steps around attention (--op):
  multi    n new query tokens per sequence (--tokens, default 4: verifying
           speculative-decoding drafts), same KV bytes, n times the rows
  append   the KV-cache append of the step's new tokens alone
  graph    append + attention as one captured HIP graph against the same
           calls issued eagerly from bound calls (default workload: the tiny
           batch, where launch overhead dominates)
  model_step  a model's decode step over --layers layers (default 32; each
           layer's append into its own cache and its attention, the work
           order once) as one HIP graph (with one new token, each layer's
           append folded into its pass 1) against the same work as bound
           calls issued one by one (append and attention, and the folded
           pda_decode_append): per-layer microseconds (default: tiny)
  prefix   the shared-prefix workload (32 prompts x 8 samples) with each
           prompt's prefix attended once for its samples (--tokens n: n new
           tokens per sequence, the prefix read once per 64 / (n G) samples),
           against the plain step
  logprob  log-probability of each sampled token and the entropy over the
           LM-head logits of one decode step (256 rows x 128256 Llama-3
           vocabulary, bf16; --logits-f32, --config qwen_vocab, --no-entropy);
           bound calls rotate over copies of the logits (>= 512 MB in all,
           past the 256 MB Infinity Cache), so each reads them from HBM
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_GBS = 8000.0  # MI355X HBM3E, datasheet
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, datasheet (no sparsity)
METRIC = "decode-attention HBM GB/s (% of peak) + seq-steps/s, Llama-3-8B shape"
PROFILES = os.path.join(ROOT, "profiles")
CSRC = "paper_2405_11143_amd/csrc/"
# The dominant kernel and the sources it is compiled from.
KERNEL = "partition_kernel"
KERNEL_SOURCES = {
    "partition_kernel": [CSRC + "pda_partition.hip", CSRC + "pda_wave.h", CSRC + "pda_internal.h"],
    "append_kernel": [CSRC + "pda_append.hip", CSRC + "pda_internal.h"],
    "logprob_kernel": [CSRC + "pda_logprob.hip", CSRC + "pda_internal.h"],
}


def kernel_source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when it is missing or was taken on another kernel source."""
    path = os.path.join(PROFILES, f"traffic_{kernel}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_source_hash(kernel):
        return None
    return float(m_bytes.group(1))


def host_threads() -> int:
    """Threads for the oracle: every CPU this process may run on, capped by
    OMP_NUM_THREADS when that is set (a machine's share of its host)."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return max(1, min(avail, int(env)))
    return max(1, avail)


def host_cpu_fields(threads: int) -> dict:
    """What the host offers beside the threads the oracle used."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = None
    return {"cores": threads, "host_cpus": os.cpu_count(), "cpus_available_to_process": avail,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(st, q, k, v, min_seconds: float, max_reps: int):
    import numpy as np

    import oracle
    import workloads as W

    threads = host_threads()
    qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
    reps, t_total = 0, 0.0
    while reps < max_reps and (reps == 0 or t_total < min_seconds):
        t0 = time.perf_counter()
        oracle.decode(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=threads)
        t_total += time.perf_counter() - t0
        reps += 1
    per_step = t_total / reps
    # the same oracle on one thread, over the first sequences of the batch
    nb = min(st.B, 16)
    lens = st.context_lens[:nb]
    blocks = int(((lens.astype(np.int64).clip(0) + st.block_size - 1) // st.block_size).sum())
    sub_bytes = (int(lens.astype(np.int64).clip(0).sum()) * st.Hkv * st.D * 2 * 2
                 + nb * st.Hq * st.D * (2 + 4) + blocks * 4 + nb * 4)
    reps1, t1 = 0, 0.0
    while reps1 < max_reps and (reps1 == 0 or t1 < min_seconds / 2):
        t0 = time.perf_counter()
        oracle.decode(qb[:nb], kb, vb, st.block_table[:nb], lens, st.scale, threads=1)
        t1 += time.perf_counter() - t0
        reps1 += 1
    one = t1 / reps1
    return {"value": round(st.algorithmic_bytes() / per_step / 1e9, 4), "unit": "GB/s",
            "seq_steps_per_s": round(st.B / per_step, 3), "s_per_step": round(per_step, 4),
            **host_cpu_fields(threads), "kind": "oracle",
            "sample": f"the full {st.name} step (all {st.B} sequences x {st.Hq} heads), "
                      f"{reps} repetition(s), {t_total:.1f} s total, fp64, {threads} threads",
            "one_thread": {"value": round(sub_bytes / one / 1e9, 4), "unit": "GB/s",
                           "seq_steps_per_s": round(nb / one, 3), "cores": 1,
                           "sample": f"the first {nb} sequences of the step, {reps1} repetition(s), "
                                     f"{t1:.1f} s total, fp64, 1 thread"}}


def oracle_timed(run, min_seconds: float, max_reps: int):
    """Seconds per call of `run` (the oracle on the host), repeated until
    min_seconds have passed or max_reps calls were made: (seconds, reps, total)."""
    reps, total = 0, 0.0
    while reps < max_reps and (reps == 0 or total < min_seconds):
        t0 = time.perf_counter()
        run()
        total += time.perf_counter() - t0
        reps += 1
    return total / reps, reps, total


def cpu_baseline_multi(st, q, k, v, n, min_seconds: float, max_reps: int):
    """The oracle's n-token attention on the host over the batch's first
    sequences (at most 32), in GB/s of those sequences' algorithmic bytes."""
    import numpy as np

    import oracle
    import workloads as W

    threads = host_threads()
    nb = min(st.B, 32)
    qb, kb, vb = W.bf16_bits(q)[:nb], W.bf16_bits(k), W.bf16_bits(v)
    lens = st.context_lens[:nb]
    L = lens.astype(np.int64).clip(0)
    sub_bytes = (int(L.sum()) * st.Hkv * st.D * 2 * 2 + nb * n * st.Hq * st.D * (2 + 4)
                 + int(((L + st.block_size - 1) // st.block_size).sum()) * 4 + nb * 4)
    sec, reps, total = oracle_timed(
        lambda: oracle.decode_multi(qb, kb, vb, st.block_table[:nb], lens, st.scale, threads=threads),
        min_seconds, max_reps)
    return {"value": round(sub_bytes / sec / 1e9, 4), "unit": "GB/s", **host_cpu_fields(threads), "kind": "oracle",
            "sample": f"the first {nb} sequences of the {st.name} step with {n} new tokens each, {reps} "
                      f"repetition(s), {total:.1f} s total, fp64, {threads} threads"}


def timed(fn, n, stream):
    """Average ms per call of fn over n calls, HIP events on `stream`."""
    import torch

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(n):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def timed_each(fn, n, stream):
    """Median and minimum ms of single calls of fn (HIP events around each)."""
    import torch

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    return ms[len(ms) // 2], ms[0]


def timed_graph(fn, n):
    """Average ms per call of fn with n calls captured in one HIP graph (via
    torch's graph capture; fn launches on the current stream) and replayed:
    the GPU time of the kernels without the host's per-call cost."""
    import torch

    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        for _ in range(3):
            fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(n):
            fn()
    g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def step_block_ids(st):
    """Physical ids of the blocks a step reads, each once, in first-use order."""
    import numpy as np

    nb = st.blocks_used()
    ids = np.concatenate([st.block_table[b, :int(nb[b])] for b in range(st.B)] or [np.zeros(0, np.int32)])
    _, first = np.unique(ids, return_index=True)
    return ids[np.sort(first)].astype(np.int32)


CEILING_WORKGROUPS = (256, 512, 1024, 2048, 4096, 8192)


def measure_ceilings(st, k, v, stream, reps: int):
    """HBM read ceilings of a step's traffic: the K/V tiles of every block it
    reads gathered with the attention kernel's loads and no arithmetic, and a
    contiguous stream over the K and V pools, each at the best of a few
    workgroup counts.  Returns (tile bytes, gather ms, gather workgroups,
    stream GB/s, stream workgroups)."""
    import torch

    from paper_2405_11143_amd import bind_gather_ceiling, bind_stream_ceiling

    ids = torch.from_numpy(step_block_ids(st)).to(k.device)
    tile_bytes = int(ids.numel()) * st.Hkv * 2 * st.block_size * st.D * 2
    best = None
    for wg in CEILING_WORKGROUPS:
        g = bind_gather_ceiling(ids, k, v, wg, stream=stream)
        for _ in range(3):
            g()
        ms = timed(g, reps, stream)
        if best is None or ms < best[0]:
            best = (ms, wg)
    best_stream = None
    for wg in CEILING_WORKGROUPS:
        gbs = []
        for buf in (k, v):
            sfn = bind_stream_ceiling(buf, wg, stream=stream)
            for _ in range(3):
                sfn()
            ms = timed(sfn, reps, stream)
            gbs.append(buf.numel() * buf.element_size() / (ms * 1e-3) / 1e9)
        rate = sum(gbs) / len(gbs)
        if best_stream is None or rate > best_stream[0]:
            best_stream = (rate, wg)
    return tile_bytes, best[0], best[1], best_stream[0], best_stream[1]


def ceiling_fields(st, k, v, stream, reps: int, ms_kernel: float) -> dict:
    """The attention kernel against the ceilings of its own traffic: the same
    K/V tiles gathered without arithmetic (ceiling_frac = gather time / kernel
    time, both reading whole 16-token tiles) and a contiguous stream."""
    tile_bytes, ms_g, wg, stream_gbs, stream_wg = measure_ceilings(st, k, v, stream, reps)
    return {"ceiling_gbs": round(tile_bytes / (ms_g * 1e-3) / 1e9, 2),
            "ceiling_frac": round(ms_g / ms_kernel, 4),
            "ceiling_kind": f"gather of the step's {tile_bytes} bytes of K/V tiles with the kernel's loads, "
                            f"no arithmetic ({wg} workgroups, {ms_g:.5f} ms)",
            "tile_gbs_kernel": round(tile_bytes / (ms_kernel * 1e-3) / 1e9, 2),
            "stream_read_gbs": round(stream_gbs, 2), "stream_read_workgroups": stream_wg}


def base_result(args, value, unit, ms_step, metric, config, dtype="bf16"):
    return {"metric": metric, "value": round(value, 2), "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": dtype,
            "data": "synthetic (seeded N(0,1) bf16 q/K/V, random block placement)", "config": config}


def roofline(achieved_gbs, ms, kernel, workload):
    return {"bound": "hbm", "kernel": kernel, "achieved": round(achieved_gbs, 2), "peak": PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved_gbs / PEAK_GBS, 4), "traffic": measured_traffic(kernel, workload),
            "ms_per_launch": round(ms, 5)}


def roofline_mfma(flops, ms, kernel):
    """Dense bf16 MFMA roofline of a launch whose work is bound by its
    contractions rather than by its bytes.  The kernel runs P.V twice (the
    bf16 high and low halves of the probabilities), so the MFMA work it
    issues is 1.5x the algorithmic flops (q.k once, p.v twice):
    `issued_frac` is the MFMA units' busy share that implies."""
    achieved = flops / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "kernel": kernel, "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
            "ms_per_launch": round(ms, 5), "algorithmic_flops_per_launch": int(flops),
            "issued_flops_factor": 1.5, "issued_frac": round(1.5 * achieved / PEAK_BF16_TFLOPS, 4)}


def config_of(st, cfg_desc, name, plan=None, **extra):
    c = {"workload": cfg_desc, "name": name, "batch": st.B, "q_heads": st.Hq, "kv_heads": st.Hkv,
         "head_dim": st.D, "block_size": st.block_size, "pool_blocks": st.num_blocks,
         "context_tokens": st.logical_tokens, "unique_context_tokens": st.unique_tokens}
    if plan is not None:
        c.update(partition_tokens=plan["partition_tokens"], partitions=plan["num_partitions"])
    c.update(extra)
    return c


def setup(args, n_tokens=1):
    import torch

    import workloads as W
    from paper_2405_11143_amd import make_problem, pda_plan

    dev = torch.device("cuda:0")
    st = W.make_structure(args.config)
    q, k, v = W.fill_values(st, dev, fill="nan")
    if n_tokens > 1:
        q = W.fill_multi_q(st, n_tokens, dev)
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(st.context_lens).to(dev)
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len,
                        args.partition_tokens, num_query_tokens=n_tokens)
    plan = pda_plan(prob)
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    ws = torch.empty(max(plan["workspace_bytes"], 16), dtype=torch.uint8, device=dev)
    return dev, st, q, k, v, bt, lens, plan, out, ws


def op_decode(args, n_tokens=1):
    import torch

    import workloads as W
    from paper_2405_11143_amd import bind_decode, pda_decode

    dev, st, q, k, v, bt, lens, plan, out, ws = setup(args, n_tokens)
    stream = torch.cuda.current_stream(dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=args.partition_tokens, workspace=ws,
              stream=stream)
    # A serving loop binds its buffers once: each step is then one call into
    # the library, which validates, plans and launches the whole step.
    step = bind_decode(q, k, v, bt, lens, st.scale, out, **kw)
    pass1 = bind_decode(q, k, v, bt, lens, st.scale, out, pass1_only=True, **kw)
    # a model's later layers reuse the work order the step's first call left in `ws`
    reused = bind_decode(q, k, v, bt, lens, st.scale, out, reuse_order=True, **kw)
    # the attention kernel by itself: pass 1 on the order the step's calls leave in `ws`
    kernel_only = bind_decode(q, k, v, bt, lens, st.scale, out, pass1_only=True, reuse_order=True, **kw)

    def per_call():  # the per-call binding: Python checks and descriptor every step
        pda_decode(q, k, v, bt, lens, st.scale, out, **kw)

    fn = pass1 if args.pass1_only else step
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    ms_step = timed(fn, args.steps, stream)
    ms_pass1 = ms_step if args.pass1_only else timed(pass1, args.steps, stream)
    ms_kernel = timed(kernel_only, args.steps, stream)
    ms_per_call = timed(per_call, args.steps, stream)
    ms_reused = timed(reused, args.steps, stream)
    ms_median, ms_min = timed_each(fn, args.steps, stream)  # a separate pass: one event pair per step
    alg = st.algorithmic_bytes(query_tokens=n_tokens)
    value = alg / (ms_step * 1e-3) / 1e9
    cfg = W.CONFIGS[args.config]
    if n_tokens == 1:
        metric, desc = METRIC, cfg["desc"]
    else:
        metric = f"multi-token attention HBM GB/s ({n_tokens} new tokens per sequence), {args.config} shape"
        desc = f"{cfg['desc']}; {n_tokens} new query tokens per sequence (causal)"
    result = base_result(args, value, "GB/s", ms_step, metric,
                         config_of(st, desc, args.config, plan, query_tokens=n_tokens,
                                   timed="pass1 only" if args.pass1_only else "full step"))
    result.update({"seq_steps_per_s": round(st.B / (ms_step * 1e-3), 1),
                   "ms_per_step_per_call_binding": round(ms_per_call, 5),
                   "ms_per_step_order_reused": round(ms_reused, 5),
                   "ms_per_step_median": round(ms_median, 5), "ms_per_step_min": round(ms_min, 5),
                   "ms_pass1_with_order": round(ms_pass1, 5),
                   "pct_of_peak": round(100.0 * value / PEAK_GBS, 2), "algorithmic_bytes_per_step": alg,
                   "roofline": roofline(alg / (ms_kernel * 1e-3) / 1e9, ms_kernel, KERNEL,
                                        args.config if n_tokens == 1 else f"{args.config}_x{n_tokens}"),
                   "cpu_baseline": None})
    if not args.no_ceiling:
        result["roofline"].update(ceiling_fields(st, k, v, stream, args.steps, ms_kernel))
    if n_tokens > 1:
        result["query_tokens_per_s"] = round(st.B * n_tokens / (ms_step * 1e-3), 1)
        # many new tokens make the step a contraction: then the MFMA roofline binds
        flops = st.algorithmic_flops(n_tokens)
        if flops / (PEAK_BF16_TFLOPS * 1e12) > alg / (PEAK_GBS * 1e9):
            result["roofline"] = roofline_mfma(flops, ms_kernel, KERNEL)
    if n_tokens == 1 and not args.no_cpu_baseline and not args.pass1_only:
        result["cpu_baseline"] = cpu_baseline(st, q, k, v, args.cpu_min_seconds, args.cpu_max_reps)
    elif not args.no_cpu_baseline and not args.pass1_only:
        result["cpu_baseline"] = cpu_baseline_multi(st, q, k, v, n_tokens, args.cpu_min_seconds / 2,
                                                    args.cpu_max_reps)
    return result


def op_append(args):
    import torch

    import workloads as W
    from paper_2405_11143_amd import pda_append_kv

    n = args.tokens
    dev = torch.device("cuda:0")
    st = W.make_structure(args.config)
    _, k, v = W.fill_values(st, dev, fill="nan")
    kn, vn = W.fill_new_kv(st, n, dev)
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(st.context_lens).to(dev)
    stream = torch.cuda.current_stream(dev)

    def step():  # rewrites the same slots every time, on the current stream
        pda_append_kv(kn, vn, bt, lens, k, v, max_context_len=st.max_context_len, num_q_heads=st.Hq)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms_eager = timed(step, args.steps, stream)
    ms = timed_graph(step, args.steps)
    alg = st.append_bytes(n)
    value = alg / (ms * 1e-3) / 1e9
    cfg = W.CONFIGS[args.config]
    result = base_result(args, value, "GB/s", ms, f"KV-cache append HBM GB/s ({n} new tokens per sequence)",
                         config_of(st, f"{cfg['desc']}; append of {n} new token(s) per sequence", args.config,
                                   new_tokens=n))
    result["config"]["timed"] = "HIP graph of the timed calls (GPU time); ms_per_call_eager: issued from Python"
    result.update({"seq_steps_per_s": round(st.B / (ms * 1e-3), 1), "algorithmic_bytes_per_step": alg,
                   "ms_per_call_eager": round(ms_eager, 5),
                   "roofline": roofline(value, ms, "append_kernel", args.config), "cpu_baseline": None})
    return result


def op_graph(args):
    import torch

    import workloads as W
    from paper_2405_11143_amd import StepGraph, bind_append_kv, bind_decode, pda_append_kv, pda_decode

    n = args.tokens
    dev, st, q, k, v, bt, lens, plan, out, ws = setup(args, n)
    kn, vn = W.fill_new_kv(st, n, dev)
    stream = torch.cuda.current_stream(dev)
    graph = StepGraph(q, kn, vn, k, v, bt, lens, st.scale, out, max_context_len=st.max_context_len,
                      partition_tokens=args.partition_tokens, workspace=ws)
    append = bind_append_kv(kn, vn, bt, lens, k, v, max_context_len=st.max_context_len, num_q_heads=st.Hq,
                            stream=stream)
    attend = bind_decode(q, k, v, bt, lens, st.scale, out, max_context_len=st.max_context_len,
                         partition_tokens=args.partition_tokens, workspace=ws, stream=stream)

    def eager():  # the same launches issued from bound calls
        append()
        attend()

    def replay():
        graph.launch(stream)

    def eager_current():  # the same calls on the current stream (for the GPU-time capture)
        pda_append_kv(kn, vn, bt, lens, k, v, max_context_len=st.max_context_len, num_q_heads=st.Hq)
        pda_decode(q, k, v, bt, lens, st.scale, out, max_context_len=st.max_context_len,
                   partition_tokens=args.partition_tokens, workspace=ws)

    try:
        for f in (eager, replay):
            for _ in range(args.warmup):
                f()
        torch.cuda.synchronize()
        ms_eager = timed(eager, args.steps, stream)
        ms_graph = timed(replay, args.steps, stream)
        ms_gpu = timed_graph(eager_current, args.steps)  # the kernels alone, without per-step host cost
    finally:
        graph.close()
    alg = st.algorithmic_bytes(query_tokens=n) + st.append_bytes(n)
    value = st.B / (ms_graph * 1e-3)
    cfg = W.CONFIGS[args.config]
    result = base_result(args, value, "seq-steps/s", ms_graph,
                         "decode step (append + attention) as one HIP graph, seq-steps/s",
                         config_of(st, f"{cfg['desc']}; append + attention of {n} new token(s)", args.config, plan,
                                   query_tokens=n))
    result.update({"ms_per_step_eager": round(ms_eager, 5), "graph_speedup": round(ms_eager / ms_graph, 3),
                   "ms_per_step_gpu_only": round(ms_gpu, 5),
                   "algorithmic_bytes_per_step": alg,
                   "roofline": roofline(alg / (ms_graph * 1e-3) / 1e9, ms_graph, KERNEL, args.config),
                   "cpu_baseline": None})
    return result


def op_model_step(args):
    """A model's decode step: for each of --layers layers, the KV append into
    that layer's own cache and its attention step (work order once per step),
    as bound calls issued one by one and as one captured HIP graph
    (pda_model_step_graph_create)."""
    import torch

    import workloads as W
    from paper_2405_11143_amd import BoundCall, ModelStepGraph, bind_append_kv, bind_decode
    from paper_2405_11143_amd.pda import _stream_handle

    n, nl = args.tokens, args.layers
    dev = torch.device("cuda:0")
    st = W.make_structure(args.config)
    bt = torch.from_numpy(st.block_table).to(dev)
    lens = torch.from_numpy(st.context_lens).to(dev)
    stream = torch.cuda.current_stream(dev)
    layers = []
    shared = None
    for l in range(nl):
        if shared is None or not args.shared_cache:
            _, k, v = W.fill_values(st, dev, fill="nan")
            shared = (k, v)
        k, v = shared
        q = W.fill_multi_q(st, n, dev) if n > 1 else W.fill_values(st, dev, fill="nan")[0][:, None].contiguous()
        kn, vn = W.fill_new_kv(st, n, dev)
        layers.append(dict(q=q, k_new=kn, v_new=vn, k_cache=k, v_cache=v,
                           out=torch.empty(q.shape, dtype=torch.float32, device=dev)))
    from paper_2405_11143_amd import make_problem, pda_plan
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len,
                        args.partition_tokens, num_query_tokens=n)
    plan = pda_plan(prob)
    ws = torch.empty(max(plan["workspace_bytes"], 16), dtype=torch.uint8, device=dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=args.partition_tokens, workspace=ws, stream=stream)
    order = BoundCall("pda_work_order", (ctypes_ref(prob), lens.data_ptr(), ws.data_ptr(), ws.numel(),
                                         _stream_handle(stream, dev)), (prob, lens, ws))
    calls = []
    for L in layers:
        calls.append(bind_append_kv(L["k_new"], L["v_new"], bt, lens, L["k_cache"], L["v_cache"],
                                    max_context_len=st.max_context_len, num_q_heads=st.Hq, stream=stream))
        calls.append(bind_decode(L["q"], L["k_cache"], L["v_cache"], bt, lens, st.scale, L["out"],
                                 reuse_order=True, **kw))

    def eager():  # the same work, one bound call per launch
        order()
        for c in calls:
            c()

    fused = None
    if n == 1:  # one new token: pda_decode_append folds each layer's append into its pass 1
        from paper_2405_11143_amd import bind_decode_append
        fused_calls = [bind_decode_append(L["q"], L["k_new"], L["v_new"], L["k_cache"], L["v_cache"], bt, lens,
                                          st.scale, L["out"], **kw) for L in layers]

        def fused():
            for c in fused_calls:
                c()

    graph = ModelStepGraph(layers, bt, lens, st.scale, max_context_len=st.max_context_len,
                           partition_tokens=args.partition_tokens, workspace=ws)
    try:
        for f in (eager, lambda: graph.launch(stream)):
            for _ in range(args.warmup):
                f()
        torch.cuda.synchronize()
        ms_eager = timed(eager, args.steps, stream)
        ms_graph = timed(lambda: graph.launch(stream), args.steps, stream)
        ms_fused = None
        if fused is not None:
            for _ in range(args.warmup):
                fused()
            ms_fused = timed(fused, args.steps, stream)
    finally:
        graph.close()
    alg = nl * (st.algorithmic_bytes(query_tokens=n) + st.append_bytes(n))
    cfg = W.CONFIGS[args.config]
    result = base_result(args, st.B / (ms_graph * 1e-3), "seq-steps/s", ms_graph,
                         f"{nl}-layer decode step (append + attention per layer) as one HIP graph, seq-steps/s",
                         config_of(st, f"{cfg['desc']}; {nl} layers, {n} new token(s) per sequence"
                                       + (", one cache shared by every layer" if args.shared_cache else
                                          ", a cache per layer"), args.config, plan, layers=nl, query_tokens=n))
    result.update({"us_per_layer_graph": round(1000 * ms_graph / nl, 3),
                   "us_per_layer_eager": round(1000 * ms_eager / nl, 3),
                   "ms_per_step_eager": round(ms_eager, 5), "graph_speedup": round(ms_eager / ms_graph, 3),
                   "us_per_layer_eager_folded_append": None if ms_fused is None else round(1000 * ms_fused / nl, 3),
                   "algorithmic_bytes_per_step": alg,
                   "roofline": roofline(alg / (ms_graph * 1e-3) / 1e9, ms_graph, KERNEL, args.config),
                   "cpu_baseline": None})
    return result


def ctypes_ref(x):
    import ctypes

    return ctypes.byref(x)


def op_prefix(args):
    """The shared-prefix workload with each prompt's prefix attended once per
    row group of its samples (pda_decode_shared_prefix; one or --tokens new
    tokens per sequence), against the plain step on the same inputs."""
    import torch

    import workloads as W
    from paper_2405_11143_amd import pda_decode, pda_decode_shared_prefix

    args.config = args.config if W.CONFIGS.get(args.config, {}).get("prompts") else "shared_prefix"
    n = args.tokens
    dev, st, q, k, v, bt, lens, plan, out, ws = setup(args, n)
    gs = torch.from_numpy(st.group_start).to(dev)
    gp = torch.from_numpy(st.group_prefix_len).to(dev)
    cfg = W.CONFIGS[args.config]
    stream = torch.cuda.current_stream(dev)
    kw = dict(max_context_len=st.max_context_len, partition_tokens=args.partition_tokens, stream=stream)
    out2 = torch.empty_like(out)

    def shared():
        pda_decode_shared_prefix(q, k, v, bt, lens, st.scale, gs, gp, out2, max_group_size=cfg["samples"],
                                 max_prefix_len=cfg["prefix_len"], workspace=ws_sp, **kw)

    def plain():
        pda_decode(q, k, v, bt, lens, st.scale, out, workspace=ws, **kw)

    from paper_2405_11143_amd import make_prefix_groups, make_problem, pda_plan_shared_prefix
    prob = make_problem(st.B, st.Hq, st.Hkv, st.D, st.num_blocks, st.max_blocks_per_seq, st.max_context_len,
                        args.partition_tokens, num_query_tokens=n)
    need = pda_plan_shared_prefix(prob, make_prefix_groups(len(gp), cfg["samples"], cfg["prefix_len"]))
    ws_sp = torch.empty(max(need["workspace_bytes"], 16), dtype=torch.uint8, device=dev)
    for f in (shared, plain):
        for _ in range(args.warmup):
            f()
    torch.cuda.synchronize()
    ms = timed(shared, args.steps, stream)
    ms_plain = timed(plain, args.steps, stream)
    alg = st.algorithmic_bytes(query_tokens=n)
    value = alg / (ms * 1e-3) / 1e9
    if n == 1:
        metric, extra = "shared-prefix decode HBM GB/s (unique bytes), each prompt's prefix attended once", {}
    else:
        metric = (f"shared-prefix attention HBM GB/s (unique bytes), {n} new tokens per sequence, each prompt's "
                  f"prefix attended once per {64 // (n * st.Hq // st.Hkv)} samples")
        extra = {"query_tokens": n}
    result = base_result(args, value, "GB/s", ms, metric,
                         config_of(st, cfg["desc"], args.config, need, prompts=cfg["prompts"], samples=cfg["samples"],
                                   prefix_len=cfg["prefix_len"], **extra))
    result.update({"seq_steps_per_s": round(st.B / (ms * 1e-3), 1), "pct_of_peak": round(100.0 * value / PEAK_GBS, 2),
                   "algorithmic_bytes_per_step": alg, "ms_per_step_plain_decode": round(ms_plain, 5),
                   "speedup_vs_plain_decode": round(ms_plain / ms, 3),
                   "roofline": roofline(value, ms, KERNEL, args.config + ("_shared" if n == 1 else f"_shared_x{n}")),
                   "cpu_baseline": None})
    result["roofline"]["timed"] = "the whole step: work order, pass 1 (partition_kernel) and merge"

    if n == 1 and not args.no_cpu_baseline:
        # the oracle computes the same attention (it reads each member's prefix itself); the rate is
        # per unique byte like the GPU's
        import oracle

        threads = host_threads()
        qb, kb, vb = W.bf16_bits(q), W.bf16_bits(k), W.bf16_bits(v)
        sec, reps, total = oracle_timed(
            lambda: oracle.decode(qb, kb, vb, st.block_table, st.context_lens, st.scale, threads=threads),
            args.cpu_min_seconds / 2, args.cpu_max_reps)
        result["cpu_baseline"] = {"value": round(alg / sec / 1e9, 4), "unit": "GB/s", **host_cpu_fields(threads),
                                  "kind": "oracle", "seq_steps_per_s": round(st.B / sec, 3),
                                  "sample": f"the full {st.name} step, {reps} repetition(s), {total:.1f} s "
                                            f"total, fp64, {threads} threads"}
    return result


def op_logprob(args):
    import torch

    import workloads as W
    from paper_2405_11143_amd import bind_token_logprobs

    name = args.config if args.config in W.LOGIT_CONFIGS else "llama3_vocab"
    dtype = torch.float32 if args.logits_f32 else torch.bfloat16
    dev = torch.device("cuda:0")
    x, tok = W.logits_for(name, dev, dtype)
    tokens = torch.from_numpy(tok).to(dev)
    B, V = x.shape
    lp = torch.empty(B, dtype=torch.float32, device=dev)
    ent = None if args.no_entropy else torch.empty(B, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    # One batch of logits (66 MB in bf16) fits MI355X's 256 MB Infinity Cache,
    # so back-to-back calls on one buffer would read it from there.  The
    # calls rotate over copies totalling at least 512 MB, so each reads its
    # logits from HBM.
    nbuf = args.logits_buffers or max(1, -(-512 * 2 ** 20 // (x.numel() * x.element_size())))
    bufs = [x] + [x.clone() for _ in range(nbuf - 1)]
    ws_arg = None if args.logprob_one_workgroup else "auto"
    calls = [bind_token_logprobs(xb, tokens, 1.0, entropy=not args.no_entropy, logprobs=lp, entropies=ent,
                                 stream=stream, workspace=ws_arg) for xb in bufs]  # bound once, as a serving loop would
    from paper_2405_11143_amd.pda import PDA_DTYPE_BF16, PDA_DTYPE_F32, pda_logprob_workspace_bytes
    ws_bytes = pda_logprob_workspace_bytes(B, V, PDA_DTYPE_BF16 if dtype == torch.bfloat16 else PDA_DTYPE_F32)
    slices = 1 if (args.logprob_one_workgroup or ws_bytes == 0) else ws_bytes // (16 * B)
    turn = [0]

    def step():  # on the current stream
        calls[turn[0] % nbuf]()
        turn[0] += 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms = timed(step, args.steps, stream)
    alg = B * V * x.element_size() + B * 4 + B * (4 if args.no_entropy else 8)
    value = alg / (ms * 1e-3) / 1e9
    cfg = W.LOGIT_CONFIGS[name]
    what = "token log-prob" if args.no_entropy else "token log-prob + entropy"
    result = base_result(args, value, "GB/s", ms, f"{what} HBM GB/s over the LM-head logits",
                         {"workload": cfg["desc"] + f", {str(dtype).split('.')[-1]} logits", "name": name,
                          "rows": B, "vocab": V, "logits_buffers": nbuf, "workgroups_per_row": slices},
                         dtype="bf16" if dtype == torch.bfloat16 else "f32")
    result["config"]["timed"] = "bound calls back to back on one stream"
    result.update({"rows_per_s": round(B / (ms * 1e-3), 1), "algorithmic_bytes_per_step": alg,
                   "pct_of_peak": round(100.0 * value / PEAK_GBS, 2),
                   "roofline": roofline(value, ms, "logprob_kernel", name), "cpu_baseline": None})
    if not args.no_cpu_baseline:
        import oracle

        nr = min(B, 64)  # the oracle is single-threaded: the first rows
        xh = x[:nr].float().cpu().numpy() if dtype == torch.float32 else W.bf16_bits(x[:nr])
        sec, reps, total = oracle_timed(lambda: oracle.logprob(xh, tok[:nr], 1.0, entropy=not args.no_entropy),
                                        args.cpu_min_seconds / 2, args.cpu_max_reps)
        sub = nr * V * x.element_size() + nr * 4 + nr * (4 if args.no_entropy else 8)
        result["cpu_baseline"] = {"value": round(sub / sec / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                                  "rows_per_s": round(nr / sec, 3),
                                  "sample": f"the first {nr} rows, {reps} repetition(s), {total:.1f} s total, "
                                            f"fp64, 1 thread"}
    return result


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--op", default="decode",
                    choices=["decode", "multi", "append", "graph", "model_step", "logprob", "prefix"])
    ap.add_argument("--layers", type=int, default=32, help="--op model_step: layers of the decode step")
    ap.add_argument("--shared-cache", action="store_true",
                    help="--op model_step: every layer reads (and appends to) one KV cache")
    ap.add_argument("--logits-f32", action="store_true", help="--op logprob: float32 logits (default bf16)")
    ap.add_argument("--logits-buffers", type=int, default=0,
                    help="--op logprob: copies of the logits the calls rotate over (default: >= 512 MB in all)")
    ap.add_argument("--logprob-one-workgroup", action="store_true",
                    help="--op logprob: no workspace, one workgroup per row (default: rows split over workgroups)")
    ap.add_argument("--no-entropy", action="store_true",
                    help="--op logprob: log-probabilities only (what a rollout records), no entropies")
    ap.add_argument("--config", default=None, help="workload (default: llama3_8b; tiny for --op graph)")
    ap.add_argument("--tokens", type=int, default=None,
                    help="new tokens per sequence (--op multi: 4; append, graph, prefix: 1)")
    ap.add_argument("--partition-tokens", type=int, default=0,
                    help="> 0: split-K partition size in tokens (0: the library's choice)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the read-ceiling kernels (gather of the step's tiles, contiguous stream)")
    ap.add_argument("--cpu-min-seconds", type=float, default=10.0)
    ap.add_argument("--cpu-max-reps", type=int, default=60)
    ap.add_argument("--pass1-only", action="store_true",
                    help="time and launch only the pass-1 kernels (for counter runs)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a device copy of this many MiB (counter calibration) and exit")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the decode step shards by "
              "sequence or KV head with no exchange, and the benchmark runs on a single MI355X.",
              file=sys.stderr)
        return 2
    if args.config is None:
        args.config = {"graph": "tiny", "model_step": "tiny", "logprob": "llama3_vocab",
                       "prefix": "shared_prefix"}.get(args.op, "llama3_8b")
    if args.tokens is None:
        args.tokens = 4 if args.op == "multi" else 1

    import torch

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calibration:
        n = args.copy_calibration << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "copies": 3}))
        return 0

    if args.op == "decode":
        result = op_decode(args, 1)
    elif args.op == "multi":
        result = op_decode(args, args.tokens)
    elif args.op == "append":
        result = op_append(args)
    elif args.op == "logprob":
        result = op_logprob(args)
    elif args.op == "prefix":
        result = op_prefix(args)
    elif args.op == "model_step":
        result = op_model_step(args)
    else:
        result = op_graph(args)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
