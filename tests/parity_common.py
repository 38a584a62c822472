"""Helpers shared by the GPU parity tests: the bar and the host thread count.

The bar (floating point): over every compared element, max-abs error <= 8e-3
and mean-abs error <= 1e-3 against the oracle's fp64 result.
"""
import os

import numpy as np

MAX_ABS, MEAN_ABS = 8e-3, 1e-3


def host_threads() -> int:
    """Threads the oracle may use: the CPUs this process may run on, capped by
    OMP_NUM_THREADS when it is set (a machine's share of its host cores)."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # not Linux
        avail = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return max(1, min(avail, int(env)))
    return max(1, avail)


THREADS = host_threads()


def check(got, ref, what, shape_note: str = ""):
    """Assert the bar over every element of `got` against `ref` (same shape)."""
    got = np.asarray(got).astype(np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    over = f"over {shape_note} = {err.size} elements" if shape_note else f"over {err.size} elements"
    print(f"{what}: max-abs {err.max():.3e} mean-abs {err.mean():.3e} {over}", flush=True)
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, what
