"""Oracle attention over many (query rows, one KV head) jobs in CPU worker
processes.

Test infrastructure only.  The workers are fresh interpreters (``spawn``)
that import numpy and the oracle and nothing else: they never touch the GPU.
Each job carries the seeded inputs as bf16 bit patterns (uint16), which the
worker turns into their exact float64 values before calling the oracle, so
a full-size check of many rows costs one oracle evaluation per row spread
over the host's cores.
"""

from __future__ import annotations

import multiprocessing as mp
import os

import numpy as np


def _bf16_value(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def _one(job):
    from oracle import attention as oatt
    q, k_bits, v_bits, scale, group = job
    k = _bf16_value(k_bits)[:, None, :]
    v = _bf16_value(v_bits)[:, None, :]
    return oatt.attention(q, k, v, scale, group)


def workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def attention_many(jobs):
    """jobs: [(q f64 [G, D], k bf16 bits uint16 [L, D], v bits [L, D], scale,
    G)]; returns the oracle's [G, D] output of each, in order."""
    if not jobs:
        return []
    ctx = mp.get_context("spawn")
    with ctx.Pool(min(workers(), len(jobs))) as pool:
        return pool.map(_one, jobs, chunksize=1)
