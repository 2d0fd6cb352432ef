"""Workload drivers: replay a seeded synthetic workload through the library.

Each builder creates a store, draws its inputs from ``workload`` and issues
the library calls that set the scenario up (append, fork, span marking).  The
inputs it drew are returned too, so a caller can check sampled outputs
against a reference computed from the same inputs.
"""

from __future__ import annotations

from . import sq as _sq
from . import workload as wl


def build_shared128k(tasks=8, ctx=131072, aux_private=512, parallel=256, extra_tokens=256,
                     keep_inputs=(0,), device="cuda"):
    """``tasks`` main threads of ``ctx`` tokens, each with an auxiliary thread
    forked at ctx - parallel (the main thread then decodes ``parallel`` more
    tokens) that adds ``aux_private`` tokens.  Returns (store, seqs, inputs)
    with seqs = [main_0, aux_0, main_1, aux_1, ...] and inputs[t] =
    (k, v, k_aux, v_aux) for the tasks in ``keep_inputs``."""
    import torch
    w = wl.shared128k(n_tasks=tasks, main_len=ctx, fork_at=ctx - parallel, aux_private=aux_private)
    pages_task = ctx // 16 + aux_private // 16 + 2 * (extra_tokens // 16 + 2)
    store = _sq.Store(1, 32, 8, 128, num_pages=tasks * pages_task + 64, max_seqs=2 * tasks + 4,
                      max_pages_per_seq=ctx // 16 + extra_tokens // 16 + 64, device=device)
    seqs, inputs = [], {}
    for t in range(tasks):
        k, v, ka, va = shared_task_inputs(w, t, device)
        main = store.seq_create()
        store.append(main, k[:, : w.fork_at], v[:, : w.fork_at])
        aux = store.fork(main, w.fork_at)
        store.append(main, k[:, w.fork_at:], v[:, w.fork_at:])
        store.append(aux, ka, va)
        seqs += [main, aux]
        torch.cuda.synchronize()
        if t in keep_inputs:
            inputs[t] = (k, v, ka, va)
        else:
            del k, v, ka, va
    return store, seqs, inputs


def shared_task_inputs(w, t, device="cuda"):
    """The K/V inputs of task t of a Shared128K workload (regenerable)."""
    k = wl.device_normal_bf16((1, w.main_len, 8, 128), w.seed * 1000 + 4 * t, device)
    v = wl.device_normal_bf16((1, w.main_len, 8, 128), w.seed * 1000 + 4 * t + 1, device)
    ka = wl.device_normal_bf16((1, w.aux_private, 8, 128), w.seed * 1000 + 4 * t + 2, device)
    va = wl.device_normal_bf16((1, w.aux_private, 8, 128), w.seed * 1000 + 4 * t + 3, device)
    return k, v, ka, va


def build_compaction64k(device="cuda", extra_tokens=256):
    """The 64K compaction workload: one sequence with its 40 tool spans
    marked.  Returns (store, base_seq, workload, k, v)."""
    w = wl.compaction64k()
    L = w.length
    store = _sq.Store(1, 32, 8, 128, num_pages=2 * (L // 16) + 2 * (extra_tokens // 16) + 64,
                      max_seqs=4, max_pages_per_seq=L // 16 + extra_tokens // 16 + 32,
                      device=device)
    k = wl.device_normal_bf16((1, L, 8, 128), w.seed * 1000, device)
    v = wl.device_normal_bf16((1, L, 8, 128), w.seed * 1000 + 1, device)
    base = store.seq_create()
    store.append(base, k, v)
    for c, (s, e) in enumerate(w.spans):
        store.span_mark(base, c, s, e)
    return store, base, w, k, v


def build_outlier32k(device="cuda"):
    """The 32K outlier-channel workload up to its eviction: main (30 tool
    spans) forked at its end, the auxiliary thread's 512 private tokens, then
    the main thread evicts >= 50% of its tokens.  Returns
    (store, main, aux, workload, evict_stats)."""
    w = wl.outlier32k()
    L = w.main_len
    store = _sq.Store(1, 32, 8, 128, num_pages=3 * (L // 16) + 256, max_seqs=4,
                      max_pages_per_seq=L // 16 + 128, device=device)
    main = store.seq_create()
    store.append(main, wl.to_torch_bf16(w.main_k, device), wl.to_torch_bf16(w.main_v, device))
    aux = store.fork(main, L)
    store.append(aux, wl.to_torch_bf16(w.aux_k, device), wl.to_torch_bf16(w.aux_v, device))
    for c, (s, e) in enumerate(w.spans):
        store.span_mark(main, c, s, e)
    stats = store.evict(main, w.evict_ids)
    return store, main, aux, w, stats
