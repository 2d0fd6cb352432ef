"""Workload drivers: replay a seeded synthetic workload through the library.

Each builder creates a store, draws its inputs from ``workload`` and issues
the library calls that set the scenario up (append, fork, span marking).  The
inputs it drew are returned too, so a caller can check sampled outputs
against a reference computed from the same inputs.
"""

from __future__ import annotations

import time

from . import sq as _sq
from . import workload as wl


def build_shared128k(tasks=8, ctx=131072, aux_private=512, parallel=256, extra_tokens=256,
                     keep_inputs=(0,), device="cuda", layers=1, heads=(32, 8, 128),
                     kv_scales=None):
    """``tasks`` main threads of ``ctx`` tokens, each with an auxiliary thread
    forked at ctx - parallel (the main thread then decodes ``parallel`` more
    tokens) that adds ``aux_private`` tokens.  Returns (store, seqs, inputs)
    with seqs = [main_0, aux_0, main_1, aux_1, ...] and inputs[t] =
    (k, v, k_aux, v_aux) for the tasks in ``keep_inputs``.  heads = (query
    heads, KV heads, head_dim); kv_scales: an 8-bit store's [layers][2] scales."""
    import torch
    w = wl.shared128k(n_tasks=tasks, main_len=ctx, fork_at=ctx - parallel, aux_private=aux_private)
    pages_task = ctx // 16 + aux_private // 16 + 2 * (extra_tokens // 16 + 2)
    hq, hkv, d = heads
    store = _sq.Store(layers, hq, hkv, d, num_pages=tasks * pages_task + 64, max_seqs=2 * tasks + 4,
                      max_pages_per_seq=ctx // 16 + extra_tokens // 16 + 64, device=device,
                      kv_scales=kv_scales)
    seqs, inputs = [], {}
    for t in range(tasks):
        k, v, ka, va = shared_task_inputs(w, t, device, layers, hkv, d)
        main = store.seq_create()
        cut = lambda x, a, b: x[:, a:b].contiguous() if layers > 1 else x[:, a:b]
        store.append(main, cut(k, 0, w.fork_at), cut(v, 0, w.fork_at))
        aux = store.fork(main, w.fork_at)
        store.append(main, cut(k, w.fork_at, None), cut(v, w.fork_at, None))
        store.append(aux, ka, va)
        seqs += [main, aux]
        torch.cuda.synchronize()
        if t in keep_inputs:
            inputs[t] = (k, v, ka, va)
        else:
            del k, v, ka, va
    return store, seqs, inputs


def shared_task_inputs(w, t, device="cuda", layers=1, hkv=8, d=128):
    """The K/V inputs of task t of a Shared128K workload (regenerable)."""
    k = wl.device_normal_bf16((layers, w.main_len, hkv, d), w.seed * 1000 + 4 * t, device)
    v = wl.device_normal_bf16((layers, w.main_len, hkv, d), w.seed * 1000 + 4 * t + 1, device)
    ka = wl.device_normal_bf16((layers, w.aux_private, hkv, d), w.seed * 1000 + 4 * t + 2, device)
    va = wl.device_normal_bf16((layers, w.aux_private, hkv, d), w.seed * 1000 + 4 * t + 3, device)
    return k, v, ka, va


def build_compaction64k(device="cuda", extra_tokens=256, evict_chunk_pages=0, align=0,
                        evict_remap=False, evict_inplace=False):
    """The 64K compaction workload: one sequence with its 40 tool spans
    marked (with ``align`` > 0 each span's ends rounded down to a multiple of
    it, as when every tool response starts on a page).  Returns (store,
    base_seq, workload, k, v)."""
    w = wl.compaction64k()
    L = w.length
    store = _sq.Store(1, 32, 8, 128, num_pages=2 * (L // 16) + 2 * (extra_tokens // 16) + 64,
                      max_seqs=4, max_pages_per_seq=L // 16 + extra_tokens // 16 + 32,
                      device=device, evict_chunk_pages=evict_chunk_pages, evict_remap=evict_remap,
                      **({"evict_inplace": True} if evict_inplace else {}))
    k = wl.device_normal_bf16((1, L, 8, 128), w.seed * 1000, device)
    v = wl.device_normal_bf16((1, L, 8, 128), w.seed * 1000 + 1, device)
    base = store.seq_create()
    store.append(base, k, v)
    for c, (s, e) in enumerate(w.spans):
        if align:
            s, e = s // align * align, e // align * align
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


def full_stack_inputs(w, turn, device="cuda"):
    """K/V of main-thread turn ``turn`` ([NL, turn_len, 8, 128] each) and of
    the auxiliary thread forked at that turn ([NL, aux_private, 8, 128]).
    turn = -1 gives the prefix ([NL, prefix, 8, 128])."""
    n = w.prefix if turn < 0 else w.turn_len
    base = w.seed * 1000 + 4 * (turn + 1)
    k = wl.device_normal_bf16((w.num_layers, n, 8, 128), base, device)
    v = wl.device_normal_bf16((w.num_layers, n, 8, 128), base + 1, device)
    return k, v


def full_stack_aux_inputs(w, turn, device="cuda"):
    base = w.seed * 1000 + 4 * (turn + 1) + 2
    k = wl.device_normal_bf16((w.num_layers, w.aux_private, 8, 128), base, device)
    v = wl.device_normal_bf16((w.num_layers, w.aux_private, 8, 128), base + 1, device)
    return k, v


def _extend_all_layers(store, seq, n, num_layers, seed, device):
    """Causal extend attention of seq's last n tokens on every layer (one
    query tensor reused across layers); returns the elapsed ms."""
    import torch
    q = wl.device_normal_bf16((n, store.num_q_heads, store.head_dim), seed, device)
    out = torch.empty(q.shape, dtype=torch.float32, device=device)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for layer in range(num_layers):
        store.extend(layer, seq, q, out=out)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3


def run_full_stack(evict=True, turns=30, turn_len=8192, prefix=16384, num_layers=36,
                   device="cuda", decode=True, on_turn=None, store=None, evict_chunk_pages=0,
                   extend=False, evict_inplace=False):
    """Algorithm 1 over a synthetic task: a non-evictable prefix, then turns
    of reasoning plus one tool response each.  Phase 1 evicts the cursors the
    auxiliary thread named (when it has finished) and releases it; Phase 2
    forks a new auxiliary thread every ``interval`` turns, which appends its
    private tokens and names seeded-random live tool spans until at least
    60% of the live tool tokens are covered; Phase 3 appends the turn.
    With ``decode``, one decode step ([main] or [main, aux], every layer) is
    timed at the end of each turn (median of three after an untimed one; the
    steps read the cache and change nothing) and ``on_turn(t, store, seqs,
    q, out)`` is called after it.  Returns (store, main, aux, log, workload): aux is the
    auxiliary thread still alive after the last turn (or None); log has one
    record per turn.  evict_chunk_pages > 0 evicts in chunks of that many
    fresh pages (bounded transient pages); ``evict_inplace`` rewrites the
    sequence's own pages (no transient pages).  With ``extend`` every appended
    chunk (the auxiliary prompt, each turn) also runs its causal extend
    attention over every layer, timed in the record."""
    import torch
    w = wl.full_stack(turns=turns, turn_len=turn_len, prefix=prefix, num_layers=num_layers)
    rng = w._rng
    max_tok = prefix + turns * turn_len
    pages = max_tok // 16 + w.aux_private // 16 + 8
    if store is None:
        store = _sq.Store(num_layers, 32, 8, 128, num_pages=pages + pages // 8 + 64, max_seqs=4,
                          max_pages_per_seq=max_tok // 16 + 64, device=device,
                          evict_chunk_pages=evict_chunk_pages, evict_inplace=evict_inplace)
    main = store.seq_create()
    k, v = full_stack_inputs(w, -1, device)
    store.append(main, k, v)
    del k, v
    aux, pending = None, []
    log = []
    for t in range(turns):
        rec = dict(turn=t)
        if aux is not None:                                  # Phase 1
            store.release(aux)     # the finished thread's transient tokens go first
            if evict and pending:
                spans = store.spans(main)
                rec["evicted_spans"] = sorted(spans[c] for c in pending)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                rec["evict"] = store.evict(main, pending)
                torch.cuda.synchronize()
                rec["evict_ms"] = (time.perf_counter() - t0) * 1e3
            aux, pending = None, []
        if t % w.interval == 0:                              # Phase 2
            aux = store.fork(main, store.seq_info(main)["length"])
            ka, va = full_stack_aux_inputs(w, t, device)
            store.append(aux, ka, va)
            del ka, va
            if extend:
                rec["aux_extend_ms"] = _extend_all_layers(store, aux, w.aux_private, num_layers,
                                                          w.seed * 1000 + 6151 + t, device)
            live = store.spans(main)
            cur = sorted(live)
            tool_total = sum(e - s for s, e in live.values())
            if cur:
                order = rng.permutation(len(cur))
                got = 0
                for i in order:
                    if got >= w.evict_frac * tool_total:
                        break
                    c = cur[i]
                    pending.append(c)
                    got += live[c][1] - live[c][0]
        r = w.reasoning[t]                                   # Phase 3
        k, v = full_stack_inputs(w, t, device)
        start = store.seq_info(main)["length"]
        store.append(main, k, v)
        store.span_mark(main, t, start + r, start + turn_len)
        del k, v
        if extend:
            rec["extend_ms"] = _extend_all_layers(store, main, turn_len, num_layers,
                                                  w.seed * 1000 + 4049 + t, device)
        seqs = [main] if aux is None else [main, aux]
        rec["length"] = store.seq_info(main)["length"]
        rec["batch"] = len(seqs)
        if decode:
            q = wl.device_normal_bf16((len(seqs), 32, 128), w.seed * 1000 + 7919 + t, device)
            out = torch.empty((len(seqs), 32, 128), dtype=torch.float32, device=device)
            # the median of three timed steps after an untimed one: a single
            # sample also carries one-time costs (the first reads of the
            # turn's new pages, the clocks ramping up after host-only work),
            # which differ between runs that do and do not extend each turn
            walls = []
            for rep in range(4):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for layer in range(num_layers):
                    store.decode(layer, seqs, q, out=out)
                torch.cuda.synchronize()
                if rep:
                    walls.append((time.perf_counter() - t0) * 1e3)
            rec["decode_ms"] = sorted(walls)[1]
            rec["kv_bytes"] = store.plan_info(seqs)["kv_bytes"] * num_layers
            if on_turn is not None:
                on_turn(t, store, seqs, q, out)
        rec["live_pages"] = store.stats()["live_pages"]
        rec["aux_fork_len"] = (store.seq_info(aux)["length"] - w.aux_private) if aux is not None else None
        rec["aux_turn"] = (t - t % w.interval) if aux is not None else None
        log.append(rec)
    return store, main, aux, log, w
