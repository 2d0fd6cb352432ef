#!/usr/bin/env python3
"""Benchmark of the SideQuest KV hot path on one MI355X.

Workload (the step that is timed): one decode step of 8 concurrent agent
tasks at 128K context, each a main thread plus a forked auxiliary thread that
shares all but the last pages of the main thread's cache (16 queries; 32
query heads, 8 KV heads, head size 128, bf16 K/V).  A step appends the new
token of every sequence (sq_append_batch) and runs decode attention over the
shared paged cache (sq_decode_attn, AUTO mode: the shared prefix of each
main/auxiliary pair is read once by the multi-query MFMA tile).

value  = decode K/V bytes the method must read per step (shared pages once)
         / measured step time, in GB/s (inputs resident in HBM).
Also reported: tokens/s, the per-sequence modes, span eviction (64K context,
65% of tokens in whole tool spans removed) in GB/s, the dominant kernel's
roofline (HIP events on the library's stream), and the CPU oracle timed on a
bounded sample of the same workload.

Prints ONE JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "decode-attn HBM GB/s (% of 8 TB/s) + tokens/s at 128K ctx; evict GB/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--tasks", type=int, default=8)
    ap.add_argument("--ctx", type=int, default=131072)
    ap.add_argument("--legs",
                    default="decode,modes,evict,extend,outlier,variants,fp8,fullstack,postevict,cpu",
                    help="comma list of: decode, modes, evict, extend, outlier, variants, fp8, "
                         "fullstack, postevict, cpu, copy (a plain 1 GiB device copy used to "
                         "calibrate HBM byte counters)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-graph", action="store_true",
                    help="leave out the graph-replay timings (for rocprofv3 counter runs, "
                         "whose collection does not follow graph replays)")
    return ap.parse_args()


GRAPH_TIMINGS = True


DECODE_SOURCES = ("decode_kernels.hip", "decode_args.hpp", "sq_common.hpp", "fp8.hpp")
EXTEND_SOURCES = ("extend_kernels.hip", "extend_args.hpp", "sq_common.hpp", "fp8.hpp")


def kernel_sha(files=DECODE_SOURCES):
    """Hash of the sources a kernel is built from (the committed counter
    summaries are valid only for the sources they were taken on)."""
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2602_22603_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic(name):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_sources_sha") != kernel_sha():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def time_steps(sq, torch, store, seqs, mode, steps, warmup, kb, vb, qs, out):
    """Warm up, then time `steps` decode steps (append + attention) twice:
    first bare (wall clock between two synchronisations; the headline rate),
    then instrumented (HIP events around every step and, inside the library,
    around every kernel on its launch stream; these events cost the GPU some
    microseconds per step, so the second pass gives the kernel durations and
    step percentiles, not the rate)."""
    n = len(seqs)
    for i in range(warmup):
        store.append_batch(seqs, kb[i], vb[i])
        store.decode(0, seqs, qs[i], out=out, mode=mode)
    torch.cuda.synchronize()
    st0 = store.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(warmup, warmup + steps):
        store.append_batch(seqs, kb[i], vb[i])
        store.decode(0, seqs, qs[i], out=out, mode=mode)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st1 = store.stats()
    ms = (t1 - t0) * 1e3 / steps
    kv_bytes = (st1["decode_kv_bytes"] - st0["decode_kv_bytes"]) / steps
    logical = (st1["decode_kv_bytes_logical"] - st0["decode_kv_bytes_logical"]) / steps

    store.profile_enable(True)
    store.profile_read()
    plan = store.plan_info(seqs, mode)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for j, i in enumerate(range(warmup, warmup + steps)):
        ev[j][0].record()
        store.append_batch(seqs, kb[i], vb[i])
        store.decode(0, seqs, qs[i], out=out, mode=mode)
        ev[j][1].record()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    prof = store.profile_read()
    store.profile_enable(False)
    return dict(ms_per_step=ms, kv_bytes_per_step=kv_bytes, kv_bytes_logical_per_step=logical,
                gbps=kv_bytes / (ms * 1e-3) / 1e9, tokens_per_s=n / (ms * 1e-3), prof=prof,
                plan=plan, step_ms=percentiles([a.elapsed_time(b) for a, b in ev]),
                instrumented_ms_per_step=(t3 - t2) * 1e3 / steps)


def time_fused_steps(sq, torch, store, seqs, mode, steps, warmup, kb, vb, qs, out):
    """The same decode steps through sq_step_begin + sq_step_attn (the append
    fused into the merge kernel): bare wall clock, then instrumented."""
    n = len(seqs)

    def step(i):
        store.step_begin(seqs, mode)
        store.step_attn(0, kb[i][0], vb[i][0], qs[i], out=out)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    st0 = store.stats()
    t0 = time.perf_counter()
    for i in range(warmup, warmup + steps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st1 = store.stats()
    ms = (t1 - t0) * 1e3 / steps
    kv_bytes = (st1["decode_kv_bytes"] - st0["decode_kv_bytes"]) / steps
    store.profile_enable(True)
    store.profile_read()
    for i in range(warmup, warmup + steps):
        step(i)
    torch.cuda.synchronize()
    prof = store.profile_read()
    store.profile_enable(False)
    kern = prof["decode_mfma_ms"] / max(1, prof["decode_mfma_launches"])
    return dict(ms_per_step=round(ms, 4), gbps=round(kv_bytes / (ms * 1e-3) / 1e9, 1),
                tokens_per_s=round(n / (ms * 1e-3), 1), kv_bytes_per_step=kv_bytes,
                kernel_ms=round(kern, 5),
                merge_ms=round(prof["decode_merge_ms"] / max(1, prof["decode_merge_launches"]), 5))


def decode_step_paths(torch, wl, store, seqs, reps=10):
    """One decode step of every layer at the store's current state, three ways:
    sq_append_batch then sq_decode_attn per layer; sq_step_begin then
    sq_step_attn per layer; sq_step_begin then a replay of the captured
    sq_step_attn calls.  Median wall clock per step (synchronised after each),
    so host time counts."""
    nl, b = store.num_layers, len(seqs)
    kn = wl.device_normal_bf16((nl, b, store.num_kv_heads, store.head_dim), 71, "cuda")
    vn = wl.device_normal_bf16((nl, b, store.num_kv_heads, store.head_dim), 72, "cuda")
    q = wl.device_normal_bf16((nl, b, store.num_q_heads, store.head_dim), 73, "cuda")
    outs = [torch.empty((b, store.num_q_heads, store.head_dim), dtype=torch.float32, device="cuda")
            for _ in range(nl)]

    def per_call():
        store.append_batch(seqs, kn, vn)
        for l in range(nl):
            store.decode(l, seqs, q[l], out=outs[l])

    def layers():
        for l in range(nl):
            store.step_attn(l, kn[l], vn[l], q[l], out=outs[l])

    def fused():
        store.step_begin(seqs)
        layers()
    fused()                       # an open step for the capture to record
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layers()

    def graph():
        store.step_begin(seqs)
        g.replay()
    res = {}
    kv = store.plan_info(seqs)["kv_bytes"] * nl
    for name, fn in (("per_call", per_call), ("fused", fused), ("fused_graph", graph)):
        for _ in range(2):
            fn()
        walls = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            walls.append((time.perf_counter() - t0) * 1e3)
        med = sorted(walls)[len(walls) // 2]
        res[name + "_ms"] = round(med, 3)
        res[name + "_gbps"] = round(kv / (med * 1e-3) / 1e9, 1)
    del g
    return res


def percentiles(xs):
    """p10 / median / p90 of a list of step times (ms)."""
    xs = sorted(xs)
    pick = lambda f: xs[min(len(xs) - 1, int(round(f * (len(xs) - 1))))]
    return dict(p10=round(pick(0.1), 4), median=round(pick(0.5), 4), p90=round(pick(0.9), 4))


class Flusher:
    """Writes a 1 GiB buffer (untimed) so that the next step starts with the
    256 MB MALL and the L2 holding none of its data."""

    def __init__(self, torch):
        self.torch = torch
        self.buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        self.n = 0

    def __call__(self):
        self.n += 1
        self.buf.fill_(self.n & 255)


def time_events(torch, fn, reps, flush=None):
    """Per-call GPU time of fn() (HIP events on the current stream), optionally
    with a cache flush before each call; returns percentiles in ms."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        if flush is not None:
            flush()
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return percentiles([a.elapsed_time(b) for a, b in ev])


def graph_time(torch, fn, reps, flush=None):
    """GPU time of fn() with the host out of the way: fn's launches captured
    in a HIP graph of 20 calls and replayed, time per call.  Cold (flush
    given): the graph holds 20 (cache flush, call) pairs, and the time of a
    graph of the 20 flushes alone is taken off.  Percentiles in ms over
    reps replays; None with --no-graph."""
    if not GRAPH_TIMINGS:
        return None
    n = 20

    def replay_ms(body):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                body()
        g.replay()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record()
            g.replay()
            b.record()
        torch.cuda.synchronize()
        del g
        return [a.elapsed_time(b) for a, b in ev]

    if flush is None:
        return percentiles([t / n for t in replay_ms(fn)])

    def both():
        flush()
        fn()
    with_call = replay_ms(both)
    alone = sorted(replay_ms(flush))[len(with_call) // 2]
    return percentiles([(t - alone) / n for t in with_call])


def evict_gpu_time(torch, store, victim, ids, reps, flush):
    """GPU time of one eviction call's device work (index, gather and the
    page-table writes, with the gaps between them on the GPU), the host out
    of the way: one event pair around the call, recorded while the GPU is
    still busy with work queued before it - a spin kernel (warm: it touches
    no memory) or the 1 GiB cache flush (cold) - so that the call's
    launches are all queued before the GPU reaches the first event.
    Percentiles in ms."""
    res = {}
    for temp in ("warm", "cold"):
        times = []
        for r in range(reps + 1):
            f = victim()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            if temp == "cold":
                flush()
            else:
                torch.cuda._sleep(1_000_000)
            a.record()
            store.evict(f, ids)
            b.record()
            torch.cuda.synchronize()
            if r >= 1:
                times.append(a.elapsed_time(b))
            store.release(f)
        res[temp] = percentiles(times)
    return res


def evict_bytes(stats, length, kept):
    """Algorithmic bytes of one eviction: the moved tokens' K, V (every layer
    and head) and positions read and written, plus the index arrays (keep
    u8 and dst i32 per old token, src_of i32 per kept token) and the fresh
    page ids written to the page table."""
    return 2 * stats["bytes_moved"] + 5 * length + 4 * kept + 4 * stats["pages_allocated"]


def evict_leg(sq, torch, wl, reps=8, chunk=0, decode=True, align=0, remap=False, inplace=False):
    """The 64K compaction: sq_evict_spans of 40 tool spans (>= 65% of the
    tokens) on a branch forked over the whole context, repeated.  Timed
    warm (back to back: the ~180 MB read and written fit the 256 MB MALL)
    and cold (a 1 GiB write flushes the MALL and L2 before each call).
    GB/s divide the algorithmic bytes by the index kernel plus the gather
    (the library's HIP events around each launch, which also see the
    host's submission of the launch when the GPU waits for it), by the
    call's device work with the host out of the way (evict_gpu_time), and
    by the wall clock of the whole call."""
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k(evict_chunk_pages=chunk, align=align,
                                                       evict_remap=remap, evict_inplace=inplace)
    L = w.length
    if not inplace:
        del k, v
    torch.cuda.synchronize()
    flush = Flusher(torch)
    med = lambda xs: sorted(xs)[len(xs) // 2]
    runs = {}
    stats = None

    def victim():
        """The sequence to evict from: a branch forked over the whole
        context (aligned: it aliases every page of the base), or, in place,
        a sequence that alone holds its pages (appended anew)."""
        if not inplace:
            return store.fork(base, L)
        h = store.seq_create()
        store.append(h, k, v)
        for c, (s0, e0) in enumerate(w.spans):
            store.span_mark(h, c, s0, e0)
        return h
    for temp in ("warm", "cold"):
        walls = []
        store.profile_enable(True)
        for r in range(reps + 1):
            f = victim()
            if temp == "cold":
                flush()
            torch.cuda.synchronize()
            if r == 1:
                store.profile_read()  # the first call warms up
            t0 = time.perf_counter()
            stats = store.evict(f, w.evict_ids)
            torch.cuda.synchronize()
            if r >= 1:
                walls.append(time.perf_counter() - t0)
            store.release(f)
        prof = store.profile_read()
        store.profile_enable(False)
        kern = (prof["evict_scan_ms"] + prof["evict_gather_ms"]) / reps
        runs[temp] = dict(walls=walls, kern=kern, prof=prof)
    gpu = evict_gpu_time(torch, store, victim, w.evict_ids, reps, flush)
    kept = L - stats["tokens_removed"]
    alg = evict_bytes(stats, L, kept)
    wall = {t: med(runs[t]["walls"]) for t in runs}
    prof = runs["cold"]["prof"]
    per = lambda key, n: prof[key] / max(1, prof[n])
    info = dict(
        workload=f"64K tokens, 40 tool + 40 reasoning spans, evict >= 65% (got "
                 f"{stats['tokens_removed'] / L:.3f})",
        evict_chunk_pages=chunk, remap=remap, inplace=inplace, span_align=align,
        tokens_removed=stats["tokens_removed"], tokens_moved=stats["tokens_moved"],
        pages_allocated=stats["pages_allocated"], pages_remapped=stats["pages_remapped"],
        bytes_read_plus_written=2 * stats["bytes_moved"], algorithmic_bytes=alg,
        gather_launches_per_call=prof["evict_gather_launches"] // reps,
        index_ms_cold=round(per("evict_scan_ms", "evict_scan_launches"), 5),
        gather_ms_per_call_cold=round(prof["evict_gather_ms"] / reps, 5),
        kernel_ms_per_call={t: round(runs[t]["kern"], 5) for t in runs},
        evict_gbps_cold=round(alg / (runs["cold"]["kern"] * 1e-3) / 1e9, 1) if runs["cold"]["kern"] else None,
        evict_gbps_warm=round(alg / (runs["warm"]["kern"] * 1e-3) / 1e9, 1) if runs["warm"]["kern"] else None,
        evict_wall_ms_median={t: round(wall[t] * 1e3, 4) for t in wall},
        evict_gbps_wall={t: round(alg / wall[t] / 1e9, 1) for t in wall},
        evict_gpu_ms=gpu,
        evict_gbps_gpu={t: round(alg / (gpu[t]["median"] * 1e-3) / 1e9, 1) for t in gpu})
    if info["evict_gbps_cold"]:
        info["frac_of_hbm_peak_cold"] = round(info["evict_gbps_cold"] / HBM_PEAK_GBPS, 4)
    if not decode:
        del flush
        if inplace:
            del k, v
        store.close()
        return info
    # decode on the compacted cache vs the full cache (batch 1)
    f = store.fork(base, L)
    store.evict(f, w.evict_ids)
    q = wl.device_normal_bf16((1, 32, 128), 77, "cuda")
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
    res, pct = {}, {}
    for name, seq in (("compacted", f), ("full", base)):
        step = lambda: store.decode(0, [seq], q, out=out)
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(32):
            step()
        torch.cuda.synchronize()
        res[name] = (time.perf_counter() - t0) * 1e3 / 32
        pct[name] = dict(warm=time_events(torch, step, 32), cold=time_events(torch, step, 16, flush),
                         graph_warm=graph_time(torch, step, 16),
                         graph_cold=graph_time(torch, step, 16, flush))
    del flush
    info.update(decode_ms_compacted=res["compacted"], decode_ms_full=res["full"],
                decode_step_ms=pct)
    store.close()
    return info


def _decode_split(torch, store, seqs, q, out, reps, flush=None, layers=(0,)):
    """A decode call (every layer in ``layers``, batch ``seqs``): GPU time
    per call from HIP events around it on the current stream (median over
    ``reps``, each after a cache flush when ``flush`` is given; the events
    also see the host's submission of the call when the GPU waits for it),
    the same from replays of the call captured in a HIP graph (no host
    between the events), then, in a second pass with the library's
    per-kernel events on (which add gaps of their own), the decode kernel
    and merge times within a call."""
    def call():
        for layer in layers:
            store.decode(layer, seqs, q, out=out)
    for _ in range(3):
        call()
    torch.cuda.synchronize()
    gpu = time_events(torch, call, reps, flush)
    graph = graph_time(torch, call, reps, flush)
    store.profile_enable(True)
    store.profile_read()
    for _ in range(reps):
        if flush is not None:
            flush()
        call()
    torch.cuda.synchronize()
    prof = store.profile_read()
    store.profile_enable(False)
    kv = store.plan_info(seqs)["kv_bytes"] * len(layers)
    med = gpu["median"]
    dec = (prof["decode_mfma_ms"] + prof["decode_valu_ms"]) / reps
    mrg = prof["decode_merge_ms"] / reps
    plan = store.plan_info(seqs)
    return dict(call_ms=gpu, graph_call_ms=graph, kv_bytes=kv,
                gbps_call=round(kv / (med * 1e-3) / 1e9, 1),
                gbps_graph=round(kv / (graph["median"] * 1e-3) / 1e9, 1) if graph else None,
                decode_kernel_ms=round(dec, 4), merge_ms=round(mrg, 4),
                launch_gaps_ms=round(med - dec - mrg, 4),
                gbps_decode_kernel=round(kv / (dec * 1e-3) / 1e9, 1) if dec else None,
                workgroups=plan["n_items_mfma"] + plan["n_items_valu"])


def post_eviction_leg(sq, torch, wl, reps=20):
    """Decode where eviction leaves it: the 64K context after its tool spans
    were evicted (22.7K tokens, batch 1), warm and cold; and the final
    36-layer step of the full-stack task after one-shot, chunked and
    in-place eviction (every layer, batch 1).  Each call split into decode
    kernel, merge and the rest (launch gaps, host)."""
    from paper_2602_22603_amd import drivers
    res = {}
    store, base, w, k, v = drivers.build_compaction64k()
    del k, v
    store.evict(base, w.evict_ids)
    q = wl.device_normal_bf16((1, 32, 128), 77, "cuda")
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
    flush = Flusher(torch)
    res["compacted64k"] = dict(tokens=store.seq_info(base)["length"],
                               warm=_decode_split(torch, store, [base], q, out, 50),
                               cold=_decode_split(torch, store, [base], q, out, 20, flush))
    store.close()
    del flush
    torch.cuda.empty_cache()
    for name, chunk, inplace in (("one_shot", 0, False), ("chunked_64", 64, False),
                                 ("in_place", 0, True)):
        store, main, aux, log, w = drivers.run_full_stack(evict=True, evict_chunk_pages=chunk,
                                                          evict_inplace=inplace, decode=False)
        seqs = [main] + ([aux] if aux is not None else [])
        qq = wl.device_normal_bf16((len(seqs), 32, 128), 79, "cuda")
        oo = torch.empty((len(seqs), 32, 128), dtype=torch.float32, device="cuda")
        pt = store.page_table(main)
        runs = 1 + sum(1 for i in range(1, len(pt)) if pt[i] != pt[i - 1] + 1)
        res["full_stack_final_" + name] = dict(
            tokens=store.seq_info(main)["length"], batch=len(seqs), page_id_runs=runs,
            peak_pages=store.stats()["peak_pages"],
            step=_decode_split(torch, store, seqs, qq, oo, 10, layers=range(w.num_layers)))
        store.close()
        torch.cuda.empty_cache()
    return res


def deferred_leg(sq, torch, wl, reps=8):
    """The 64K compaction's spans evicted deferred: the call's wall time
    (masks only, nothing moves), decode over the masked cache (every slot is
    still read, masked ones are skipped), then the compaction's wall time and
    decode over the compacted cache (batch 1)."""
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k()
    del k, v
    L = w.length
    q = wl.device_normal_bf16((1, 32, 128), 78, "cuda")
    out = torch.empty((1, 32, 128), dtype=torch.float32, device="cuda")
    defer_walls, compact_walls, dec = [], [], {}
    for r in range(reps + 2):
        f = store.fork(base, L)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = store.evict(f, w.evict_ids, deferred=True)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        if r == reps + 1:
            step = lambda: store.decode(0, [f], q, out=out)
            for _ in range(3):
                step()
            dec["masked"] = time_events(torch, step, 32)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        cst = store.compact(f)
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        if r >= 2:
            defer_walls.append(t1 - t0)
            compact_walls.append(t3 - t2)
        if r == reps + 1:
            step = lambda: store.decode(0, [f], q, out=out)
            for _ in range(3):
                step()
            dec["compacted"] = time_events(torch, step, 32)
        store.release(f)
    med = lambda xs: sorted(xs)[len(xs) // 2] * 1e3
    store.close()
    return dict(workload=f"64K tokens, the same 40 tool spans as the eviction leg, deferred "
                         f"(masked {st['tokens_masked']} of {L}), then compacted",
                tokens_masked=st["tokens_masked"], tokens_removed_by_compact=cst["tokens_removed"],
                defer_wall_ms_median=round(med(defer_walls), 4),
                compact_wall_ms_median=round(med(compact_walls), 4),
                decode_ms_masked=dec["masked"], decode_ms_compacted=dec["compacted"])


def outlier_leg(sq, torch, wl):
    """32K context with outlier channels: eviction of >= 50% of the tokens
    while the auxiliary thread is alive, then 64 decode steps of [main, aux]
    (append + attention)."""
    from paper_2602_22603_amd import drivers
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    store, main, aux, w, stats = drivers.build_outlier32k()
    torch.cuda.synchronize()
    kb = [wl.to_torch_bf16(w.step_k[i], "cuda") for i in range(w.steps)]
    vb = [wl.to_torch_bf16(w.step_v[i], "cuda") for i in range(w.steps)]
    qs = [wl.to_torch_bf16(w.q[i], "cuda") for i in range(w.steps)]
    out = torch.empty((2, 32, 128), dtype=torch.float32, device="cuda")
    st0 = store.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(w.steps):
        store.append_batch([main, aux], kb[i], vb[i])
        store.decode(0, [main, aux], qs[i], out=out)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / w.steps
    st1 = store.stats()
    kv = (st1["decode_kv_bytes"] - st0["decode_kv_bytes"]) / w.steps
    # the same steps' attention again, warm (back to back) and cold (MALL and
    # L2 flushed before each): ~110 MB per step fits the 256 MB MALL
    step = lambda: store.decode(0, [main, aux], qs[-1], out=out)
    flush = Flusher(torch)
    warm = time_events(torch, step, 32)
    cold = time_events(torch, step, 16, flush)
    del flush
    store.close()
    return dict(workload="32K tokens, 30 spans, 4 outlier channels x8, aux +512, evict >= 50% "
                         f"(got {stats['tokens_removed'] / w.main_len:.3f}), 64 steps [main, aux]",
                ms_per_step=round(ms, 4), kv_bytes_per_step=kv,
                gbps=round(kv / (ms * 1e-3) / 1e9, 1), tokens_per_s=round(2 / (ms * 1e-3), 1),
                attention_ms_warm=warm, attention_ms_cold=cold,
                gbps_cold_median=round(kv / (cold["median"] * 1e-3) / 1e9, 1))


BF16_PEAK_TFLOPS = 2500.0


def extend_leg(sq, torch, wl, reps=10):
    """An 8192-token chunk (a turn's tool output) appended to the 64K context
    after its tool spans were evicted, and to the same context uncompacted:
    causal extend attention over the cache (1 layer, 32q/8kv heads, 128)."""
    from paper_2602_22603_amd import drivers
    n = 8192
    store, base, w, k, v = drivers.build_compaction64k(extra_tokens=n + 64)
    del k, v
    full = store.fork(base, w.length)       # keeps the uncompacted view
    store.evict(base, w.evict_ids)
    kn = wl.device_normal_bf16((1, n, 8, 128), 91, "cuda")
    vn = wl.device_normal_bf16((1, n, 8, 128), 92, "cuda")
    store.append(base, kn, vn)
    store.append(full, kn, vn)
    del kn, vn
    q = wl.device_normal_bf16((n, 32, 128), 93, "cuda")
    out = torch.empty((n, 32, 128), dtype=torch.float32, device="cuda")
    res = {}
    for name, seq in (("compacted", base), ("full", full)):
        L = store.seq_info(seq)["length"]
        step = lambda: store.extend(0, seq, q, out=out)
        for _ in range(2):
            step()
        store.profile_enable(True)
        store.profile_read()
        pct = time_events(torch, step, reps)
        prof = store.profile_read()
        store.profile_enable(False)
        kern_ms = prof["extend_ms"] / max(1, prof["extend_launches"])
        # useful flops: q.k and p.v for every (query head, visible key) pair
        pairs = n * (L - n) + n * (n + 1) // 2
        flops = 32 * 4 * 128 * pairs
        tflops = flops / (kern_ms * 1e-3) / 1e12
        res[name] = dict(prefix_tokens=L - n, chunk_tokens=n, call_ms=pct,
                         kernel_ms=round(kern_ms, 4), useful_tflops=round(tflops, 1),
                         frac_of_bf16_peak=round(tflops / BF16_PEAK_TFLOPS, 4),
                         tokens_per_s=round(n / (kern_ms * 1e-3), 1))
    # an auxiliary thread's 512-token prompt over the compacted context: a
    # short chunk, so the key range is split over several workgroups
    aux = store.fork(base, store.seq_info(base)["length"])
    ka = wl.device_normal_bf16((1, 512, 8, 128), 94, "cuda")
    store.append(aux, ka, ka)
    qa = wl.device_normal_bf16((512, 32, 128), 95, "cuda")
    oa = torch.empty((512, 32, 128), dtype=torch.float32, device="cuda")
    L = store.seq_info(aux)["length"]
    step = lambda: store.extend(0, aux, qa, out=oa)
    for _ in range(2):
        step()
    pct = time_events(torch, step, reps)
    pairs = 512 * (L - 512) + 512 * 513 // 2
    tf = 32 * 4 * 128 * pairs / (pct["median"] * 1e-3) / 1e12
    res["aux_prompt_512"] = dict(prefix_tokens=L - 512, chunk_tokens=512, call_ms=pct,
                                 useful_tflops=round(tf, 1),
                                 frac_of_bf16_peak=round(tf / BF16_PEAK_TFLOPS, 4))
    res["workload"] = ("8192-token chunk after the 64K context's tool spans were evicted "
                       f"(>= 65%), vs the uncompacted 64K context; 1 layer, 32q/8kv, 128; "
                       f"peak {BF16_PEAK_TFLOPS:.0f} TFLOP/s dense bf16")
    res["compute_saved"] = round(1 - res["compacted"]["kernel_ms"] / res["full"]["kernel_ms"], 4)
    store.close()
    return res


def variants_leg(sq, torch, wl, reps=20, window=128):
    """Attention options on the 128K shared-prefix batch with 64 query / 8 KV
    heads of dimension 64 and two layers: layer 0 attends to a window of the
    last 128 keys, layer 1 to every key, both with per-head sinks (a model
    whose layers alternate).  Times each layer's decode call and a fused
    step over both layers."""
    from paper_2602_22603_amd import drivers
    store, seqs, _ = drivers.build_shared128k(layers=2, heads=(64, 8, 64), keep_inputs=(),
                                              extra_tokens=2 * (reps + 8) + 16)
    B = len(seqs)
    q = wl.device_normal_bf16((B, 64, 64), 700, "cuda")
    kn = wl.device_normal_bf16((B, 8, 64), 701, "cuda")
    out = torch.empty((B, 64, 64), dtype=torch.float32, device="cuda")
    sinks = torch.randn(64, generator=torch.Generator().manual_seed(702)).float().to("cuda")
    res = {}
    for name, layer, w, sk in (("full", 1, 0, None), ("full_sinks", 1, 0, sinks),
                               ("window_sinks", 0, window, sinks)):
        call = lambda: store.decode(layer, seqs, q, out=out, window=w, sinks=sk)
        for _ in range(3):
            call()
        st0 = store.stats()
        store.profile_enable(True)
        store.profile_read()
        pct = time_events(torch, call, reps)
        prof = store.profile_read()
        store.profile_enable(False)
        kv = (store.stats()["decode_kv_bytes"] - st0["decode_kv_bytes"]) / reps
        kern = (prof["decode_mfma_ms"] + prof["decode_valu_ms"]) / max(1, reps)
        res[name] = dict(call_ms=pct, kernel_ms=round(kern, 5), kv_bytes=kv,
                         merge_ms=round(prof["decode_merge_ms"] / max(1, prof["decode_merge_launches"]), 5),
                         kernel_gbps=round(kv / (kern * 1e-3) / 1e9, 1))

    def step():
        store.step_begin(seqs, window=window)
        store.step_attn(0, kn, kn, q, out=out, window=window, sinks=sinks)
        store.step_attn(1, kn, kn, q, out=out, sinks=sinks)
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    st0 = store.stats()
    t0 = time.perf_counter()
    for _ in range(reps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    kv = (store.stats()["decode_kv_bytes"] - st0["decode_kv_bytes"]) / reps
    res["fused_step_two_layers"] = dict(ms_per_step=round(ms, 4), kv_bytes=kv,
                                        gbps=round(kv / (ms * 1e-3) / 1e9, 1))
    res["workload"] = (f"8 tasks x (main 131072 + forked aux 130816+512) tokens, 16 queries, "
                       f"64q/8kv heads, head_dim 64, layer 0 window {window} + sinks, "
                       f"layer 1 full (+ sinks), AUTO mode")
    store.close()
    return res


def fp8_leg(sq, torch, wl, steps=20, warmup=3):
    """The headline decode step on an 8-bit (E4M3) store: the same 128K
    shared-prefix batch, K/V scales 0.011 / 0.0095 (unit-variance K/V),
    append + attention per step; STREAM mode on the main threads alone."""
    from paper_2602_22603_amd import drivers
    total = steps + warmup
    chunk = 2048
    store, seqs, _ = drivers.build_shared128k(keep_inputs=(), extra_tokens=3 * total + 16 + chunk,
                                              kv_scales=[[0.011, 0.0095]])
    B = len(seqs)
    kb = [wl.device_normal_bf16((1, B, 8, 128), 800 + 3 * i, "cuda") for i in range(total)]
    vb = [wl.device_normal_bf16((1, B, 8, 128), 801 + 3 * i, "cuda") for i in range(total)]
    qs = [wl.device_normal_bf16((B, 32, 128), 802 + 3 * i, "cuda") for i in range(total)]
    out = torch.empty((B, 32, 128), dtype=torch.float32, device="cuda")
    r = time_steps(sq, torch, store, seqs, sq.ATTN_AUTO, steps, warmup, kb, vb, qs, out)
    prof, plan = r["prof"], r["plan"]
    kern = prof["decode_mfma_ms"] / max(1, prof["decode_mfma_launches"])
    # STREAM mode (the VALU kernel) on the 8 main threads alone (unique pages)
    mains = seqs[0::2]
    rs = time_steps(sq, torch, store, mains, sq.ATTN_STREAM, steps, warmup,
                    [x[:, 0::2].contiguous() for x in kb], [x[:, 0::2].contiguous() for x in vb],
                    [x[0::2].contiguous() for x in qs], out[0::2].contiguous())
    skern = rs["prof"]["decode_valu_ms"] / max(1, rs["prof"]["decode_valu_launches"])
    # a 2048-token chunk appended to one main thread (131K prefix), extended
    kn = wl.device_normal_bf16((1, chunk, 8, 128), 890, "cuda")
    store.append(seqs[0], kn, kn)
    qx = wl.device_normal_bf16((chunk, 32, 128), 891, "cuda")
    ox = torch.empty((chunk, 32, 128), dtype=torch.float32, device="cuda")
    call = lambda: store.extend(0, seqs[0], qx, out=ox)
    for _ in range(2):
        call()
    ext = time_events(torch, call, 5)
    L = store.seq_info(seqs[0])["length"]
    pairs = chunk * (L - chunk) + chunk * (chunk + 1) // 2
    ext_tflops = 32 * 4 * 128 * pairs / (ext["median"] * 1e-3) / 1e12
    store.close()
    return dict(workload="8 tasks x (main 131072 + forked aux 130816+512) tokens, 16-query step "
                         "(append + attention), 32q/8kv heads, head_dim 128, E4M3 K/V",
                ms_per_step=round(r["ms_per_step"], 4), gbps=round(r["gbps"], 1),
                tokens_per_s=round(r["tokens_per_s"], 1),
                kv_bytes_per_step=r["kv_bytes_per_step"], kernel_ms=round(kern, 5),
                kernel_gbps=round(plan["kv_bytes_mfma"] / (kern * 1e-3) / 1e9, 1),
                kernel_frac_of_hbm_peak=round(plan["kv_bytes_mfma"] / (kern * 1e-3) / 1e9 /
                                              HBM_PEAK_GBPS, 4),
                mains_only_stream_valu=dict(
                    ms_per_step=round(rs["ms_per_step"], 4), kernel_ms=round(skern, 5),
                    kernel_gbps=round(rs["kv_bytes_per_step"] / (skern * 1e-3) / 1e9, 1)),
                extend_2048_over_131k=dict(call_ms=ext, useful_tflops=round(ext_tflops, 1)))


def fullstack_leg(sq, torch, wl):
    """36 layers, 16K prefix + 30 turns of 8K tokens, auxiliary thread every 4
    turns; with one-shot eviction, with eviction in 64-page chunks (bounded
    transient pages), in place (no transient pages) and without eviction:
    peak KV bytes, the causal extend
    attention of every appended chunk (one-shot and no eviction) and the
    decode step (all 36 layers) at each turn's end."""
    from paper_2602_22603_amd import drivers
    page_bytes = 36 * 8 * 16 * 128 * 2 * 2
    res = {}
    for name, ev, chunk, inplace in (("with_eviction", True, 0, False),
                                     ("with_chunked_eviction", True, 64, False),
                                     ("with_inplace_eviction", True, 0, True),
                                     ("without_eviction", False, 0, False)):
        full = chunk == 0 and not inplace
        store, main, aux, log, w = drivers.run_full_stack(evict=ev, evict_chunk_pages=chunk,
                                                          extend=full, evict_inplace=inplace)
        st = store.stats()
        paths = decode_step_paths(torch, wl, store, [main] + ([aux] if aux is not None else [])) \
            if full else None
        final = log[-1]
        dec = [r["decode_ms"] for r in log]
        ev_ms = [r["evict_ms"] for r in log if "evict_ms" in r]
        moved = sum(r["evict"]["bytes_moved"] for r in log if "evict" in r)
        res[name] = dict(
            peak_kv_bytes=st["peak_pages"] * page_bytes, final_tokens=final["length"],
            decode_ms_final_step=round(final["decode_ms"], 3),
            decode_gbps_final_step=round(final["kv_bytes"] / (final["decode_ms"] * 1e-3) / 1e9, 1),
            decode_ms_sum_over_turns=round(sum(dec), 2),
            kv_bytes_read_over_turns=sum(r["kv_bytes"] for r in log),
            evictions=len(ev_ms), evict_ms_total=round(sum(ev_ms), 3),
            evict_gbps_wall=round(2 * moved / (sum(ev_ms) * 1e-3) / 1e9, 1) if ev_ms else None,
            extend_ms_over_turns=round(sum(r.get("extend_ms", 0) + r.get("aux_extend_ms", 0)
                                           for r in log), 1) if full else None,
            decode_step_paths_final=paths)
        store.close()
        torch.cuda.empty_cache()
    a, b = res["with_eviction"], res["without_eviction"]
    res["peak_kv_reduction"] = round(1 - a["peak_kv_bytes"] / b["peak_kv_bytes"], 4)
    res["extend_time_reduction"] = round(1 - a["extend_ms_over_turns"] / b["extend_ms_over_turns"], 4)
    res["peak_kv_reduction_chunked"] = round(
        1 - res["with_chunked_eviction"]["peak_kv_bytes"] / b["peak_kv_bytes"], 4)
    res["peak_kv_reduction_inplace"] = round(
        1 - res["with_inplace_eviction"]["peak_kv_bytes"] / b["peak_kv_bytes"], 4)
    res["kv_read_reduction"] = round(1 - a["kv_bytes_read_over_turns"] / b["kv_bytes_read_over_turns"], 4)
    return res


def _bf16_bits_to_f64(bits):
    import numpy as np
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _oracle_part(args):
    """The oracle's split partial (m, l, acc) of one KV head's query heads
    over one token range of the sample (runs in a worker, BLAS on 1 thread);
    returns (seconds, partial)."""
    from threadpoolctl import threadpool_limits
    from oracle import attention as oatt
    q, kbits, vbits = args
    with threadpool_limits(limits=1):
        kf = _bf16_bits_to_f64(kbits)[:, None, :]
        vf = _bf16_bits_to_f64(vbits)[:, None, :]
        t0 = time.perf_counter()
        part = oatt.partial(q, kf, vf, 1 / math.sqrt(128), 4)
        return time.perf_counter() - t0, part


def _oracle_warm(_):
    """Import what _oracle_part needs and wait a moment, so that every
    worker of the pool is up before the timed map."""
    from threadpoolctl import threadpool_limits  # noqa: F401
    from oracle import attention  # noqa: F401
    time.sleep(0.2)
    return 0


def _cpu_model():
    """The host CPU as /proc/cpuinfo names it, with its family / model /
    stepping (some virtual machines give only a short model name)."""
    info = {}
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if ":" in line:
                    k, v = line.split(":", 1)
                    info.setdefault(k.strip(), v.strip())
    except OSError:
        pass
    name = info.get("model name", "unknown")
    ids = "/".join(info.get(k, "?") for k in ("cpu family", "model", "stepping"))
    return f"{name} ({info.get('vendor_id', '?')}, family/model/stepping {ids})"


def cpu_leg(sample, wl, budget_s):
    """The float64 oracle on the host, over KV heads of task 0's main thread:
    first on one thread (BLAS pinned to 1), then split over every CPU the
    process may use, each worker taking one token range of one head (the
    oracle's split partials, combined by its merge and checked against the
    single-thread outputs)."""
    import multiprocessing as mp
    import numpy as np
    import torch
    from oracle import attention as oatt
    k, v = sample
    ctx = k.shape[1]
    rng = np.random.default_rng([2602, 2, 7])
    q = wl.bf16_value(wl.normal_bf16(rng, (32, 128)))
    bits = lambda t, g: t[0, :, g].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    heads = [(q[4 * g: 4 * g + 4], bits(k, g), bits(v, g)) for g in range(8)]
    bytes_per_head = ctx * 512
    t_one, single = 0.0, {}
    for g, h in enumerate(heads):
        dt, part = _oracle_part(h)
        t_one += dt
        single[g] = oatt.merge([part])
        if t_one >= budget_s:
            break
    one = bytes_per_head * len(single) / t_one / 1e9
    avail = len(os.sched_getaffinity(0))
    workers = max(1, min(avail, 64))
    chunks = max(1, -(-2 * workers // len(heads)))      # >= 2 units per worker
    bounds = [ctx * c // chunks for c in range(chunks + 1)]
    units = [(g, (h[0], h[1][a:b], h[2][a:b])) for g, h in enumerate(heads)
             for a, b in zip(bounds[:-1], bounds[1:])]
    # every worker is started and has imported the oracle before the clock runs
    with mp.get_context("spawn").Pool(workers) as pool:
        pool.map(_oracle_warm, range(workers), chunksize=1)
        t0 = time.perf_counter()
        parts = pool.map(_oracle_part, [u[1] for u in units], chunksize=1)
        t_all = time.perf_counter() - t0
    by_head = {}
    for (g, _), (_, part) in zip(units, parts):
        by_head.setdefault(g, []).append(part)
    err = max(float(np.max(np.abs(oatt.merge(by_head[g]) - single[g]))) for g in single)
    par = bytes_per_head * len(heads) / t_all / 1e9
    return dict(value=par, unit="GB/s", cores=workers, kind="oracle",
                sample=f"main thread of task 0: {ctx} tokens x 8 KV heads (4 query heads each), "
                       f"float64 NumPy oracle split into {len(units)} (head, token range) "
                       f"partials over {workers} worker processes ({t_all:.1f} s wall), merged "
                       f"by the oracle (max diff {err:.1e} from the single-thread outputs); "
                       f"single thread: {len(single)} heads in {t_one:.1f} s",
                value_1_thread=one, cpu_model=_cpu_model(), affinity_cpus=avail,
                blas_threads=1)


def main():
    global GRAPH_TIMINGS
    args = parse_args()
    GRAPH_TIMINGS = not args.no_graph
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2602_22603_amd import sq
    from paper_2602_22603_amd import workload as wl
    sq.lib()
    legs = set(args.legs.split(","))
    torch.cuda.set_device(0)
    total = args.warmup + args.steps
    n_modes = 5 if "modes" in legs else 0
    per_call = args.warmup + 2 * args.steps      # tokens one time_steps call appends
    extra = per_call * (2 + n_modes) + total + 16
    log(f"building {args.tasks} tasks at {args.ctx} tokens ...")
    from paper_2602_22603_amd import drivers
    store, seqs, inputs = drivers.build_shared128k(tasks=args.tasks, ctx=args.ctx,
                                                   extra_tokens=extra)
    sample = inputs[0][:2]
    B = len(seqs)
    kb = [wl.device_normal_bf16((1, B, 8, 128), 500 + 3 * i, "cuda") for i in range(total)]
    vb = [wl.device_normal_bf16((1, B, 8, 128), 501 + 3 * i, "cuda") for i in range(total)]
    qs = [wl.device_normal_bf16((B, 32, 128), 502 + 3 * i, "cuda") for i in range(total)]
    out = torch.empty((B, 32, 128), dtype=torch.float32, device="cuda")

    log("timing decode steps (AUTO) ...")
    main_res = time_steps(sq, torch, store, seqs, sq.ATTN_AUTO, args.steps, args.warmup,
                          kb, vb, qs, out)
    flush = Flusher(torch)
    ci = iter(range(total, 2 * total))

    def cold_step():
        i = next(ci)
        store.append_batch(seqs, kb[i % total], vb[i % total])
        store.decode(0, seqs, qs[i % total], out=out)
    step_cold = time_events(torch, cold_step, min(args.steps, total), flush)
    del flush
    log("timing fused decode steps (append in the merge) ...")
    fused = time_fused_steps(sq, torch, store, seqs, sq.ATTN_AUTO, args.steps, args.warmup,
                             kb, vb, qs, out)
    prof, plan = main_res["prof"], main_res["plan"]
    if plan["n_items_mfma"]:
        kname, kms, kn, kbytes = ("k_decode_mfma", prof["decode_mfma_ms"],
                                  prof["decode_mfma_launches"], plan["kv_bytes_mfma"])
    else:
        kname, kms, kn, kbytes = ("k_decode_valu", prof["decode_valu_ms"],
                                  prof["decode_valu_launches"], plan["kv_bytes_valu"])
    kavg = kms / max(1, kn)
    achieved = kbytes / (kavg * 1e-3) / 1e9
    traffic = read_traffic("decode_mfma_shared128k_traffic.txt")
    roofline = dict(bound="hbm", kernel=kname, achieved=round(achieved, 1), peak=HBM_PEAK_GBPS,
                    unit="GB/s", frac=round(achieved / HBM_PEAK_GBPS, 4), traffic=traffic,
                    algorithmic_bytes_per_launch=kbytes, avg_launch_ms=round(kavg, 5),
                    merge_avg_ms=round(prof["decode_merge_ms"] / max(1, prof["decode_merge_launches"]), 5),
                    append_avg_ms=round(prof["append_ms"] / max(1, prof["append_launches"]), 5))
    modes = {}
    if "modes" in legs:
        for name, m in (("stream_valu", sq.ATTN_STREAM), ("per_sequence_mfma", sq.ATTN_MFMA),
                        ("shared_prefix", sq.ATTN_SHARED_PREFIX)):
            log(f"timing mode {name} ...")
            r = time_steps(sq, torch, store, seqs, m, args.steps, args.warmup, kb, vb, qs, out)
            # requested: the bytes the mode's launches read (a per-sequence
            # mode reads each shared prefix once per sequence, and the
            # caches serve part of the repeats); unique: each page once
            modes[name] = dict(ms_per_step=round(r["ms_per_step"], 4),
                               kv_bytes_requested_per_step=r["kv_bytes_per_step"],
                               gbps_requested_bytes=round(r["gbps"], 1),
                               gbps_unique_bytes=round(main_res["kv_bytes_per_step"] /
                                                       (r["ms_per_step"] * 1e-3) / 1e9, 1),
                               tokens_per_s=round(r["tokens_per_s"], 1))
        # the per-sequence kernels on unique pages: the 8 main threads alone
        mains = seqs[0::2]
        for name, m in (("mains_only_stream_valu", sq.ATTN_STREAM),
                        ("mains_only_mfma", sq.ATTN_MFMA)):
            log(f"timing {name} ...")
            r = time_steps(sq, torch, store, mains, m, args.steps, args.warmup,
                           [x[:, 0::2].contiguous() for x in kb], [x[:, 0::2].contiguous() for x in vb],
                           [x[0::2].contiguous() for x in qs], out[0::2].contiguous())
            kern = r["prof"]["decode_valu_ms" if m == sq.ATTN_STREAM else "decode_mfma_ms"]
            nk = r["prof"]["decode_valu_launches" if m == sq.ATTN_STREAM else "decode_mfma_launches"]
            modes[name] = dict(ms_per_step=round(r["ms_per_step"], 4),
                               gbps=round(r["gbps"], 1),
                               kernel_ms=round(kern / max(1, nk), 4),
                               kernel_gbps=round(r["kv_bytes_per_step"] / (kern / max(1, nk) * 1e-3) / 1e9, 1))
    store.close()
    del kb, vb, qs
    torch.cuda.empty_cache()
    evict = None
    if "evict" in legs:
        log("eviction leg (64K compaction) ...")
        evict = evict_leg(sq, torch, wl)
        torch.cuda.empty_cache()
        evict["chunked_256_pages"] = evict_leg(sq, torch, wl, chunk=256, decode=False)
        # tool spans that start and end on page boundaries: gathered, or remapped
        evict["page_aligned_spans_copy"] = evict_leg(sq, torch, wl, decode=False, align=16)
        evict["page_aligned_spans_remap"] = evict_leg(sq, torch, wl, decode=False, align=16,
                                                      remap=True)
        # the tail rewritten in the sequence's own pages (no transient page)
        evict["in_place"] = evict_leg(sq, torch, wl, decode=False, inplace=True)
        evict["deferred"] = deferred_leg(sq, torch, wl)
    if "copy" in legs:
        log("calibration copy: 1 GiB device-to-device ...")
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    extend = None
    if "extend" in legs:
        log("extend leg (8192-token chunk over the 64K context) ...")
        extend = extend_leg(sq, torch, wl)
        torch.cuda.empty_cache()
    outlier = None
    if "outlier" in legs:
        log("32K outlier leg ...")
        outlier = outlier_leg(sq, torch, wl)
    fp8 = None
    if "fp8" in legs:
        log("8-bit KV store leg (128K shared prefix) ...")
        fp8 = fp8_leg(sq, torch, wl, args.steps, args.warmup)
        torch.cuda.empty_cache()
    variants = None
    if "variants" in legs:
        log("attention options leg (windows and sinks, 64q/8kv/64) ...")
        variants = variants_leg(sq, torch, wl)
        torch.cuda.empty_cache()
    fullstack = None
    if "fullstack" in legs:
        log("full-stack leg (36 layers, 16K -> 256K) ...")
        fullstack = fullstack_leg(sq, torch, wl)
    post = None
    if "postevict" in legs:
        log("post-eviction decode leg (compacted 64K; 36-layer final steps) ...")
        post = post_eviction_leg(sq, torch, wl)
        torch.cuda.empty_cache()
    cpu = None
    if "cpu" in legs:
        log("oracle CPU baseline ...")
        cpu = cpu_leg(sample, wl, args.cpu_seconds)
    res = {
        "metric": METRIC,
        "value": round(main_res["gbps"], 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.tasks} tasks x (main {args.ctx} + forked aux "
                               f"{args.ctx - 256}+512) tokens, 16-query decode step "
                               f"(append + attention), 1 layer, 32q/8kv heads, head_dim 128, "
                               f"page 16, AUTO mode",
                   "global_batch": B, "seq_len": args.ctx, "parallelism": "single GPU"},
        "frac_of_hbm_peak": round(main_res["gbps"] / HBM_PEAK_GBPS, 4),
        "tokens_per_s": round(main_res["tokens_per_s"], 1),
        "step_ms_warm": main_res["step_ms"],
        "instrumented_ms_per_step": round(main_res["instrumented_ms_per_step"], 4),
        "fused_step": fused,
        "step_ms_cold": step_cold,
        "kv_bytes_per_step": main_res["kv_bytes_per_step"],
        "kv_bytes_logical_per_step": main_res["kv_bytes_logical_per_step"],
        "roofline": roofline,
        "modes": modes,
        "evict": evict,
        "extend": extend,
        "outlier32k": outlier,
        "attention_options": variants,
        "kv_fp8": fp8,
        "full_stack": fullstack,
        "post_eviction_decode": post,
        "cpu_baseline": cpu,
        "kernel_sources_sha": kernel_sha(),
        "extend_kernel_sources_sha": kernel_sha(EXTEND_SOURCES),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
