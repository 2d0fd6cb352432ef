"""Span eviction reduced to index arithmetic, in plain Python/NumPy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

``clear_kv(Delta_ids)`` (Algorithm 1, Phase 1) removes from the context every
token of the tool responses named by the auxiliary thread's ``del_cursors``
command (§3.1, steps 3-4).  A cursor names a tool call together with its
response (the footnote to the Goal paragraph of §3), read here as one
half-open range [start, end) of the sequence's current logical positions.
Training presents the model with the same deletion as a mask (Algorithm 2
``BuildMask``; "Simulated Eviction" in §3.3), so the served (compacted) cache
must attend exactly like the masked one.

With ``L`` tokens and the evicted ranges:

    keep[i]   = 0 if i lies in an evicted range, else 1
    dst[i]    = sum_{j < i} keep[j]          (exclusive prefix sum)
    L'        = sum_i keep[i]
    src_of[t] = the i with keep[i] = 1 and dst[i] = t,   t in [0, L')

The compacted logical view is ``view[src_of]``: kept tokens keep their order
and their values, and the position array is carried along (retained keys keep
the RoPE positions they were cached with; nothing is re-rotated).
"""

from __future__ import annotations

import numpy as np


def keep_mask(length, spans):
    """keep[i] = 0 iff i is inside one of the half-open ``spans``."""
    keep = np.ones(int(length), dtype=np.uint8)
    for start, end in spans:
        if not (0 <= start <= end <= length):
            raise ValueError(f"span [{start}, {end}) outside [0, {length})")
        keep[start:end] = 0
    return keep


def exclusive_scan(keep):
    """dst[i] = number of kept tokens before i (a running count)."""
    dst = np.zeros(len(keep), dtype=np.int64)
    run = 0
    for i, flag in enumerate(np.asarray(keep).tolist()):
        dst[i] = run
        run += int(flag)
    return dst


def inverse_map(keep, dst):
    """src_of[dst[i]] = i for every kept i."""
    keep = np.asarray(keep)
    n_kept = int(keep.astype(np.int64).sum())
    src_of = np.full(n_kept, -1, dtype=np.int64)
    for i in range(len(keep)):
        if keep[i]:
            src_of[dst[i]] = i
    return src_of


def plan(length, spans):
    """(keep, dst, src_of, L', f) for evicting ``spans`` from ``length`` tokens.

    f is the first evicted index (``length`` when nothing is evicted).
    """
    keep = keep_mask(length, spans)
    dst = exclusive_scan(keep)
    src_of = inverse_map(keep, dst)
    evicted = np.flatnonzero(keep == 0)
    first = int(evicted[0]) if len(evicted) else int(length)
    return keep, dst, src_of, len(src_of), first


def compact(view, keep):
    """Rows of ``view`` (first axis = token) whose keep flag is set, in order."""
    keep = np.asarray(keep).astype(bool)
    return np.asarray(view)[keep]


def shift_span(start, end, evicted_spans):
    """Where a retained span lands after the evicted spans are removed: both
    ends move left by the number of evicted tokens before them."""
    before_s = sum(max(0, min(e, start) - s) for s, e in evicted_spans)
    before_e = sum(max(0, min(e, end) - s) for s, e in evicted_spans)
    return start - before_s, end - before_e
